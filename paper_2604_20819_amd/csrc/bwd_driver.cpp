// cqsa_backward (placeholder until the backward kernels land).
#include "runtime.hpp"

extern "C" cqsa_status cqsa_backward(const cqsa_plan_t*, const cqsa_tensor*, const cqsa_tensor*,
                                     const cqsa_tensor*, const cqsa_tensor*, const float*, cqsa_mem,
                                     const cqsa_tensor*, cqsa_tensor*, cqsa_tensor*, cqsa_tensor*,
                                     float, void*) {
  cqsa::clear_error();
  return cqsa::fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: not built yet");
}
