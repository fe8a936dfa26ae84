// Inner backward kernels (placeholder).
#include "hip_common.hpp"
