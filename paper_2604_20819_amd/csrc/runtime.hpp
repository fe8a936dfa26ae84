// Per-device runtime state and helpers shared by the forward and backward
// drivers (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <chrono>
#include <mutex>
#include <string>
#include <vector>

#include "cqsa.h"
#include "errors.hpp"
#include "plan.hpp"

namespace cqsa {

// Waves the GPU holds at once at the inner kernels' occupancy (256 CUs x 4
// SIMDs x 2 waves), and the launch length, in rounds of them, from which the
// drivers run consecutive inner launches one after the other on the caller's
// stream: such a launch has a negligible tail, and two of them in flight only
// share the GPU (which costs time: in the backward, dQ beside dK/dV was 2-8 %
// slower than the two in turn from 8 rounds up).  Shorter launches go to two
// streams, so that one fills the other's tail.
constexpr int64_t kResidentWaves = 256 * 8;
constexpr int64_t kSerialRounds = 8;
inline bool serial_launch(int64_t waves) { return waves >= kSerialRounds * kResidentWaves; }

// Library-owned streams and caches of one device.  All streams use the
// default priority.
struct DevCtx {
  int device = -1;
  bool ready = false;
  hipStream_t copy = nullptr;   // staging copies (H2D or D2D)
  hipStream_t aux = nullptr;    // forward merges, or statistics device -> host
  hipStream_t lane = nullptr;   // second compute stream (short launches: odd forward groups, backward dQ)
  hipEvent_t ws_free = nullptr; // recorded after the last call's last use of the workspace
  bool ws_free_valid = false;
  void* ws = nullptr;           // cached device workspace (built-in allocator)
  size_t ws_bytes = 0;
  void* pin = nullptr;          // cached pinned host staging for host accumulation
  size_t pin_bytes = 0;
  // pinned host ring the plan images are uploaded from (see upload_image)
  void* img_pin[2] = {nullptr, nullptr};
  size_t img_bytes[2] = {0, 0};
  hipEvent_t img_done[2] = {nullptr, nullptr};
  bool img_valid[2] = {false, false};
  int img_next = 0;
  std::vector<hipEvent_t> sync_events;  // reusable non-timing events
  // the fixed scratch array of cqsa_forward_noalloc on this device (its device
  // address, from hipGetSymbolAddress at set-up) and the event after the
  // last no-allocation call's last use of it
  void* scratch = nullptr;
  hipEvent_t scratch_free = nullptr;
  bool scratch_free_valid = false;
  // the inner forward's tile-decision counters (cqsa_set_tile_counting),
  // allocated on first use; calls reach them in workspace order
  unsigned long long* tile_count = nullptr;
  std::mutex mu;
};

// Non-timing events created with the context, so that a call that must not
// allocate finds its synchronisation events in place.
constexpr size_t kSetupEvents = 16;

DevCtx* device_ctx(cqsa_status* st);  // context of the current device (created on first use)

// Workspace of one call: from the caller allocator when one is installed,
// else the cached per-device buffer.
struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  bool from_hook = false;
};
cqsa_status acquire_workspace(DevCtx* c, size_t bytes, Workspace* ws);
void release_workspace(DevCtx* c, Workspace* ws, hipStream_t s);
cqsa_status acquire_pinned(DevCtx* c, size_t bytes, void** out);
// Enqueues the H2D copy of a plan image on stream s.  The bytes go through a
// ring of two pinned host buffers: a copy from pageable memory would block
// the host until the stream reached it (serialising consecutive calls), and
// an asynchronous copy must not read a plan the caller may destroy as soon
// as the call returns.  A buffer is refilled once its previous copy is done.
cqsa_status upload_image(DevCtx* c, const std::vector<uint8_t>& image, void* dst, hipStream_t s);

// Event pairs for the optional per-stage timing of the last call.
enum Stage { kStStage = 0, kStInner, kStMerge, kStFinal, kStD2H, kStCount };
struct CallRecord {
  bool timing = false;
  // tile counting of the last call: the counters' copy in pinned host memory
  // (allocated on first use, per thread) and the event after that copy
  int counted = 0;                          // counters copied (0: none)
  unsigned long long* tile_host = nullptr;
  hipEvent_t tile_done = nullptr;
  std::vector<hipEvent_t> owned;                       // destroyed on reset
  std::vector<std::pair<hipEvent_t, hipEvent_t>> spans[kStCount];
  hipEvent_t wall0 = nullptr, wall1 = nullptr;
  double host_merge_ms = 0.0;
  double host_final_ms = 0.0;
  cqsa_run_stats stats{};
  void reset();
  hipEvent_t make();                                    // timing event owned by the record
};
CallRecord& call_record();
bool timing_enabled();
bool tile_counting_enabled();
// The device's first n tile counters (n <= 8), zeroed on stream s (allocated
// on first use).
cqsa_status tile_counters_begin(DevCtx* c, hipStream_t s, int n, unsigned long long** out);
// Copies the first n counters to the call record after the work on s (the
// call's end); cqsa_last_stats reads them: [0..2] the forward's or the dQ
// kernel's decisions, [3..5] the dK/dV kernel's.
cqsa_status tile_counters_end(DevCtx* c, CallRecord& rec, hipStream_t s, int n);

// Checks shared by forward and backward.
cqsa_status check_tensor(const cqsa_tensor* t, const char* name, const cqsa_plan_t* p,
                         cqsa_dtype want, cqsa_mem where);

inline cqsa_status hip_fail(hipError_t e, const char* what) {
  return fail(CQSA_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define CQSA_HIP(expr)                                                   \
  do {                                                                   \
    hipError_t e_ = (expr);                                              \
    if (e_ != hipSuccess) {                                              \
      if (e_ == hipErrorOutOfMemory) return fail(CQSA_ERR_DEVICE_OOM, #expr); \
      return hip_fail(e_, #expr);                                        \
    }                                                                    \
  } while (0)

}  // namespace cqsa
