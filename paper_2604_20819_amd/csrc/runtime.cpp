// Runtime shared by the drivers: per-device streams, workspace caching,
// the caller-allocator hook, per-stage timing, and the C-ABI entry points
// that are not planning or compute.
#include "runtime.hpp"
#include "kernels.hpp"
#include "streamer.hpp"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>

namespace cqsa {

// Workspace of cqsa_forward_noalloc.  In host code this name is a host-side
// stand-in, not a device address: host code uses only the address that
// hipGetSymbolAddress returns for the current device (DevCtx::scratch).
static __device__ __align__(256) char scratch[CQSA_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_ctx_mu;
DevCtx g_ctx[64];
std::mutex g_hook_mu;
void* (*g_alloc)(size_t, void*) = nullptr;
void (*g_release)(void*, void*) = nullptr;
void* g_hook_ctx = nullptr;
thread_local bool t_timing = false;
thread_local bool t_tile_counting = false;
thread_local CallRecord t_record;
}  // namespace

DevCtx* device_ctx(cqsa_status* st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= 64) {
    *st = hip_fail(e == hipSuccess ? hipErrorInvalidDevice : e, "hipGetDevice");
    return nullptr;
  }
  std::lock_guard<std::mutex> g(g_ctx_mu);
  DevCtx* c = &g_ctx[dev];
  if (!c->ready) {
    c->device = dev;
    if ((e = hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking)) != hipSuccess ||
        (e = hipStreamCreateWithFlags(&c->aux, hipStreamNonBlocking)) != hipSuccess ||
        (e = hipStreamCreateWithFlags(&c->lane, hipStreamNonBlocking)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&c->ws_free, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&c->scratch_free, hipEventDisableTiming)) != hipSuccess) {
      *st = hip_fail(e, "creating library streams");
      return nullptr;
    }
    while (c->sync_events.size() < kSetupEvents) {
      hipEvent_t ev;
      if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) {
        *st = hip_fail(e, "creating library events");
        return nullptr;
      }
      c->sync_events.push_back(ev);
    }
    // this device's copy of the scratch array (the device is current here)
    if ((e = hipGetSymbolAddress(&c->scratch, HIP_SYMBOL(scratch))) != hipSuccess ||
        c->scratch == nullptr) {
      c->scratch = nullptr;
      *st = hip_fail(e == hipSuccess ? hipErrorInvalidSymbol : e,
                     "hipGetSymbolAddress of the no-allocation scratch");
      return nullptr;
    }
    c->ready = true;
  }
  *st = CQSA_OK;
  return c;
}

cqsa_status acquire_workspace(DevCtx* c, size_t bytes, Workspace* ws) {
  ws->bytes = bytes;
  ws->from_hook = false;
  ws->ptr = nullptr;
  if (bytes == 0) return CQSA_OK;
  {
    std::lock_guard<std::mutex> g(g_hook_mu);
    if (g_alloc) {
      ws->ptr = g_alloc(bytes, g_hook_ctx);
      ws->from_hook = true;
      if (!ws->ptr) return fail(CQSA_ERR_DEVICE_OOM, "caller allocator returned NULL");
      return CQSA_OK;
    }
  }
  if (c->ws_bytes < bytes) {
    if (c->ws) {
      hipError_t e = hipDeviceSynchronize();
      if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
      (void)hipFree(c->ws);
      c->ws = nullptr;
      c->ws_bytes = 0;
      c->ws_free_valid = false;
    }
    hipError_t e = hipMalloc(&c->ws, bytes);
    if (e != hipSuccess) {
      c->ws = nullptr;
      (void)hipGetLastError();
      return fail(CQSA_ERR_DEVICE_OOM, "hipMalloc of the workspace failed");
    }
    c->ws_bytes = bytes;
  }
  ws->ptr = c->ws;
  return CQSA_OK;
}

void release_workspace(DevCtx* c, Workspace* ws, hipStream_t s) {
  if (!ws->ptr) return;
  if (ws->from_hook) {
    // the caller's allocator is not stream ordered for our side streams
    (void)hipStreamSynchronize(s);
    std::lock_guard<std::mutex> g(g_hook_mu);
    if (g_release) g_release(ws->ptr, g_hook_ctx);
  }
  ws->ptr = nullptr;
  (void)c;
}

cqsa_status acquire_pinned(DevCtx* c, size_t bytes, void** out) {
  if (c->pin_bytes < bytes) {
    if (c->pin) {
      (void)hipDeviceSynchronize();
      (void)hipHostFree(c->pin);
      c->pin = nullptr;
      c->pin_bytes = 0;
    }
    hipError_t e = hipHostMalloc(&c->pin, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      c->pin = nullptr;
      (void)hipGetLastError();
      return fail(CQSA_ERR_INTERNAL, "hipHostMalloc of the host staging buffer failed");
    }
    c->pin_bytes = bytes;
  }
  *out = c->pin;
  return CQSA_OK;
}

cqsa_status upload_image(DevCtx* c, const std::vector<uint8_t>& image, void* dst, hipStream_t s) {
  const size_t n = image.size();
  if (n == 0) return CQSA_OK;
  const int i = c->img_next;
  c->img_next ^= 1;
  if (c->img_valid[i]) CQSA_HIP(hipEventSynchronize(c->img_done[i]));
  if (c->img_bytes[i] < n) {
    if (c->img_pin[i]) (void)hipHostFree(c->img_pin[i]);
    c->img_pin[i] = nullptr;
    c->img_bytes[i] = 0;
    const hipError_t e = hipHostMalloc(&c->img_pin[i], n, hipHostMallocDefault);
    if (e != hipSuccess) {
      c->img_pin[i] = nullptr;
      (void)hipGetLastError();
      return fail(CQSA_ERR_INTERNAL, "hipHostMalloc of the plan image staging failed");
    }
    c->img_bytes[i] = n;
  }
  if (!c->img_done[i]) CQSA_HIP(hipEventCreateWithFlags(&c->img_done[i], hipEventDisableTiming));
  std::memcpy(c->img_pin[i], image.data(), n);
  CQSA_HIP(hipMemcpyAsync(dst, c->img_pin[i], n, hipMemcpyHostToDevice, s));
  CQSA_HIP(hipEventRecord(c->img_done[i], s));
  c->img_valid[i] = true;
  return CQSA_OK;
}

void CallRecord::reset() {
  for (hipEvent_t e : owned) (void)hipEventDestroy(e);
  owned.clear();
  for (auto& v : spans) v.clear();
  wall0 = wall1 = nullptr;
  host_merge_ms = 0.0;
  host_final_ms = 0.0;
  std::memset(&stats, 0, sizeof(stats));
  stats.kernel_tiles_masked = stats.kernel_tiles_clear = stats.kernel_tiles_mixed = -1;
  stats.kernel_kv_tiles_masked = stats.kernel_kv_tiles_clear = stats.kernel_kv_tiles_mixed = -1;
  timing = t_timing;
  counted = 0;
}

hipEvent_t CallRecord::make() {
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  owned.push_back(e);
  return e;
}

CallRecord& call_record() { return t_record; }
bool timing_enabled() { return t_timing; }
bool tile_counting_enabled() { return t_tile_counting; }

cqsa_status tile_counters_begin(DevCtx* c, hipStream_t s, int n, unsigned long long** out) {
  if (!c->tile_count) {
    void* p = nullptr;
    CQSA_HIP(hipMalloc(&p, 64));
    c->tile_count = (unsigned long long*)p;
  }
  CQSA_HIP(launch_zero_u64(c->tile_count, n, s));
  *out = c->tile_count;
  return CQSA_OK;
}

cqsa_status tile_counters_end(DevCtx* c, CallRecord& rec, hipStream_t s, int n) {
  if (!rec.tile_host) {
    void* p = nullptr;
    CQSA_HIP(hipHostMalloc(&p, 64, hipHostMallocDefault));
    rec.tile_host = (unsigned long long*)p;
  }
  if (!rec.tile_done) CQSA_HIP(hipEventCreateWithFlags(&rec.tile_done, hipEventDisableTiming));
  CQSA_HIP(hipMemcpyAsync(rec.tile_host, c->tile_count, size_t(n) * sizeof(unsigned long long),
                          hipMemcpyDeviceToHost, s));
  CQSA_HIP(hipEventRecord(rec.tile_done, s));
  rec.counted = n;
  return CQSA_OK;
}

cqsa_status check_tensor(const cqsa_tensor* t, const char* name, const cqsa_plan_t* p,
                         cqsa_dtype want, cqsa_mem where) {
  std::string n(name);
  if (!t) return fail(CQSA_ERR_INVALID_ARG, n + " is NULL");
  if (!t->data) return fail(CQSA_ERR_INVALID_ARG, n + ".data is NULL");
  if (reinterpret_cast<uintptr_t>(t->data) % 16 != 0)
    return fail(CQSA_ERR_INVALID_ARG, n + ".data must be 16-byte aligned");
  if (t->dtype != want) return fail(CQSA_ERR_INVALID_ARG, n + " has the wrong dtype");
  if (t->where != where)
    return fail(CQSA_ERR_INVALID_ARG, n + " residency differs from the plan");
  if (t->B != p->opts.B || t->L != p->g.L || t->H != p->g.H || t->d != p->g.d)
    return fail(CQSA_ERR_INVALID_ARG, n + " shape differs from the plan");
  return CQSA_OK;
}

std::vector<StagePiece> stage_pieces(const Task& cur, const Task* prev) {
  std::vector<StagePiece> out;
  size_t pi = 0;
  for (const Run& r : cur.runs) {
    int64_t g = r.global_start;
    const int64_t end = r.global_start + r.length;
    while (g < end) {
      // first run of prev that ends after g
      while (prev && pi < prev->runs.size() &&
             prev->runs[pi].global_start + prev->runs[pi].length <= g)
        ++pi;
      const Run* pr = (prev && pi < prev->runs.size()) ? &prev->runs[pi] : nullptr;
      const int64_t dst = r.local_start + (g - r.global_start);
      if (pr && pr->global_start <= g) {
        const int64_t e = std::min(end, pr->global_start + pr->length);
        out.push_back({dst, pr->local_start + (g - pr->global_start), e - g, true});
        g = e;
      } else {
        const int64_t e = pr ? std::min(end, pr->global_start) : end;
        out.push_back({dst, g, e - g, false});
        g = e;
      }
    }
  }
  return out;
}


}  // namespace cqsa

using namespace cqsa;

extern "C" {

cqsa_status cqsa_set_allocator(void* (*alloc)(size_t, void*), void (*release)(void*, void*),
                               void* ctx) {
  clear_error();
  if ((alloc == nullptr) != (release == nullptr))
    return fail(CQSA_ERR_INVALID_ARG, "cqsa_set_allocator: give both functions or neither");
  std::lock_guard<std::mutex> g(g_hook_mu);
  g_alloc = alloc;
  g_release = release;
  g_hook_ctx = ctx;
  return CQSA_OK;
}

cqsa_status cqsa_set_timing(int32_t enable) {
  clear_error();
  t_timing = enable != 0;
  return CQSA_OK;
}

cqsa_status cqsa_set_tile_counting(int32_t enable) {
  clear_error();
  t_tile_counting = enable != 0;
  return CQSA_OK;
}

cqsa_status cqsa_last_stats(cqsa_run_stats* out) {
  clear_error();
  if (!out) return fail(CQSA_ERR_INVALID_ARG, "cqsa_last_stats: out is NULL");
  CallRecord& r = t_record;
  cqsa_run_stats s = r.stats;
  if (r.timing && r.wall1) {
    hipError_t e = hipEventSynchronize(r.wall1);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    auto span = [](hipEvent_t a, hipEvent_t b) {
      float ms = 0.f;
      if (hipEventSynchronize(b) != hipSuccess) return 0.0;
      if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return 0.0;
      return double(ms);
    };
    s.ms_wall = span(r.wall0, r.wall1);
    double* dst[kStCount] = {&s.ms_stage, &s.ms_inner, &s.ms_merge, &s.ms_finalize, &s.ms_d2h};
    for (int k = 0; k < kStCount; ++k) {
      double acc = 0.0;
      for (auto& pr : r.spans[k]) acc += span(pr.first, pr.second);
      *dst[k] = acc;
    }
    s.ms_merge += r.host_merge_ms;
    s.ms_finalize += r.host_final_ms;
    // union of the inner-kernel spans on the device clock
    std::vector<std::pair<double, double>> iv;
    for (auto& pr : r.spans[kStInner]) {
      const double a = span(r.wall0, pr.first), b = span(r.wall0, pr.second);
      iv.push_back({a, b});
    }
    std::sort(iv.begin(), iv.end());
    double busy = 0.0, cs = 0.0, ce = -1.0;
    for (auto& x : iv) {
      if (x.first > ce) {
        if (ce > cs) busy += ce - cs;
        cs = x.first;
        ce = x.second;
      } else if (x.second > ce) {
        ce = x.second;
      }
    }
    if (ce > cs) busy += ce - cs;
    s.ms_inner_busy = busy;
  }
  if (r.counted) {
    hipError_t e = hipEventSynchronize(r.tile_done);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    s.kernel_tiles_masked = int64_t(r.tile_host[0]);
    s.kernel_tiles_clear = int64_t(r.tile_host[1]);
    s.kernel_tiles_mixed = int64_t(r.tile_host[2]);
    if (r.counted >= 6) {
      s.kernel_kv_tiles_masked = int64_t(r.tile_host[3]);
      s.kernel_kv_tiles_clear = int64_t(r.tile_host[4]);
      s.kernel_kv_tiles_mixed = int64_t(r.tile_host[5]);
    }
  }
  *out = s;
  return CQSA_OK;
}

cqsa_status cqsa_release_workspace(void) {
  clear_error();
  cqsa_status st;
  DevCtx* c = device_ctx(&st);
  if (!c) return st;
  std::lock_guard<std::mutex> g(c->mu);
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  if (c->ws) (void)hipFree(c->ws);
  c->ws = nullptr;
  c->ws_bytes = 0;
  c->ws_free_valid = false;
  if (c->pin) (void)hipHostFree(c->pin);
  c->pin = nullptr;
  c->pin_bytes = 0;
  for (int i = 0; i < 2; ++i) {
    if (c->img_pin[i]) (void)hipHostFree(c->img_pin[i]);
    c->img_pin[i] = nullptr;
    c->img_bytes[i] = 0;
    c->img_valid[i] = false;
  }
  return CQSA_OK;
}

}  // extern "C"
