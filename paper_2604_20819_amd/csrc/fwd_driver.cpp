// cqsa_forward: the task streamer of the decomposed forward.
//
// Per task (Alg. 1, computed with the max-shifted merge of App. A.1):
//   copy stream   : gather the task's runs of Q, K, V into staging slot t % S
//                   (H2D from host inputs or D2D), then signal "staged";
//   caller stream : wait "staged", run the inner forward kernel (local
//                   statistics), then either recompose into the device
//                   accumulator (acc on device) or hand the statistics to the
//                   D2H stream and a host merge thread (acc on host);
//   the slot is freed by an event once its last reader is done.
// With S >= 2 slots the gather of task t+1 overlaps the compute of task t
// (App. A.3: transfers overlap compute, at most two tasks in flight).
// Depth 0 on device-resident tensors is the undecomposed call: one kernel that
// writes O and LSE directly.
#include <algorithm>
#include <cmath>
#include <condition_variable>
#include <deque>
#include <functional>
#include <thread>

#include "kernels.hpp"
#include "runtime.hpp"

namespace cqsa {

namespace {

int host_threads() {
  unsigned n = std::thread::hardware_concurrency();
  if (n == 0) n = 4;
  return int(std::min(16u, n));
}

template <typename F>
void parallel_rows(int64_t n, F f) {
  const int nt = int(std::min<int64_t>(host_threads(), std::max<int64_t>(1, n / 256)));
  if (nt <= 1) {
    f(int64_t(0), n);
    return;
  }
  std::vector<std::thread> th;
  for (int i = 0; i < nt; ++i) {
    const int64_t a = n * i / nt, b = n * (i + 1) / nt;
    th.emplace_back([=] { f(a, b); });
  }
  for (auto& t : th) t.join();
}

// Max-shifted merge of one task's statistics into the host accumulator
// (Eq. "merge", log2 domain, null rows skipped).
void host_merge(const Task& task, const float* acc_i, const float* m_i, const float* l_i,
                float* acc, float* m, float* l, int64_t B, int64_t L, int64_t H, int64_t d) {
  const int64_t Li = task.L_local;
  parallel_rows(B * Li, [&](int64_t lo, int64_t hi) {
    size_t ri = 0;
    for (int64_t x = lo; x < hi; ++x) {
      const int64_t b = x / Li, r = x % Li;
      while (ri + 1 < task.runs.size() && r >= task.runs[ri].local_start + task.runs[ri].length)
        ++ri;
      while (ri > 0 && r < task.runs[ri].local_start) --ri;
      const Run& run = task.runs[ri];
      const int64_t g = run.global_start + (r - run.local_start);
      for (int64_t h = 0; h < H; ++h) {
        const int64_t si = (b * H + h) * Li + r, gi = (b * H + h) * L + g;
        const float mi = m_i[si];
        if (mi == -INFINITY) continue;
        const float mo = m[gi];
        const float mn = std::max(mo, mi);
        const float fo = mo == -INFINITY ? 0.f : std::exp2(mo - mn);
        const float fi = std::exp2(mi - mn);
        const float* src = acc_i + ((b * Li + r) * H + h) * d;
        float* dst = acc + ((b * L + g) * H + h) * d;
        for (int64_t k = 0; k < d; ++k) dst[k] = dst[k] * fo + src[k] * fi;
        l[gi] = l[gi] * fo + l_i[si] * fi;
        m[gi] = mn;
      }
    }
  });
}

void host_finalize(float* acc, float* m, const float* l, int64_t B, int64_t L, int64_t H,
                   int64_t d) {
  parallel_rows(B * L, [&](int64_t lo, int64_t hi) {
    for (int64_t x = lo; x < hi; ++x) {
      const int64_t b = x / L, g = x % L;
      for (int64_t h = 0; h < H; ++h) {
        const int64_t gi = (b * H + h) * L + g;
        const float inv = 1.f / l[gi];
        float* row = acc + ((b * L + g) * H + h) * d;
        for (int64_t k = 0; k < d; ++k) row[k] *= inv;
        m[gi] = (m[gi] + std::log2(l[gi])) * 0.69314718055994530942f;
      }
    }
  });
}

// One consumer thread that runs host merges strictly in submission order
// (merges of different tasks touch shared rows).
class HostMerger {
 public:
  ~HostMerger() { finish(); }
  // Queues a job; returns its sequence number.
  int64_t push(std::function<bool()> job) {
    std::unique_lock<std::mutex> g(mu_);
    if (!th_.joinable()) th_ = std::thread([this] { run(); });
    q_.push_back(std::move(job));
    cv_.notify_all();
    return pushed_++;
  }
  // Blocks until job `id` (and all before it) finished; false on failure.
  bool wait_done(int64_t id) {
    std::unique_lock<std::mutex> g(mu_);
    cv_.wait(g, [&] { return done_ > id || !ok_; });
    return ok_;
  }
  bool finish() {
    {
      std::unique_lock<std::mutex> g(mu_);
      stop_ = true;
      cv_.notify_all();
    }
    if (th_.joinable()) th_.join();
    return ok_;
  }

 private:
  void run() {
    for (;;) {
      std::function<bool()> job;
      {
        std::unique_lock<std::mutex> g(mu_);
        cv_.wait(g, [&] { return !q_.empty() || stop_; });
        if (q_.empty()) return;
        job = std::move(q_.front());
        q_.pop_front();
      }
      const bool ok = ok_ && job();
      std::unique_lock<std::mutex> g(mu_);
      if (!ok) ok_ = false;
      ++done_;
      cv_.notify_all();
    }
  }
  std::mutex mu_;
  std::condition_variable cv_;
  std::deque<std::function<bool()>> q_;
  std::thread th_;
  int64_t pushed_ = 0, done_ = 0;
  bool stop_ = false, ok_ = true;
};

}  // namespace

cqsa_status forward_impl(const cqsa_plan_t* p, const cqsa_tensor* Q, const cqsa_tensor* K,
                         const cqsa_tensor* V, cqsa_tensor* O, float* LSE, cqsa_mem lse_where,
                         float scale, hipStream_t st) {
  if (!p) return fail(CQSA_ERR_INVALID_ARG, "cqsa_forward: plan is NULL");
  const cqsa_plan_opts& o = p->opts;
  const cqsa_mem in_where = o.inputs_on_device ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  const cqsa_mem acc_where = o.acc_on_device ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  cqsa_status s;
  if ((s = check_tensor(Q, "Q", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(K, "K", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(V, "V", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(O, "O", p, CQSA_F32, acc_where)) != CQSA_OK) return s;
  if (!LSE) return fail(CQSA_ERR_INVALID_ARG, "LSE is NULL");
  if (lse_where != acc_where)
    return fail(CQSA_ERR_INVALID_ARG, "LSE residency must equal the output residency");

  DevCtx* C = device_ctx(&s);
  if (!C) return s;
  std::lock_guard<std::mutex> lock(C->mu);

  const int64_t B = o.B, L = p->g.L, H = p->g.H, d = p->g.d;
  const size_t elem = dtype_size(o.dtype);
  const size_t row_bytes = size_t(H) * d * elem;
  const float sc = scale > 0.f ? scale : float(1.0 / std::sqrt(double(d)));
  const float scale_log2 = sc * 1.4426950408889634f;
  const bool in_dev = o.inputs_on_device, acc_dev = o.acc_on_device;
  const int depth = p->depth;
  const int64_t ntask = int64_t(p->tasks.size());
  const bool direct = depth == 0 && in_dev && acc_dev;

  CallRecord& rec = call_record();
  rec.reset();
  rec.stats.depth = depth;
  rec.stats.num_tasks = ntask;
  rec.stats.modelled_device_bytes = p->fp.peak;
  if (rec.timing) {
    rec.wall0 = rec.make();
    rec.wall1 = rec.make();
    CQSA_HIP(hipEventRecord(rec.wall0, st));
  }

  // ---- workspace layout ----
  const uint64_t tab_bytes = align_up(p->packed.size());
  const uint64_t gl_bytes = (acc_dev && !direct) ? align_up(uint64_t(B) * H * L * 4) : 0;
  const uint64_t slot_bytes = direct ? 0 : fwd_slot_bytes(p->g, o, p->max_L_local, true, true);
  const int64_t nslot = std::min<int64_t>(o.n_slots, std::max<int64_t>(1, ntask));
  const uint64_t total = tab_bytes + gl_bytes + uint64_t(nslot) * slot_bytes;
  Workspace ws;
  if ((s = acquire_workspace(C, total, &ws)) != CQSA_OK) return s;
  rec.stats.workspace_bytes = total;
  char* base = (char*)ws.ptr;
  char* d_tab = base;
  float* d_gl = (float*)(base + tab_bytes);
  struct Slot {
    char *q, *k, *v;
    float *acc, *m, *l;
  };
  std::vector<Slot> slots(nslot);
  {
    const uint64_t rows = uint64_t(B) * p->max_L_local * H;
    const uint64_t in_b = align_up(rows * d * elem), acc_b = align_up(rows * d * 4),
                   st_b = align_up(rows * 4);
    for (int64_t i = 0; i < nslot; ++i) {
      char* sb = base + tab_bytes + gl_bytes + uint64_t(i) * slot_bytes;
      slots[i].q = sb;
      slots[i].k = sb + in_b;
      slots[i].v = sb + 2 * in_b;
      slots[i].acc = (float*)(sb + 3 * in_b);
      slots[i].m = (float*)(sb + 3 * in_b + acc_b);
      slots[i].l = (float*)(sb + 3 * in_b + acc_b + st_b);
    }
  }

  // ---- ordering against the caller's stream and the previous call ----
  while (C->sync_events.size() < size_t(4 * nslot + 3)) {
    hipEvent_t e;
    CQSA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    C->sync_events.push_back(e);
  }
  hipEvent_t ev_start = C->sync_events[0];
  hipEvent_t* ev_staged = &C->sync_events[2];
  hipEvent_t* ev_free = &C->sync_events[2 + nslot];
  hipEvent_t* ev_done = &C->sync_events[2 + 2 * nslot];
  hipEvent_t ev_rec = C->sync_events[2 + 4 * nslot];  // last recompose issued
  if (C->ws_free_valid) CQSA_HIP(hipStreamWaitEvent(st, C->ws_free, 0));
  CQSA_HIP(hipEventRecord(ev_start, st));
  CQSA_HIP(hipStreamWaitEvent(C->copy, ev_start, 0));
  CQSA_HIP(hipMemcpyAsync(d_tab, p->packed.data(), p->packed.size(), hipMemcpyHostToDevice,
                          C->copy));

  float* Od = (float*)O->data;
  if (direct) {
    CQSA_HIP(hipEventRecord(ev_staged[0], C->copy));
    CQSA_HIP(hipStreamWaitEvent(st, ev_staged[0], 0));
    const Task& t = p->tasks[0];
    const TableOffsets& to = p->table_off[0];
    FwdArgs a{};
    a.q = Q->data; a.k = K->data; a.v = V->data;
    a.seq_rows = L; a.row0 = 0; a.L = int32_t(t.L_local); a.B = int32_t(B); a.H = int32_t(H);
    a.causal = p->g.causal; a.scale_log2 = scale_log2;
    a.runs = d_tab + to.runs; a.n_runs = int32_t(t.runs.size());
    a.blk_or = (const uint32_t*)(d_tab + to.blk_or);
    a.blk_and = (const uint32_t*)(d_tab + to.blk_and);
    a.acc = Od; a.m = LSE; a.l = nullptr; a.out_rows = L;
    std::pair<hipEvent_t, hipEvent_t> sp{nullptr, nullptr};
    if (rec.timing) {
      sp = {rec.make(), rec.make()};
      CQSA_HIP(hipEventRecord(sp.first, st));
    }
    CQSA_HIP(launch_fwd(o.dtype, int(d), kModeFinal, a, st));
    if (rec.timing) {
      CQSA_HIP(hipEventRecord(sp.second, st));
      rec.spans[kStInner].push_back(sp);
    }
    rec.stats.inner_launches = 1;
  } else {
    // accumulator: the O buffer holds acc, the LSE buffer holds m (log2)
    float* acc = Od;
    float* m = LSE;
    float* l = d_gl;
    std::vector<float> l_host;
    char* pin = nullptr;
    uint64_t pin_slot = 0;
    if (acc_dev) {
      CQSA_HIP(launch_acc_init(acc, m, l, B * L * H * d, B * H * L, st));
    } else {
      l_host.assign(size_t(B * H * L), 0.f);
      l = l_host.data();
      parallel_rows(B * L, [&](int64_t lo, int64_t hi) {
        std::fill(acc + lo * H * d, acc + hi * H * d, 0.f);
      });
      std::fill(m, m + B * H * L, -INFINITY);
      const uint64_t rows = uint64_t(B) * p->max_L_local * H;
      pin_slot = align_up(rows * d * 4) + 2 * align_up(rows * 4);
      void* pv = nullptr;
      if ((s = acquire_pinned(C, size_t(pin_slot * nslot), &pv)) != CQSA_OK) return s;
      pin = (char*)pv;
    }
    HostMerger merger;
    std::vector<int64_t> last_item(nslot, -1);
    bool rec_issued = false;
    std::vector<bool> used(nslot, false);
    const hipMemcpyKind kind = in_dev ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    for (int64_t t = 0; t < ntask; ++t) {
      const Task& task = p->tasks[t];
      const int64_t Li = task.L_local;
      if (Li == 0) continue;
      const int64_t si = t % nslot;
      Slot& S = slots[si];
      const TableOffsets& to = p->table_off[t];
      if (used[si]) CQSA_HIP(hipStreamWaitEvent(C->copy, ev_free[si], 0));
      // gather
      std::pair<hipEvent_t, hipEvent_t> sp{nullptr, nullptr};
      if (rec.timing) {
        sp = {rec.make(), rec.make()};
        CQSA_HIP(hipEventRecord(sp.first, C->copy));
      }
      const char* srcs[3] = {(const char*)Q->data, (const char*)K->data, (const char*)V->data};
      char* dsts[3] = {S.q, S.k, S.v};
      if (in_dev) {
        // device inputs: one gather kernel over the runs of all three tensors
        StageArgs sa{};
        for (int x = 0; x < 3; ++x) {
          sa.src[x] = srcs[x];
          sa.dst[x] = dsts[x];
        }
        sa.n_tensors = 3; sa.row_bytes = int64_t(row_bytes); sa.Li = Li; sa.Lg = L;
        sa.B = int32_t(B); sa.runs = d_tab + to.runs; sa.n_runs = int32_t(task.runs.size());
        CQSA_HIP(launch_stage(sa, C->copy));
      } else {
        // host inputs: one asynchronous H2D copy per run and batch element
        for (int x = 0; x < 3; ++x)
          for (const Run& r : task.runs)
            for (int64_t b = 0; b < B; ++b)
              CQSA_HIP(hipMemcpyAsync(dsts[x] + (b * Li + r.local_start) * row_bytes,
                                      srcs[x] + (b * L + r.global_start) * row_bytes,
                                      r.length * row_bytes, kind, C->copy));
      }
      const uint64_t moved = uint64_t(3) * B * Li * row_bytes;
      if (in_dev)
        rec.stats.d2d_bytes += moved;
      else
        rec.stats.h2d_bytes += moved;
      if (rec.timing) {
        CQSA_HIP(hipEventRecord(sp.second, C->copy));
        rec.spans[kStStage].push_back(sp);
      }
      CQSA_HIP(hipEventRecord(ev_staged[si], C->copy));
      // Consecutive tasks alternate between the caller's stream and a second
      // compute stream, so a task's kernel fills the tail of the previous one
      // (two tasks in flight, App. A.3).  Inner kernels write only their slot.
      const hipStream_t ls = (t & 1) ? C->lane : st;
      CQSA_HIP(hipStreamWaitEvent(ls, ev_staged[si], 0));
      // inner kernel
      FwdArgs a{};
      a.q = S.q; a.k = S.k; a.v = S.v;
      a.seq_rows = Li; a.row0 = 0; a.L = int32_t(Li); a.B = int32_t(B); a.H = int32_t(H);
      a.causal = p->g.causal; a.scale_log2 = scale_log2;
      a.runs = d_tab + to.runs; a.n_runs = int32_t(task.runs.size());
      a.blk_or = (const uint32_t*)(d_tab + to.blk_or);
      a.blk_and = (const uint32_t*)(d_tab + to.blk_and);
      a.acc = S.acc; a.m = S.m; a.l = S.l; a.out_rows = Li;
      if (rec.timing) {
        sp = {rec.make(), rec.make()};
        CQSA_HIP(hipEventRecord(sp.first, ls));
      }
      CQSA_HIP(launch_fwd(o.dtype, int(d), kModeStats, a, ls));
      rec.stats.inner_launches += 1;
      if (rec.timing) {
        CQSA_HIP(hipEventRecord(sp.second, ls));
        rec.spans[kStInner].push_back(sp);
      }
      if (acc_dev) {
        // recomposes touch shared rows: each waits for the one before it
        if (rec_issued) CQSA_HIP(hipStreamWaitEvent(ls, ev_rec, 0));
        MergeArgs mg{};
        mg.acc_i = S.acc; mg.m_i = S.m; mg.l_i = S.l;
        mg.acc = acc; mg.m = m; mg.l = l;
        mg.runs = d_tab + to.runs; mg.n_runs = int32_t(task.runs.size());
        mg.Li = Li; mg.L = L; mg.B = int32_t(B); mg.H = int32_t(H); mg.d = int32_t(d);
        if (rec.timing) {
          sp = {rec.make(), rec.make()};
          CQSA_HIP(hipEventRecord(sp.first, ls));
        }
        CQSA_HIP(launch_recompose(mg, ls));
        if (rec.timing) {
          CQSA_HIP(hipEventRecord(sp.second, ls));
          rec.spans[kStMerge].push_back(sp);
        }
        CQSA_HIP(hipEventRecord(ev_rec, ls));
        rec_issued = true;
        CQSA_HIP(hipEventRecord(ev_free[si], ls));
      } else {
        // hand the statistics to the host: D2H into pinned staging, then merge;
        // the staging of this slot must have been consumed by its last merge
        if (!merger.wait_done(last_item[si])) return fail(CQSA_ERR_HIP, "host merge failed");
        char* hp = pin + uint64_t(si) * pin_slot;
        const uint64_t rows = uint64_t(B) * Li * H;
        float* h_acc = (float*)hp;
        float* h_m = (float*)(hp + align_up(uint64_t(B) * p->max_L_local * H * d * 4));
        float* h_l = (float*)((char*)h_m + align_up(uint64_t(B) * p->max_L_local * H * 4));
        CQSA_HIP(hipEventRecord(ev_done[si], ls));
        CQSA_HIP(hipStreamWaitEvent(C->d2h, ev_done[si], 0));
        if (rec.timing) {
          sp = {rec.make(), rec.make()};
          CQSA_HIP(hipEventRecord(sp.first, C->d2h));
        }
        CQSA_HIP(hipMemcpyAsync(h_acc, S.acc, rows * d * 4, hipMemcpyDeviceToHost, C->d2h));
        CQSA_HIP(hipMemcpyAsync(h_m, S.m, rows * 4, hipMemcpyDeviceToHost, C->d2h));
        CQSA_HIP(hipMemcpyAsync(h_l, S.l, rows * 4, hipMemcpyDeviceToHost, C->d2h));
        rec.stats.d2h_bytes += rows * (d + 2) * 4;
        if (rec.timing) {
          CQSA_HIP(hipEventRecord(sp.second, C->d2h));
          rec.spans[kStD2H].push_back(sp);
        }
        CQSA_HIP(hipEventRecord(ev_free[si], C->d2h));
        const hipEvent_t wait_ev = ev_free[si];
        const Task* tp = &p->tasks[t];
        last_item[si] = merger.push([=, &rec]() -> bool {
          auto t0 = std::chrono::steady_clock::now();
          if (hipEventSynchronize(wait_ev) != hipSuccess) return false;
          host_merge(*tp, h_acc, h_m, h_l, acc, m, l, B, L, H, d);
          auto t1 = std::chrono::steady_clock::now();
          rec.host_merge_ms += std::chrono::duration<double, std::milli>(t1 - t0).count();
          return true;
        });
      }
      used[si] = true;
    }
    if (acc_dev) {
      if (rec_issued) CQSA_HIP(hipStreamWaitEvent(st, ev_rec, 0));
      std::pair<hipEvent_t, hipEvent_t> sp{nullptr, nullptr};
      if (rec.timing) {
        sp = {rec.make(), rec.make()};
        CQSA_HIP(hipEventRecord(sp.first, st));
      }
      CQSA_HIP(launch_finalize(acc, m, l, B, L, H, int(d), st));
      if (rec.timing) {
        CQSA_HIP(hipEventRecord(sp.second, st));
        rec.spans[kStFinal].push_back(sp);
      }
    } else {
      if (!merger.finish()) return fail(CQSA_ERR_HIP, "host merge: event wait failed");
      host_finalize(acc, m, l, B, L, H, d);
      // the second compute stream's last kernel precedes its D2H, which the
      // merges waited for; order the caller's stream after it all the same
      CQSA_HIP(hipEventRecord(ev_done[0], C->d2h));
      CQSA_HIP(hipStreamWaitEvent(st, ev_done[0], 0));
    }
  }
  if (rec.timing) CQSA_HIP(hipEventRecord(rec.wall1, st));
  CQSA_HIP(hipEventRecord(C->ws_free, st));
  C->ws_free_valid = true;
  release_workspace(C, &ws, st);
  if (!acc_dev) {
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  }
  return CQSA_OK;
}

}  // namespace cqsa

extern "C" cqsa_status cqsa_forward(const cqsa_plan_t* plan, const cqsa_tensor* Q,
                                    const cqsa_tensor* K, const cqsa_tensor* V, cqsa_tensor* O,
                                    float* LSE, cqsa_mem lse_where, float scale,
                                    void* hip_stream) {
  cqsa::clear_error();
  try {
    return cqsa::forward_impl(plan, Q, K, V, O, LSE, lse_where, scale, (hipStream_t)hip_stream);
  } catch (const std::exception& e) {
    return cqsa::fail(CQSA_ERR_INTERNAL, std::string("cqsa_forward: ") + e.what());
  } catch (...) {
    return cqsa::fail(CQSA_ERR_INTERNAL, "cqsa_forward: unknown exception");
  }
}
