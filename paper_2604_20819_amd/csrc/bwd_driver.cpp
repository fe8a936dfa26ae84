// cqsa_backward: decomposed backward in the global-LSE form (App. A.1,
// Eq. "globallse"), equal to Alg. 2.
//
// Q, K, V, dO sit where the plan's inputs do; O, LSE, dQ, dK, dV where its
// accumulator does (the forward's outputs), each on the host or the device.
//
// caller stream : D = rowsum(dO * O) over the full sequence (host-resident O
//                 or dO arrive in chunks through the staging slots); zero
//                 dQ/dK/dV when they are device-resident; per task wait
//                 "staged", run the key-parallel dK/dV kernel, then the
//                 query-parallel dQ kernel when the dK/dV launches span many
//                 rounds of resident waves;
// second stream : otherwise the dQ kernels, beside the dK/dV kernels;
// copy stream   : gather each task's runs of Q, K, V, dO into slot t % S once
//                 both kernels of the slot's previous task are done: a gather
//                 kernel from device-resident inputs, host-to-device copies
//                 from host-resident ones (tokens the previously staged task
//                 also holds come from its staged rows on the device); a plan
//                 that reads device-resident inputs in place stages nothing;
// device gradients, several tasks per launch (inputs read in place): per
//                 launch group one dK/dV launch and one dQ launch over all its
//                 tasks store every task's rows in its own buffer, and a
//                 gather-merge on the caller's stream adds them into dQ, dK,
//                 dV in task order;
// device gradients, one task per launch: each kernel's epilogue adds the
//                 task's rows into the global fp32 gradients.  All dQ launches
//                 of a call run on one stream, which keeps the tasks in order,
//                 and a task holds each token once, so these
//                 read-modify-writes never race (undecomposed, the single
//                 task's rows are stored);
// host gradients: the kernels store the task's rows in the slot's own
//                 gradient buffers; the auxiliary stream copies them to pinned
//                 host memory and a host thread adds them into dQ, dK, dV at
//                 their global rows, task after task (App. A.3, accumulator on
//                 the host).
// Depth 0 on device-resident inputs reads the caller's tensors in place (the
// undecomposed backward).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>

#include "guard.hpp"
#include "kernels.hpp"
#include "runtime.hpp"
#include "streamer.hpp"

namespace cqsa {

namespace {

// dst[global rows of the task] += src[task rows] for the three gradients
// (fp32 [B, L, H, d] and [B, Li, H, d]); rows split across host threads.
void host_scatter_add(const Task& task, const float* const src[3], float* const dst[3], int64_t B,
                      int64_t L, int64_t H, int64_t d) {
  const int64_t Li = task.L_local, rw = H * d;
  parallel_rows(B * Li, [&](int64_t lo, int64_t hi) {
    size_t ri = 0;
    for (int64_t x = lo; x < hi;) {
      const int64_t b = x / Li, r = x % Li;
      while (ri + 1 < task.runs.size() && r >= task.runs[ri].local_start + task.runs[ri].length)
        ++ri;
      while (ri > 0 && r < task.runs[ri].local_start) --ri;
      const Run& run = task.runs[ri];
      // rows [r, r + n) of this batch element lie in one run: one span each
      const int64_t n = std::min({hi - x, Li - r, run.local_start + run.length - r});
      const int64_t g = run.global_start + (r - run.local_start);
      for (int t = 0; t < 3; ++t) {
        const float* s = src[t] + (b * Li + r) * rw;
        float* o = dst[t] + (b * L + g) * rw;
        for (int64_t k = 0; k < n * rw; ++k) o[k] += s[k];
      }
      x += n;
    }
  });
}

void host_zero(float* const p[3], int64_t n) {
  for (int t = 0; t < 3; ++t)
    parallel_rows(n / 4096 + 1, [&](int64_t lo, int64_t hi) {
      const int64_t a = lo * 4096, b = std::min(n, hi * 4096);
      if (b > a) std::memset(p[t] + a, 0, size_t(b - a) * sizeof(float));
    });
}

}  // namespace

cqsa_status backward_impl(const cqsa_plan_t* p, const cqsa_tensor* Q, const cqsa_tensor* K,
                          const cqsa_tensor* V, const cqsa_tensor* O, const float* LSE,
                          cqsa_mem lse_where, const cqsa_tensor* dO, cqsa_tensor* dQ,
                          cqsa_tensor* dK, cqsa_tensor* dV, float scale, hipStream_t st) {
  if (!p) return fail(CQSA_ERR_INVALID_ARG, "cqsa_backward: plan is NULL");
  const cqsa_plan_opts& o = p->opts;
  if (o.dtype == CQSA_F32)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: fp16 and bf16 inputs only");
  if (p->g.d % 32 != 0 || p->g.d > 256)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: head dims 32, 64, ..., 256 only");
  if (!o.with_backward && p->budget != 0)
    return fail(CQSA_ERR_INVALID_ARG,
                "cqsa_backward: the plan's budget was fitted without the backward "
                "(plan with with_backward = 1)");
  const bool dev_in = o.inputs_on_device != 0, dev_acc = o.acc_on_device == 1;
  const cqsa_mem in_where = dev_in ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  const cqsa_mem acc_where = dev_acc ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  cqsa_status s;
  if ((s = check_tensor(Q, "Q", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(K, "K", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(V, "V", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(dO, "dO", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(O, "O", p, CQSA_F32, acc_where)) != CQSA_OK) return s;
  if ((s = check_tensor(dQ, "dQ", p, CQSA_F32, acc_where)) != CQSA_OK) return s;
  if ((s = check_tensor(dK, "dK", p, CQSA_F32, acc_where)) != CQSA_OK) return s;
  if ((s = check_tensor(dV, "dV", p, CQSA_F32, acc_where)) != CQSA_OK) return s;
  if (!LSE) return fail(CQSA_ERR_INVALID_ARG, "LSE is NULL");
  if (lse_where != acc_where)
    return fail(CQSA_ERR_INVALID_ARG, "LSE residency must equal the output residency");

  DevCtx* C = device_ctx(&s);
  if (!C) return s;
  std::lock_guard<std::mutex> lock(C->mu);

  const int64_t B = o.B, L = p->g.L, H = p->g.H, d = p->g.d;
  const size_t elem = dtype_size(o.dtype);
  const int64_t row_bytes = int64_t(H) * d * int64_t(elem);
  const float sc = scale > 0.f ? scale : float(1.0 / std::sqrt(double(d)));
  const int depth = p->depth;
  const int64_t ntask = int64_t(p->tasks.size());
  const bool staged = bwd_staged(o, depth);
  // device-resident inputs not staged: read in place (decomposed) or the
  // caller's tensors themselves (undecomposed)
  const bool in_place = !staged && depth > 0;

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

  // ---- workspace: [plan image][D][LSE copy, host LSE only][slot 0]...[slot S-1];
  // a slot holds the staged Q, K, V, dO (staged plans) and then the task's
  // own dQ, dK, dV (host gradients), each sized for the longest task
  const uint64_t tab_bytes = align_up(p->packed.size());
  const uint64_t stat_bytes = align_up(uint64_t(B) * H * L * 4);
  const uint64_t lse_bytes = dev_acc ? 0 : stat_bytes;
  const uint64_t slot_bytes = bwd_slot_bytes(p->g, o, p->max_L_local, staged);
  const int64_t nslot = std::min<int64_t>(o.n_slots, std::max<int64_t>(1, ntask));
  // several tasks per launch: their local dQ, dK, dV after the slots
  const bool batched = !p->bwd_groups.empty();
  const bool direct = depth == 0 && !staged && dev_acc;  // the single task stores its rows
  const int64_t gmax = batched ? p->fp.bwd_group_size : 0;
  const uint64_t loc_b = align_up(uint64_t(B) * p->max_L_local * H * d * 4);
  const uint64_t total = tab_bytes + stat_bytes + lse_bytes + uint64_t(nslot) * slot_bytes +
                         3 * uint64_t(gmax) * loc_b;
  Workspace ws;
  if ((s = acquire_workspace(C, total, &ws)) != CQSA_OK) return s;
  rec.stats.workspace_bytes = total;
  rec.stats.resident_tasks = batched ? gmax : (staged || !dev_acc) ? nslot : 0;
  char* base = (char*)ws.ptr;
  char* d_tab = base;
  float* d_D = (float*)(base + tab_bytes);
  const float* d_lse = dev_acc ? LSE : (const float*)(base + tab_bytes + stat_bytes);
  const uint64_t in_b = staged ? align_up(uint64_t(B) * p->max_L_local * H * d * elem) : 0;
  const uint64_t g_b = align_up(uint64_t(B) * p->max_L_local * H * d * 4);
  auto slot_base = [&](int64_t si) {
    return base + tab_bytes + stat_bytes + lse_bytes + uint64_t(si) * slot_bytes;
  };

  while (C->sync_events.size() < size_t(5 * nslot + 4)) {
    hipEvent_t e;
    CQSA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    C->sync_events.push_back(e);
  }
  hipEvent_t ev_start = C->sync_events[0];
  hipEvent_t ev_tab = C->sync_events[1];
  hipEvent_t ev_pre = C->sync_events[2];
  hipEvent_t ev_join = C->sync_events[3];
  hipEvent_t* ev_staged = &C->sync_events[4];
  hipEvent_t* ev_free = &C->sync_events[4 + nslot];      // dK/dV kernel done with the slot
  hipEvent_t* ev_free_q = &C->sync_events[4 + 2 * nslot]; // dQ kernel done with the slot
  hipEvent_t* ev_d2h = &C->sync_events[4 + 3 * nslot];    // the slot's gradients copied out
  hipEvent_t* ev_chunk = &C->sync_events[4 + 4 * nslot];  // preprocess done with the slot
  const int64_t dq_rows = dq_rows_per_wg(int(d)), kv_rows = dkdv_rows_per_wg(int(d));
  // work groups of a launch over tasks [t0, t0 + n): each task's strips
  auto wgs_of = [&](int64_t t0, int64_t n, int64_t rows) {
    int64_t w = 0;
    for (int64_t t = t0; t < t0 + n; ++t) w += (p->tasks[t].L_local + rows - 1) / rows * B * H;
    return w;
  };
  // the dQ stream, one for the whole call: the caller's stream when the
  // longest dK/dV launch spans many rounds of resident waves (one wave per 32
  // keys), else the second compute stream
  int64_t kv_waves = 0;
  if (batched)
    for (const Group& gr : p->bwd_groups)
      kv_waves = std::max(kv_waves, wgs_of(gr.task0, gr.count, kv_rows) * (kv_rows / 32));
  else
    for (int64_t t = 0; t < ntask; ++t) kv_waves = std::max(kv_waves, wgs_of(t, 1, kv_rows) * (kv_rows / 32));
  const hipStream_t cs = C->copy, qs = serial_launch(kv_waves) ? st : C->lane, ms = C->aux;
  if (C->ws_free_valid) CQSA_HIP(hipStreamWaitEvent(st, C->ws_free, 0));
  // tile-decision counters, zeroed before every kernel (the other streams
  // start after events recorded on st below)
  unsigned long long* tile_count = nullptr;
  if (tile_counting_enabled())
    if ((s = tile_counters_begin(C, st, 6, &tile_count)) != CQSA_OK) return s;
  CQSA_HIP(hipEventRecord(ev_start, st));
  CQSA_HIP(hipStreamWaitEvent(cs, ev_start, 0));
  if ((s = upload_image(C, p->packed, d_tab, cs)) != CQSA_OK) return s;
  if (!dev_acc) {
    CQSA_HIP(hipMemcpyAsync((void*)d_lse, LSE, uint64_t(B) * H * L * 4, hipMemcpyHostToDevice, cs));
    rec.stats.h2d_bytes += uint64_t(B) * H * L * 4;
  }
  CQSA_HIP(hipEventRecord(ev_tab, cs));

  auto span_begin = [&](hipStream_t sm) -> std::pair<hipEvent_t, hipEvent_t> {
    std::pair<hipEvent_t, hipEvent_t> sp{nullptr, nullptr};
    if (rec.timing) {
      sp = {rec.make(), rec.make()};
      if (hipEventRecord(sp.first, sm) != hipSuccess) sp = {nullptr, nullptr};
    }
    return sp;
  };
  auto span_end = [&](std::pair<hipEvent_t, hipEvent_t> sp, hipStream_t sm, Stage k) {
    if (sp.first && hipEventRecord(sp.second, sm) == hipSuccess) rec.spans[k].push_back(sp);
  };

  // ---- D = rowsum(dO * O) on the caller's stream ----
  if (dev_in && dev_acc) {
    auto sp = span_begin(st);
    CQSA_HIP(launch_bwd_preprocess(dO->data, (const float*)O->data, d_D, o.dtype, B, L, H, int(d),
                                   L, st));
    span_end(sp, st, kStFinal);
  } else {
    // rows of one batch element in chunks of the longest task's length: a
    // host-resident dO chunk goes to the slot's staged-input area, a
    // host-resident O chunk to its gradient area (both at least that large)
    const int64_t crows = std::max<int64_t>(1, p->max_L_local);
    int64_t c = 0;
    for (int64_t b = 0; b < B; ++b)
      for (int64_t g0 = 0; g0 < L; g0 += crows, ++c) {
        const int64_t n = std::min(crows, L - g0);
        const int64_t si = c % nslot;
        char* sb = slot_base(si);
        if (c >= nslot) CQSA_HIP(hipStreamWaitEvent(cs, ev_chunk[si], 0));
        const uint64_t off_in = uint64_t(b * L + g0) * row_bytes;
        const uint64_t off_o = uint64_t(b * L + g0) * H * d * 4;
        const void* pdo = (const char*)dO->data + off_in;
        const float* po = (const float*)((const char*)O->data + off_o);
        auto sp = span_begin(cs);
        if (!dev_in) {
          CQSA_HIP(hipMemcpyAsync(sb, pdo, n * row_bytes, hipMemcpyHostToDevice, cs));
          pdo = sb;
          rec.stats.h2d_bytes += uint64_t(n) * row_bytes;
        }
        if (!dev_acc) {
          char* dst = sb + 4 * in_b;
          CQSA_HIP(hipMemcpyAsync(dst, po, n * H * d * 4, hipMemcpyHostToDevice, cs));
          po = (const float*)dst;
          rec.stats.h2d_bytes += uint64_t(n) * H * d * 4;
        }
        span_end(sp, cs, kStStage);
        CQSA_HIP(hipEventRecord(ev_staged[si], cs));
        CQSA_HIP(hipStreamWaitEvent(st, ev_staged[si], 0));
        auto sq = span_begin(st);
        CQSA_HIP(launch_bwd_preprocess(pdo, po, d_D + b * H * L + g0, o.dtype, 1, n, H, int(d), L,
                                       st));
        span_end(sq, st, kStFinal);
        CQSA_HIP(hipEventRecord(ev_chunk[si], st));
      }
    // task staging reuses the slots once every chunk is consumed
    CQSA_HIP(hipEventRecord(ev_pre, st));
    CQSA_HIP(hipStreamWaitEvent(cs, ev_pre, 0));
  }

  HostMerger merger;
  float* const hgrad[3] = {(float*)dQ->data, (float*)dK->data, (float*)dV->data};
  char* pin = nullptr;
  const uint64_t pin_slot = 3 * g_b;
  if (dev_acc && !batched && !direct) {
    // the fused scatter-adds accumulate into zeroed gradients
    auto sp = span_begin(st);
    for (int x = 0; x < 3; ++x) CQSA_HIP(launch_fill_zero(hgrad[x], B * L * H * d, st));
    span_end(sp, st, kStMerge);
  } else if (!dev_acc) {
    void* pv = nullptr;
    if ((s = acquire_pinned(C, size_t(pin_slot * nslot), &pv)) != CQSA_OK) return s;
    pin = (char*)pv;
    // the host zero-fill runs on the merge thread while the device computes
    const int64_t n = B * L * H * d;
    merger.push([=, &rec]() -> bool {
      auto t0 = std::chrono::steady_clock::now();
      host_zero(hgrad, n);
      auto t1 = std::chrono::steady_clock::now();
      rec.host_merge_ms += std::chrono::duration<double, std::milli>(t1 - t0).count();
      return true;
    });
  }
  CQSA_HIP(hipStreamWaitEvent(st, ev_tab, 0));
  // dQ kernels write dQ only and dK/dV kernels dK and dV only, so on the
  // second stream a task's two kernels overlap; each stream keeps its own
  // tasks in order.  (With qs the caller's stream these waits are no-ops.)
  CQSA_HIP(hipEventRecord(ev_pre, st));
  CQSA_HIP(hipStreamWaitEvent(qs, ev_pre, 0));

  auto common_args = [&](BwdArgs& a, int64_t t0, int64_t n) {
    a.tab = d_tab;
    a.tasks = (const DevTask*)d_tab + t0;
    a.ntask = int32_t(n);
    a.B = int32_t(B); a.H = int32_t(H); a.causal = p->g.causal;
    a.scale_log2 = sc * 1.4426950408889634f; a.scale = sc;
    a.lse = d_lse; a.D = d_D; a.Lg = L;
    a.tile_count = tile_count;
  };
  if (batched) {
    float* loc = (float*)(base + tab_bytes + stat_bytes + lse_bytes + uint64_t(nslot) * slot_bytes);
    const int64_t stride = int64_t(loc_b / 4);
    float* lg[3] = {loc, loc + gmax * stride, loc + 2 * gmax * stride};
    for (size_t k = 0; k < p->bwd_groups.size(); ++k) {
      const Group& gr = p->bwd_groups[k];
      BwdArgs a{};
      a.q = Q->data; a.k = K->data; a.v = V->data; a.dO = dO->data;
      a.in_place = 1;
      common_args(a, gr.task0, gr.count);
      a.local_out = 1;
      a.out_stride = stride;
      a.dq = lg[0]; a.dk = lg[1]; a.dv = lg[2];
      // the previous group's merge has read the local buffers (it runs on the
      // caller's stream, ahead of this group's dK/dV launch)
      if (k > 0) {
        CQSA_HIP(hipEventRecord(ev_pre, st));
        CQSA_HIP(hipStreamWaitEvent(qs, ev_pre, 0));
      }
      auto sk = span_begin(st);
      CQSA_HIP(launch_bwd_dkdv(o.dtype, int(d), a, wgs_of(gr.task0, gr.count, kv_rows), st));
      span_end(sk, st, kStInner);
      auto sq = span_begin(qs);
      CQSA_HIP(launch_bwd_dq(o.dtype, int(d), a, wgs_of(gr.task0, gr.count, dq_rows), qs));
      span_end(sq, qs, kStInner);
      rec.stats.inner_launches += 2;
      CQSA_HIP(hipEventRecord(ev_join, qs));
      CQSA_HIP(hipStreamWaitEvent(st, ev_join, 0));
      GradMergeArgs m{};
      m.segs = (const DevSeg*)(d_tab + gr.seg_off);
      m.n_seg = gr.n_seg;
      m.contribs = (const DevContrib*)(d_tab + gr.contrib_off);
      m.tasks = (const DevTask*)d_tab + gr.task0;
      for (int x = 0; x < 3; ++x) {
        m.src[x] = lg[x];
        m.dst[x] = hgrad[x];
      }
      m.stride = stride;
      m.L = L; m.B = int32_t(B); m.H = int32_t(H); m.d = int32_t(d);
      auto sm = span_begin(st);
      CQSA_HIP(launch_grad_merge(m, gr.blocks, st));
      rec.stats.merge_launches += 1;
      span_end(sm, st, kStMerge);
    }
  }

  std::vector<bool> used(nslot, false);
  std::vector<int64_t> last_item(nslot, -1);
  const Task* prev_task = nullptr;
  const char* prev_sb = nullptr;
  const char* srcs[4] = {(const char*)Q->data, (const char*)K->data, (const char*)V->data,
                         (const char*)dO->data};
  for (int64_t t = 0; t < (batched ? 0 : ntask); ++t) {
    const Task& task = p->tasks[t];
    const int64_t Li = task.L_local;
    if (Li == 0) continue;
    const int64_t si = t % nslot;
    const TableOffsets& to = p->table_off[t];
    char* sb = slot_base(si);
    BwdArgs a{};
    if (!staged) {
      a.q = Q->data; a.k = K->data; a.v = V->data; a.dO = dO->data;
      a.in_place = in_place ? 1 : 0;
    } else {
      if (used[si]) {
        CQSA_HIP(hipStreamWaitEvent(cs, ev_free[si], 0));
        CQSA_HIP(hipStreamWaitEvent(cs, ev_free_q[si], 0));
      }
      char* dsts[4] = {sb, sb + in_b, sb + 2 * in_b, sb + 3 * in_b};
      auto sp = span_begin(cs);
      if (dev_in) {
        StageArgs sa{};
        for (int x = 0; x < 4; ++x) {
          sa.src[x] = srcs[x];
          sa.dst[x] = dsts[x];
        }
        sa.n_tensors = 4; sa.row_bytes = row_bytes; sa.Li = Li; sa.Lg = L; sa.B = int32_t(B);
        sa.runs = d_tab + to.runs; sa.n_runs = int32_t(task.runs.size());
        CQSA_HIP(launch_stage(sa, cs));
        rec.stats.d2d_bytes += uint64_t(4) * B * Li * row_bytes;
      } else {
        // host inputs: tokens the previously staged task also holds come
        // from its staged rows (intact until a later staging on this copy
        // stream overwrites them), the rest over the host link
        const bool can_reuse = prev_task && prev_sb != sb;
        const int64_t Lp = can_reuse ? prev_task->L_local : 0;
        for (const StagePiece& pc : stage_pieces(task, can_reuse ? prev_task : nullptr)) {
          for (int x = 0; x < 4; ++x)
            for (int64_t b = 0; b < B; ++b) {
              char* dst = dsts[x] + (b * Li + pc.dst) * row_bytes;
              if (pc.reuse)
                CQSA_HIP(hipMemcpyAsync(dst, prev_sb + x * in_b + (b * Lp + pc.src) * row_bytes,
                                        pc.length * row_bytes, hipMemcpyDeviceToDevice, cs));
              else
                CQSA_HIP(hipMemcpyAsync(dst, srcs[x] + (b * L + pc.src) * row_bytes,
                                        pc.length * row_bytes, hipMemcpyHostToDevice, cs));
            }
          const uint64_t moved = uint64_t(4) * B * pc.length * row_bytes;
          if (pc.reuse)
            rec.stats.d2d_bytes += moved;
          else
            rec.stats.h2d_bytes += moved;
        }
        prev_task = &task;
        prev_sb = sb;
      }
      span_end(sp, cs, kStStage);
      CQSA_HIP(hipEventRecord(ev_staged[si], cs));
      CQSA_HIP(hipStreamWaitEvent(st, ev_staged[si], 0));
      CQSA_HIP(hipStreamWaitEvent(qs, ev_staged[si], 0));
      a.q = dsts[0]; a.k = dsts[1]; a.v = dsts[2]; a.dO = dsts[3];
    }
    common_args(a, t, 1);
    float* tg[3] = {nullptr, nullptr, nullptr};
    if (dev_acc) {
      // undecomposed, local rows are the global rows: the task stores them
      a.local_out = direct ? 1 : 0;
      a.dq = hgrad[0]; a.dk = hgrad[1]; a.dv = hgrad[2];
    } else {
      // the task's own gradients; the slot's previous ones must be copied out
      for (int x = 0; x < 3; ++x) tg[x] = (float*)(sb + 4 * in_b + x * g_b);
      a.local_out = 1;
      a.dq = tg[0]; a.dk = tg[1]; a.dv = tg[2];
      if (used[si]) {
        CQSA_HIP(hipStreamWaitEvent(st, ev_d2h[si], 0));
        CQSA_HIP(hipStreamWaitEvent(qs, ev_d2h[si], 0));
      }
    }
    auto sk = span_begin(st);
    CQSA_HIP(launch_bwd_dkdv(o.dtype, int(d), a, wgs_of(t, 1, kv_rows), st));
    span_end(sk, st, kStInner);
    auto sq = span_begin(qs);
    CQSA_HIP(launch_bwd_dq(o.dtype, int(d), a, wgs_of(t, 1, dq_rows), qs));
    span_end(sq, qs, kStInner);
    rec.stats.inner_launches += 2;
    CQSA_HIP(hipEventRecord(ev_free[si], st));
    CQSA_HIP(hipEventRecord(ev_free_q[si], qs));
    if (!dev_acc) {
      // the slot's pinned staging must have been added by its last job
      if (!merger.wait_done(last_item[si])) return fail(CQSA_ERR_HIP, "host scatter-add failed");
      float* hp[3];
      for (int x = 0; x < 3; ++x) hp[x] = (float*)(pin + uint64_t(si) * pin_slot + x * g_b);
      CQSA_HIP(hipStreamWaitEvent(ms, ev_free[si], 0));
      CQSA_HIP(hipStreamWaitEvent(ms, ev_free_q[si], 0));
      const uint64_t bytes = uint64_t(B) * Li * H * d * 4;
      auto sp = span_begin(ms);
      for (int x = 0; x < 3; ++x)
        CQSA_HIP(hipMemcpyAsync(hp[x], tg[x], bytes, hipMemcpyDeviceToHost, ms));
      span_end(sp, ms, kStD2H);
      rec.stats.d2h_bytes += 3 * bytes;
      CQSA_HIP(hipEventRecord(ev_d2h[si], ms));
      const hipEvent_t wait_ev = ev_d2h[si];
      const Task* tp = &task;
      const float* const srcp[3] = {hp[0], hp[1], hp[2]};
      last_item[si] = merger.push([=, &rec]() -> bool {
        if (hipEventSynchronize(wait_ev) != hipSuccess) return false;
        auto t0 = std::chrono::steady_clock::now();  // the adds alone, not the wait
        host_scatter_add(*tp, srcp, hgrad, B, L, H, d);
        auto t1 = std::chrono::steady_clock::now();
        rec.host_merge_ms += std::chrono::duration<double, std::milli>(t1 - t0).count();
        return true;
      });
    }
    used[si] = true;
  }
  // join the dQ stream (and the gradient copies) back into the caller's stream
  CQSA_HIP(hipEventRecord(ev_join, qs));
  CQSA_HIP(hipStreamWaitEvent(st, ev_join, 0));
  if (!dev_acc) {
    CQSA_HIP(hipEventRecord(ev_join, ms));
    CQSA_HIP(hipStreamWaitEvent(st, ev_join, 0));
  }
  if (rec.timing) CQSA_HIP(hipEventRecord(rec.wall1, st));
  if (tile_count && (s = tile_counters_end(C, rec, st, 6)) != CQSA_OK) return s;
  CQSA_HIP(hipEventRecord(C->ws_free, st));
  C->ws_free_valid = true;
  release_workspace(C, &ws, st);
  if (!dev_acc) {
    if (!merger.finish()) return fail(CQSA_ERR_HIP, "host scatter-add: event wait failed");
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  }
  return CQSA_OK;
}

}  // namespace cqsa

extern "C" cqsa_status cqsa_backward(const cqsa_plan_t* plan, const cqsa_tensor* Q,
                                     const cqsa_tensor* K, const cqsa_tensor* V,
                                     const cqsa_tensor* O, const float* LSE, cqsa_mem lse_where,
                                     const cqsa_tensor* dO, cqsa_tensor* dQ, cqsa_tensor* dK,
                                     cqsa_tensor* dV, float scale, void* hip_stream) {
  cqsa::clear_error();
  try {
    return cqsa::run_guarded(plan, true, [&](const cqsa_plan_t* q) {
      return cqsa::backward_impl(q, Q, K, V, O, LSE, lse_where, dO, dQ, dK, dV, scale,
                               (hipStream_t)hip_stream);
    });
  } catch (const std::exception& e) {
    return cqsa::fail(CQSA_ERR_INTERNAL, std::string("cqsa_backward: ") + e.what());
  } catch (...) {
    return cqsa::fail(CQSA_ERR_INTERNAL, "cqsa_backward: unknown exception");
  }
}
