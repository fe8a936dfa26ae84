// cqsa_forward: the task streamer of the decomposed forward.
//
// The plan cuts the task list into launch groups of `group_size` consecutive
// tasks (Alg. 1, computed with the max-shifted merge of App. A.1).  Per group:
//   copy stream    : gather every task's runs of Q, K, V into its sub-slot of
//                    staging slot k % S (H2D from host inputs or D2D), then
//                    signal "staged";
//   compute stream : wait "staged", run ONE inner-kernel launch over all the
//                    group's tasks (local statistics per task); groups
//                    alternate between the caller's stream and a second
//                    compute stream so that consecutive launches overlap;
//   aux stream     : device accumulator -- one gather-merge launch folds the
//                    group's statistics into the running (acc, m, l), and the
//                    last group's merge writes O and LSE; host accumulator --
//                    D2H of the statistics, merged by a host thread;
//   the slot is freed by an event once its last reader is done.
// With S >= 2 slots the gather of group k+1 overlaps the compute of group k
// (App. A.3: transfers overlap compute).  When the plan reads device-resident
// inputs in place nothing is gathered: a slot holds statistics only, and
// with a single launch group the image upload, the inner launch and the
// merge all run on the caller's stream.  Host-resident inputs reuse the
// tokens the previously staged task also holds (a device-to-device copy from
// its staged rows).  Depth 0 on device-resident tensors is the undecomposed
// call: one kernel that writes O and LSE directly.
#include <algorithm>
#include <chrono>
#include <cmath>

#include "guard.hpp"
#include "kernels.hpp"
#include "runtime.hpp"
#include "streamer.hpp"

namespace cqsa {

namespace {

// Max-shifted merge of one task's statistics into the host accumulator
// (Eq. "merge", log2 domain, null rows skipped); l and lt (the sums of the
// fp32 and of the rounded weights) merge with the same factors.  A row whose running max is
// still -inf has had no contribution yet: the first one is written, not
// blended, so the accumulator needs no zero fill beforehand (every token has
// a kept key in some task, so every row is written before finalisation).
void host_merge(const Task& task, const float* acc_i, const float* m_i, const float* l_i,
                const float* lt_i, float* acc, float* m, float* l, float* lt, int64_t B,
                int64_t L, int64_t H, int64_t d) {
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
        const float* src = acc_i + ((b * Li + r) * H + h) * d;
        float* dst = acc + ((b * L + g) * H + h) * d;
        if (mo == -INFINITY) {
          for (int64_t k = 0; k < d; ++k) dst[k] = src[k];
          l[gi] = l_i[si];
          lt[gi] = lt_i[si];
          m[gi] = mi;
          continue;
        }
        const float mn = std::max(mo, mi);
        const float fo = std::exp2(mo - mn);
        const float fi = std::exp2(mi - mn);
        for (int64_t k = 0; k < d; ++k) dst[k] = dst[k] * fo + src[k] * fi;
        l[gi] = l[gi] * fo + l_i[si] * fi;
        lt[gi] = lt[gi] * fo + lt_i[si] * fi;
        m[gi] = mn;
      }
    }
  });
}

// O = acc / lt, LSE = m + log l (natural log).
void host_finalize(float* acc, float* m, const float* l, const float* lt, int64_t B, int64_t L,
                   int64_t H, int64_t d) {
  parallel_rows(B * L, [&](int64_t lo, int64_t hi) {
    for (int64_t x = lo; x < hi; ++x) {
      const int64_t b = x / L, g = x % L;
      for (int64_t h = 0; h < H; ++h) {
        const int64_t gi = (b * H + h) * L + g;
        const float inv = 1.f / lt[gi];
        float* row = acc + ((b * L + g) * H + h) * d;
        for (int64_t k = 0; k < d; ++k) row[k] *= inv;
        m[gi] = (m[gi] + std::log2(l[gi])) * 0.69314718055994530942f;
      }
    }
  });
}

}  // namespace

// noalloc: the cqsa_forward_noalloc contract -- the workspace is the device's
// scratch array, the plan image is copied straight from the plan, and nothing
// is allocated (no workspace, pinned host buffer, timing event or new
// synchronisation event).
cqsa_status forward_impl(const cqsa_plan_t* p, const cqsa_tensor* Q, const cqsa_tensor* K,
                         const cqsa_tensor* V, cqsa_tensor* O, float* LSE, cqsa_mem lse_where,
                         float scale, hipStream_t st, bool noalloc) {
  if (!p) return fail(CQSA_ERR_INVALID_ARG, "cqsa_forward: plan is NULL");
  const cqsa_plan_opts& o = p->opts;
  const cqsa_mem in_where = o.inputs_on_device ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  const cqsa_mem acc_where = o.acc_on_device ? CQSA_MEM_DEVICE : CQSA_MEM_HOST;
  cqsa_status s;
  if ((s = check_tensor(Q, "Q", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(K, "K", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(V, "V", p, o.dtype, in_where)) != CQSA_OK) return s;
  if ((s = check_tensor(O, "O", p, o.out16 ? o.dtype : CQSA_F32, acc_where)) != CQSA_OK) return s;
  if (!LSE) return fail(CQSA_ERR_INVALID_ARG, "LSE is NULL");
  if (lse_where != acc_where)
    return fail(CQSA_ERR_INVALID_ARG, "LSE residency must equal the output residency");

  if (noalloc && !o.acc_on_device)
    return fail(CQSA_ERR_INVALID_ARG,
                "cqsa_forward_noalloc: the plan must keep O and LSE on the device "
                "(a host accumulator needs pinned staging)");

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
  const bool direct = direct_forward(o, depth);
  // kernels address the runs inside the caller's tensors: nothing is staged
  const bool in_place = o.read_in_place == 1;

  CallRecord& rec = call_record();
  rec.reset();
  if (noalloc) rec.timing = false;  // timing events would be created per call
  rec.stats.depth = depth;
  rec.stats.num_tasks = ntask;
  rec.stats.modelled_device_bytes = p->fp.peak;
  if (rec.timing) {
    rec.wall0 = rec.make();
    rec.wall1 = rec.make();
    CQSA_HIP(hipEventRecord(rec.wall0, st));
  }

  // ---- workspace layout ----
  // [plan image][running l, lt][slot 0]...[slot S-1]; a slot holds group_size
  // task sub-slots {Q, K, V, acc, m, l, lt} ({acc, m, l, lt} when the inputs
  // are read in place), each sized for the longest task.
  const int64_t ngroup = int64_t(p->groups.size());
  const int64_t gsz = p->fp.group_size;
  const uint64_t tab_bytes = align_up(p->packed.size());
  const uint64_t gl_one = align_up(uint64_t(B) * H * L * 4);
  const uint64_t gl_bytes = (acc_dev && !direct && ngroup > 1) ? 2 * gl_one : 0;
  const uint64_t sub_bytes = direct ? 0 : fwd_slot_bytes(p->g, o, p->max_L_local, !in_place, true);
  std::vector<int64_t> slot_tasks;
  if (!direct) slot_tasks = fwd_slot_tasks(ntask, int32_t(gsz), o.n_slots);
  const int64_t nslot = int64_t(slot_tasks.size());
  std::vector<uint64_t> slot_off(nslot + 1, 0);
  for (int64_t i = 0; i < nslot; ++i) slot_off[i + 1] = slot_off[i] + uint64_t(slot_tasks[i]) * sub_bytes;
  // fp32 result when O is 16-bit: [B, L, H, d] after the slots
  const uint64_t o32_bytes = o.out16 ? align_up(uint64_t(B) * L * H * d * 4) : 0;
  const uint64_t total = tab_bytes + gl_bytes + slot_off[nslot] + o32_bytes;
  const size_t events = size_t(4 * std::max<int64_t>(nslot, 1) + 3);
  Workspace ws;
  if (noalloc) {
    if (total > CQSA_NOALLOC_SCRATCH_BYTES)
      return fail(CQSA_ERR_INVALID_ARG,
                  "cqsa_forward_noalloc: the call's workspace (" + std::to_string(total) +
                      " bytes) exceeds the " + std::to_string(CQSA_NOALLOC_SCRATCH_BYTES) +
                      "-byte scratch");
    if (events > C->sync_events.size())
      return fail(CQSA_ERR_INVALID_ARG,
                  "cqsa_forward_noalloc: at most 3 staging slots (the set-up events)");
    ws.ptr = C->scratch;
    ws.bytes = total;
  } else if ((s = acquire_workspace(C, total, &ws)) != CQSA_OK) {
    return s;
  }
  rec.stats.workspace_bytes = total;
  rec.stats.resident_tasks = direct ? 0 : fwd_subslots(ntask, int32_t(gsz), o.n_slots);
  char* base = (char*)ws.ptr;
  char* d_tab = base;
  float* d_gl = gl_bytes ? (float*)(base + tab_bytes) : nullptr;
  float* d_glt = gl_bytes ? (float*)(base + tab_bytes + gl_one) : nullptr;
  const uint64_t in_b = in_place ? 0 : align_up(uint64_t(B) * p->max_L_local * H * d * elem);
  const uint64_t acc_b = align_up(uint64_t(B) * p->max_L_local * H * d * 4);
  const uint64_t st_b = align_up(uint64_t(B) * p->max_L_local * H * 4);
  auto slot_base = [&](int64_t si) { return base + tab_bytes + gl_bytes + slot_off[si]; };
  const DevTask* d_tasks = (const DevTask*)d_tab;
  const int rows_wg = fwd_rows_per_wg(o.dtype, int(d));

  // ---- ordering against the caller's stream and the previous call ----
  while (C->sync_events.size() < events) {
    hipEvent_t e;
    CQSA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    C->sync_events.push_back(e);
  }
  hipEvent_t ev_start = C->sync_events[0];
  hipEvent_t ev_tail = C->sync_events[1];
  hipEvent_t* ev_staged = &C->sync_events[2];
  hipEvent_t* ev_free = &C->sync_events[2 + nslot];
  hipEvent_t* ev_inner = &C->sync_events[2 + 2 * nslot];
  // after the previous call's last use of the same workspace
  hipEvent_t& ws_free = noalloc ? C->scratch_free : C->ws_free;
  bool& ws_free_valid = noalloc ? C->scratch_free_valid : C->ws_free_valid;
  if (ws_free_valid) CQSA_HIP(hipStreamWaitEvent(st, ws_free, 0));
  // tile-decision counters, zeroed before every inner launch (the other
  // streams start after events recorded on st below)
  unsigned long long* tile_count = nullptr;
  if (!noalloc && tile_counting_enabled() && o.dtype != CQSA_F32)
    if ((s = tile_counters_begin(C, st, 3, &tile_count)) != CQSA_OK) return s;
  // With nothing to stage and a single launch group (the direct call, or
  // inputs read in place with every task in one launch) the whole call runs
  // on the caller's stream: each hop between streams costs the GPU an event
  // round trip per call.  Otherwise the image and the staging copies go on
  // the copy stream and merges on the auxiliary stream.
  const bool one_stream = direct || (in_place && acc_dev && ngroup == 1);
  const hipStream_t cs = one_stream ? st : C->copy;  // image and staging copies
  const hipStream_t ms = one_stream ? st : C->aux;   // merges, statistics D2H
  if (cs != st) {
    CQSA_HIP(hipEventRecord(ev_start, st));
    CQSA_HIP(hipStreamWaitEvent(cs, ev_start, 0));
  }
  if (noalloc) {
    // from the plan's own (pageable) memory: no pinned staging ring
    if (!p->packed.empty())
      CQSA_HIP(hipMemcpyAsync(d_tab, p->packed.data(), p->packed.size(), hipMemcpyHostToDevice, cs));
  } else if ((s = upload_image(C, p->packed, d_tab, cs)) != CQSA_OK) {
    return s;
  }

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

  float* Od = o.out16 ? (float*)(base + tab_bytes + gl_bytes + slot_off[nslot]) : (float*)O->data;
  if (direct) {
    FwdArgs a{};
    a.q = Q->data; a.k = K->data; a.v = V->data;
    a.acc = Od; a.m = LSE; a.l = nullptr; a.lt = nullptr;
    a.tab = d_tab; a.tasks = d_tasks; a.ntask = 1;
    a.B = int32_t(B); a.H = int32_t(H); a.causal = p->g.causal; a.scale_log2 = scale_log2;
    a.tile_count = tile_count;
    const int64_t wgs = ((L + rows_wg - 1) / rows_wg) * B * H;
    auto sp = span_begin(st);
    CQSA_HIP(launch_fwd(o.dtype, int(d), kModeFinal, a, wgs, st));
    span_end(sp, st, kStInner);
    rec.stats.inner_launches = 1;
  } else {
    // running global state: acc in the O buffer, m (log2) in the LSE buffer,
    // l and lt in the workspace (device) or on the host
    float* acc = Od;
    float* m = LSE;
    float* l = d_gl;
    float* lt = d_glt;
    std::vector<float> l_host, lt_host;
    char* pin = nullptr;
    uint64_t pin_slot = 0;
    if (!acc_dev) {
      // running max -inf marks rows not yet merged (host_merge writes their
      // first contribution), so acc itself needs no fill
      l_host.assign(size_t(B * H * L), 0.f);
      lt_host.assign(size_t(B * H * L), 0.f);
      l = l_host.data();
      lt = lt_host.data();
      std::fill(m, m + B * H * L, -INFINITY);
      pin_slot = acc_b + 3 * st_b;
      void* pv = nullptr;
      if ((s = acquire_pinned(C, size_t(pin_slot * nslot), &pv)) != CQSA_OK) return s;
      pin = (char*)pv;
    }
    HostMerger merger;
    std::vector<int64_t> last_item(nslot, -1);
    std::vector<bool> used(nslot, false);
    const hipMemcpyKind kind = in_dev ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    const char* srcs[3] = {(const char*)Q->data, (const char*)K->data, (const char*)V->data};
    // the task staged last and where its rows sit (host inputs reuse them)
    const Task* prev_task = nullptr;
    const char* prev_sub = nullptr;
    for (int64_t k = 0; k < ngroup; ++k) {
      const Group& G = p->groups[k];
      const int64_t si = k % nslot;
      char* sb = slot_base(si);
      // The slot's staged inputs are free once its previous group's inner
      // kernel is done; its statistics once their merge or D2H is done.
      // Staging waits for the first only, so the H2D of this group overlaps
      // the D2H of the slot's previous statistics.
      if (used[si] && !in_place) CQSA_HIP(hipStreamWaitEvent(cs, ev_inner[si], 0));
      // gather every task of the group into its sub-slot
      int64_t wgs = 0;
      for (int64_t j = 0; j < G.count; ++j) {
        const int64_t t = G.task0 + j;
        const Task& task = p->tasks[t];
        const int64_t Li = task.L_local;
        wgs += ((Li + rows_wg - 1) / rows_wg) * B * H;
        if (Li == 0 || in_place) continue;
        char* sub = sb + uint64_t(j) * sub_bytes;
        char* dsts[3] = {sub, sub + in_b, sub + 2 * in_b};
        auto sp = span_begin(cs);
        if (in_dev) {
          // device inputs: one gather kernel over the runs of all three tensors
          StageArgs sa{};
          for (int x = 0; x < 3; ++x) {
            sa.src[x] = srcs[x];
            sa.dst[x] = dsts[x];
          }
          sa.n_tensors = 3; sa.row_bytes = int64_t(row_bytes); sa.Li = Li; sa.Lg = L;
          sa.B = int32_t(B); sa.runs = d_tab + p->table_off[t].runs;
          sa.n_runs = int32_t(task.runs.size());
          CQSA_HIP(launch_stage(sa, cs));
          rec.stats.d2d_bytes += uint64_t(3) * B * Li * row_bytes;
        } else {
          // host inputs: tokens the previously staged task also holds are
          // copied device to device from its staged rows, which stay intact
          // until a later staging (this copy stream) overwrites them; the
          // rest crosses the host link, one asynchronous copy per piece and
          // batch element.  No reuse when both tasks use the same sub-slot.
          const bool can_reuse = prev_task && prev_sub != sub;
          const int64_t Lp = can_reuse ? prev_task->L_local : 0;
          const uint64_t in_bp = in_b;  // sub-slot tensor stride, as for dsts
          for (const StagePiece& pc : stage_pieces(task, can_reuse ? prev_task : nullptr)) {
            for (int x = 0; x < 3; ++x)
              for (int64_t b = 0; b < B; ++b) {
                char* dst = dsts[x] + (b * Li + pc.dst) * row_bytes;
                if (pc.reuse)
                  CQSA_HIP(hipMemcpyAsync(dst, prev_sub + x * in_bp + (b * Lp + pc.src) * row_bytes,
                                          pc.length * row_bytes, hipMemcpyDeviceToDevice, cs));
                else
                  CQSA_HIP(hipMemcpyAsync(dst, srcs[x] + (b * L + pc.src) * row_bytes,
                                          pc.length * row_bytes, kind, cs));
              }
            const uint64_t moved = uint64_t(3) * B * pc.length * row_bytes;
            if (pc.reuse)
              rec.stats.d2d_bytes += moved;
            else
              rec.stats.h2d_bytes += moved;
          }
          prev_task = &task;
          prev_sub = sub;
        }
        span_end(sp, cs, kStStage);
      }
      // Consecutive groups alternate between the caller's stream and a second
      // compute stream, so a short launch fills the tail of the previous one
      // (App. A.3: at most two slots in flight).  A launch of many rounds of
      // resident work groups has a negligible tail; two such launches in
      // flight would only share the GPU, so they stay on the caller's stream
      // and run one after the other.  Inner kernels write only their slot.
      const int64_t waves = wgs * (rows_wg / 32);  // one wave per 32 query rows
      const bool alternate = !serial_launch(waves);
      const hipStream_t ls = (alternate && (k & 1)) ? C->lane : st;
      if (ls != cs) {
        CQSA_HIP(hipEventRecord(ev_staged[si], cs));
        CQSA_HIP(hipStreamWaitEvent(ls, ev_staged[si], 0));
      }
      // the inner kernel overwrites the slot's statistics
      if (used[si]) CQSA_HIP(hipStreamWaitEvent(ls, ev_free[si], 0));
      FwdArgs a{};
      if (in_place) {
        a.q = Q->data; a.k = K->data; a.v = V->data;
        a.in_stride = 0;
        a.in_place = 1;
        a.Lg = L;
      } else {
        a.q = sb; a.k = sb + in_b; a.v = sb + 2 * in_b;
        a.in_stride = int64_t(sub_bytes / elem);
      }
      a.acc = (float*)(sb + 3 * in_b);
      a.m = (float*)(sb + 3 * in_b + acc_b);
      a.l = (float*)(sb + 3 * in_b + acc_b + st_b);
      a.lt = (float*)(sb + 3 * in_b + acc_b + 2 * st_b);
      a.acc_stride = a.st_stride = int64_t(sub_bytes / 4);
      a.tab = d_tab; a.tasks = d_tasks + G.task0; a.ntask = int32_t(G.count);
      a.B = int32_t(B); a.H = int32_t(H); a.causal = p->g.causal; a.scale_log2 = scale_log2;
      a.tile_count = tile_count;
      {
        auto sp = span_begin(ls);
        CQSA_HIP(launch_fwd(o.dtype, int(d), kModeStats, a, wgs, ls));
        span_end(sp, ls, kStInner);
      }
      rec.stats.inner_launches += 1;
      CQSA_HIP(hipEventRecord(ev_inner[si], ls));
      if (acc_dev) {
        // merge on the auxiliary stream: combines run in group order there,
        // and the next group's inner kernel overlaps this one's combine
        if (ms != ls) CQSA_HIP(hipStreamWaitEvent(ms, ev_inner[si], 0));
        CombineArgs cb{};
        cb.segs = (const DevSeg*)(d_tab + G.seg_off); cb.n_seg = G.n_seg;
        cb.contribs = (const DevContrib*)(d_tab + G.contrib_off);
        cb.tasks = d_tasks + G.task0;
        cb.acc_i = a.acc; cb.m_i = a.m; cb.l_i = a.l; cb.lt_i = a.lt;
        cb.acc_stride = a.acc_stride; cb.st_stride = a.st_stride;
        cb.acc = acc; cb.m = m; cb.l = l; cb.lt = lt; cb.L = L;
        cb.B = int32_t(B); cb.H = int32_t(H); cb.d = int32_t(d); cb.final = G.final ? 1 : 0;
        if (G.blocks > 0) {
          auto sp = span_begin(ms);
          CQSA_HIP(launch_combine(cb, G.blocks, ms));
          span_end(sp, ms, kStMerge);
          rec.stats.merge_launches += 1;
        }
        CQSA_HIP(hipEventRecord(ev_free[si], ms));
      } else {
        // hand the statistics to the host: D2H into pinned staging, then merge;
        // the staging of this slot must have been consumed by its last merge
        // (groups hold one task when the accumulator is on the host)
        if (!merger.wait_done(last_item[si])) return fail(CQSA_ERR_HIP, "host merge failed");
        const int64_t t = G.task0;
        const int64_t Li = p->tasks[t].L_local;
        char* hp = pin + uint64_t(si) * pin_slot;
        const uint64_t rows = uint64_t(B) * Li * H;
        float* h_acc = (float*)hp;
        float* h_m = (float*)(hp + acc_b);
        float* h_l = (float*)(hp + acc_b + st_b);
        float* h_lt = (float*)(hp + acc_b + 2 * st_b);
        CQSA_HIP(hipStreamWaitEvent(ms, ev_inner[si], 0));
        auto sp = span_begin(ms);
        CQSA_HIP(hipMemcpyAsync(h_acc, a.acc, rows * d * 4, hipMemcpyDeviceToHost, ms));
        CQSA_HIP(hipMemcpyAsync(h_m, a.m, rows * 4, hipMemcpyDeviceToHost, ms));
        CQSA_HIP(hipMemcpyAsync(h_l, a.l, rows * 4, hipMemcpyDeviceToHost, ms));
        CQSA_HIP(hipMemcpyAsync(h_lt, a.lt, rows * 4, hipMemcpyDeviceToHost, ms));
        span_end(sp, ms, kStD2H);
        rec.stats.d2h_bytes += rows * (d + 3) * 4;
        CQSA_HIP(hipEventRecord(ev_free[si], ms));
        const hipEvent_t wait_ev = ev_free[si];
        const Task* tp = &p->tasks[t];
        last_item[si] = merger.push([=, &rec]() -> bool {
          if (hipEventSynchronize(wait_ev) != hipSuccess) return false;
          auto t0 = std::chrono::steady_clock::now();  // the merge alone, not the wait
          host_merge(*tp, h_acc, h_m, h_l, h_lt, acc, m, l, lt, B, L, H, d);
          auto t1 = std::chrono::steady_clock::now();
          rec.host_merge_ms += std::chrono::duration<double, std::milli>(t1 - t0).count();
          return true;
        });
      }
      used[si] = true;
    }
    if (!acc_dev) {
      if (!merger.finish()) return fail(CQSA_ERR_HIP, "host merge: event wait failed");
      auto t0 = std::chrono::steady_clock::now();
      host_finalize(acc, m, l, lt, B, L, H, d);
      auto t1 = std::chrono::steady_clock::now();
      rec.host_final_ms += std::chrono::duration<double, std::milli>(t1 - t0).count();
    }
    // every inner kernel precedes its merge or D2H on the auxiliary stream
    if (ms != st) {
      CQSA_HIP(hipEventRecord(ev_tail, ms));
      CQSA_HIP(hipStreamWaitEvent(st, ev_tail, 0));
    }
  }
  if (o.out16) {
    // O in the input dtype, rounded from the finished fp32 result
    auto sp = span_begin(st);
    CQSA_HIP(launch_cast_out(Od, O->data, B * L * H * d, o.dtype, st));
    span_end(sp, st, kStFinal);
  }
  if (rec.timing) CQSA_HIP(hipEventRecord(rec.wall1, st));
  if (tile_count && (s = tile_counters_end(C, rec, st, 3)) != CQSA_OK) return s;
  CQSA_HIP(hipEventRecord(ws_free, st));
  ws_free_valid = true;
  if (!noalloc) release_workspace(C, &ws, st);
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
    return cqsa::run_guarded(plan, false, [&](const cqsa_plan_t* q) {
      return cqsa::forward_impl(q, Q, K, V, O, LSE, lse_where, scale, (hipStream_t)hip_stream,
                                false);
    });
  } catch (const std::exception& e) {
    return cqsa::fail(CQSA_ERR_INTERNAL, std::string("cqsa_forward: ") + e.what());
  } catch (...) {
    return cqsa::fail(CQSA_ERR_INTERNAL, "cqsa_forward: unknown exception");
  }
}

extern "C" cqsa_status cqsa_forward_noalloc(const cqsa_plan_t* plan, const cqsa_tensor* Q,
                                            const cqsa_tensor* K, const cqsa_tensor* V,
                                            cqsa_tensor* O, float* LSE, cqsa_mem lse_where,
                                            float scale, void* hip_stream) {
  cqsa::clear_error();
  try {
    // no guardrail: nothing is allocated, so nothing can run out of memory
    return cqsa::forward_impl(plan, Q, K, V, O, LSE, lse_where, scale, (hipStream_t)hip_stream,
                              true);
  } catch (const std::exception& e) {
    return cqsa::fail(CQSA_ERR_INTERNAL, std::string("cqsa_forward_noalloc: ") + e.what());
  } catch (...) {
    return cqsa::fail(CQSA_ERR_INTERNAL, "cqsa_forward_noalloc: unknown exception");
  }
}
