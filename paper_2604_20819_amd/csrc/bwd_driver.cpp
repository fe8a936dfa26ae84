// cqsa_backward: decomposed backward in the global-LSE form (App. A.1,
// Eq. "globallse"), equal to Alg. 2.
//
// caller stream : D = rowsum(dO * O) over the full sequence, zero dQ/dK/dV;
//                 per task wait "staged", run the key-parallel dK/dV kernel,
//                 which adds the task's rows into the global fp32 dK and dV;
// second stream : per task the query-parallel dQ kernel, adding into dQ.
//                 Each stream keeps the tasks in order and a task holds each
//                 token once, so these read-modify-writes never race;
// copy stream   : gather each task's runs of Q, K, V, dO into slot t % S once
//                 both kernels of the slot's previous task are done (staged
//                 plans only: a plan that reads its inputs in place passes
//                 the caller's tensors and the task's block row table).
// Depth 0 reads the caller's tensors in place (the undecomposed backward).
#include <algorithm>
#include <cmath>

#include "guard.hpp"
#include "kernels.hpp"
#include "runtime.hpp"

namespace cqsa {

cqsa_status backward_impl(const cqsa_plan_t* p, const cqsa_tensor* Q, const cqsa_tensor* K,
                          const cqsa_tensor* V, const cqsa_tensor* O, const float* LSE,
                          cqsa_mem lse_where, const cqsa_tensor* dO, cqsa_tensor* dQ,
                          cqsa_tensor* dK, cqsa_tensor* dV, float scale, hipStream_t st) {
  if (!p) return fail(CQSA_ERR_INVALID_ARG, "cqsa_backward: plan is NULL");
  const cqsa_plan_opts& o = p->opts;
  if (!o.inputs_on_device || !o.acc_on_device)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: device-resident plans only");
  if (o.dtype == CQSA_F32)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: fp16 and bf16 inputs only");
  if (p->g.d % 32 != 0 || p->g.d > 256)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_backward: head dims 32, 64, ..., 256 only");
  if (!o.with_backward && p->budget != 0)
    return fail(CQSA_ERR_INVALID_ARG,
                "cqsa_backward: the plan's budget was fitted without the backward "
                "(plan with with_backward = 1)");
  cqsa_status s;
  const cqsa_mem dev = CQSA_MEM_DEVICE;
  if ((s = check_tensor(Q, "Q", p, o.dtype, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(K, "K", p, o.dtype, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(V, "V", p, o.dtype, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(dO, "dO", p, o.dtype, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(O, "O", p, CQSA_F32, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(dQ, "dQ", p, CQSA_F32, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(dK, "dK", p, CQSA_F32, dev)) != CQSA_OK) return s;
  if ((s = check_tensor(dV, "dV", p, CQSA_F32, dev)) != CQSA_OK) return s;
  if (!LSE) return fail(CQSA_ERR_INVALID_ARG, "LSE is NULL");
  if (lse_where != CQSA_MEM_DEVICE) return fail(CQSA_ERR_INVALID_ARG, "LSE must be on the device");

  DevCtx* C = device_ctx(&s);
  if (!C) return s;
  std::lock_guard<std::mutex> lock(C->mu);

  const int64_t B = o.B, L = p->g.L, H = p->g.H, d = p->g.d;
  const size_t elem = dtype_size(o.dtype);
  const int64_t row_bytes = int64_t(H) * d * int64_t(elem);
  const float sc = scale > 0.f ? scale : float(1.0 / std::sqrt(double(d)));
  const int depth = p->depth;
  const int64_t ntask = int64_t(p->tasks.size());
  const bool direct = depth == 0;
  // kernels address the runs inside the caller's tensors: nothing is staged
  const bool in_place = !direct && o.read_in_place == 1;
  const bool staged = !direct && !in_place;

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

  const uint64_t tab_bytes = align_up(p->packed.size());
  const uint64_t d_bytes = align_up(uint64_t(B) * H * L * 4);
  const uint64_t slot_bytes = bwd_slot_bytes(p->g, o, p->max_L_local, staged);
  const int64_t nslot = std::min<int64_t>(o.n_slots, std::max<int64_t>(1, ntask));
  const uint64_t total = tab_bytes + d_bytes + uint64_t(nslot) * slot_bytes;
  Workspace ws;
  if ((s = acquire_workspace(C, total, &ws)) != CQSA_OK) return s;
  rec.stats.workspace_bytes = total;
  rec.stats.resident_tasks = staged ? nslot : 0;
  char* base = (char*)ws.ptr;
  char* d_tab = base;
  float* d_D = (float*)(base + tab_bytes);
  const uint64_t in_b = align_up(uint64_t(B) * p->max_L_local * H * d * elem);

  while (C->sync_events.size() < size_t(4 * nslot + 3)) {
    hipEvent_t e;
    CQSA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    C->sync_events.push_back(e);
  }
  hipEvent_t ev_start = C->sync_events[0];
  hipEvent_t ev_tab = C->sync_events[1];
  hipEvent_t* ev_staged = &C->sync_events[2];
  hipEvent_t* ev_free = &C->sync_events[2 + nslot];      // dK/dV kernel done with the slot
  hipEvent_t* ev_free_q = &C->sync_events[2 + 2 * nslot]; // dQ kernel done with the slot
  hipEvent_t ev_pre = C->sync_events[2 + 3 * nslot];      // preprocess and zero fill done
  if (C->ws_free_valid) CQSA_HIP(hipStreamWaitEvent(st, C->ws_free, 0));
  CQSA_HIP(hipEventRecord(ev_start, st));
  CQSA_HIP(hipStreamWaitEvent(C->copy, ev_start, 0));
  if ((s = upload_image(C, p->packed, d_tab, C->copy)) != CQSA_OK) return s;
  CQSA_HIP(hipEventRecord(ev_tab, C->copy));

  // preprocess and zero-fill on the caller's stream
  std::pair<hipEvent_t, hipEvent_t> sp{nullptr, nullptr};
  if (rec.timing) {
    sp = {rec.make(), rec.make()};
    CQSA_HIP(hipEventRecord(sp.first, st));
  }
  CQSA_HIP(launch_bwd_preprocess(dO->data, (const float*)O->data, d_D, o.dtype, B, L, H, int(d), st));
  if (rec.timing) {
    CQSA_HIP(hipEventRecord(sp.second, st));
    rec.spans[kStFinal].push_back(sp);
    sp = {rec.make(), rec.make()};
    CQSA_HIP(hipEventRecord(sp.first, st));
  }
  // the fused scatter-adds accumulate into zeroed gradients
  CQSA_HIP(launch_fill_zero((float*)dQ->data, B * L * H * d, st));
  CQSA_HIP(launch_fill_zero((float*)dK->data, B * L * H * d, st));
  CQSA_HIP(launch_fill_zero((float*)dV->data, B * L * H * d, st));
  if (rec.timing) {
    CQSA_HIP(hipEventRecord(sp.second, st));
    rec.spans[kStMerge].push_back(sp);
  }
  CQSA_HIP(hipStreamWaitEvent(st, ev_tab, 0));
  // dQ kernels run on the second compute stream (they write dQ only, the dK/dV
  // kernels on the caller's stream write dK and dV only): a task's two kernels
  // overlap, and each stream keeps its own tasks in order.
  const hipStream_t qs = C->lane;
  CQSA_HIP(hipEventRecord(ev_pre, st));
  CQSA_HIP(hipStreamWaitEvent(qs, ev_pre, 0));

  std::vector<bool> used(nslot, false);
  for (int64_t t = 0; t < ntask; ++t) {
    const Task& task = p->tasks[t];
    const int64_t Li = task.L_local;
    if (Li == 0) continue;
    const int64_t si = t % nslot;
    const TableOffsets& to = p->table_off[t];
    char* sb = base + tab_bytes + d_bytes + uint64_t(si) * slot_bytes;
    BwdArgs a{};
    if (!staged) {
      a.q = Q->data; a.k = K->data; a.v = V->data; a.dO = dO->data;
      a.in_place = in_place ? 1 : 0;
      a.rows = (const int32_t*)(d_tab + to.rows);
    } else {
      if (used[si]) {
        CQSA_HIP(hipStreamWaitEvent(C->copy, ev_free[si], 0));
        CQSA_HIP(hipStreamWaitEvent(C->copy, ev_free_q[si], 0));
      }
      StageArgs sa{};
      sa.src[0] = Q->data; sa.src[1] = K->data; sa.src[2] = V->data; sa.src[3] = dO->data;
      for (int x = 0; x < 4; ++x) sa.dst[x] = sb + x * in_b;
      sa.n_tensors = 4; sa.row_bytes = row_bytes; sa.Li = Li; sa.Lg = L; sa.B = int32_t(B);
      sa.runs = d_tab + to.runs; sa.n_runs = int32_t(task.runs.size());
      if (rec.timing) {
        sp = {rec.make(), rec.make()};
        CQSA_HIP(hipEventRecord(sp.first, C->copy));
      }
      CQSA_HIP(launch_stage(sa, C->copy));
      rec.stats.d2d_bytes += uint64_t(4) * B * Li * row_bytes;
      if (rec.timing) {
        CQSA_HIP(hipEventRecord(sp.second, C->copy));
        rec.spans[kStStage].push_back(sp);
      }
      CQSA_HIP(hipEventRecord(ev_staged[si], C->copy));
      CQSA_HIP(hipStreamWaitEvent(st, ev_staged[si], 0));
      CQSA_HIP(hipStreamWaitEvent(qs, ev_staged[si], 0));
      a.q = sa.dst[0]; a.k = sa.dst[1]; a.v = sa.dst[2]; a.dO = sa.dst[3];
    }
    a.L = int32_t(Li); a.B = int32_t(B); a.H = int32_t(H); a.causal = p->g.causal;
    a.scale_log2 = sc * 1.4426950408889634f; a.scale = sc;
    a.runs = d_tab + to.runs; a.n_runs = int32_t(task.runs.size());
    a.qorder = (const int32_t*)(d_tab + to.dqorder);
    a.korder = (const int32_t*)(d_tab + to.korder);
    a.blk_or = (const uint32_t*)(d_tab + to.blk_or);
    a.blk_and = (const uint32_t*)(d_tab + to.blk_and);
    a.lse = LSE; a.D = d_D; a.Lg = L;
    a.dq = (float*)dQ->data; a.dk = (float*)dK->data; a.dv = (float*)dV->data;
    std::pair<hipEvent_t, hipEvent_t> sk{nullptr, nullptr}, sq{nullptr, nullptr};
    if (rec.timing) {
      sk = {rec.make(), rec.make()};
      sq = {rec.make(), rec.make()};
      CQSA_HIP(hipEventRecord(sk.first, st));
      CQSA_HIP(hipEventRecord(sq.first, qs));
    }
    CQSA_HIP(launch_bwd_dkdv(o.dtype, int(d), a, st));
    CQSA_HIP(launch_bwd_dq(o.dtype, int(d), a, qs));
    rec.stats.inner_launches += 2;
    if (rec.timing) {
      CQSA_HIP(hipEventRecord(sk.second, st));
      CQSA_HIP(hipEventRecord(sq.second, qs));
      rec.spans[kStInner].push_back(sk);
      rec.spans[kStInner].push_back(sq);
    }
    if (staged) {
      CQSA_HIP(hipEventRecord(ev_free[si], st));
      CQSA_HIP(hipEventRecord(ev_free_q[si], qs));
    }
    used[si] = true;
  }
  // join the dQ stream back into the caller's stream
  CQSA_HIP(hipEventRecord(ev_pre, qs));
  CQSA_HIP(hipStreamWaitEvent(st, ev_pre, 0));
  if (rec.timing) CQSA_HIP(hipEventRecord(rec.wall1, st));
  CQSA_HIP(hipEventRecord(C->ws_free, st));
  C->ws_free_valid = true;
  release_workspace(C, &ws, st);
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
