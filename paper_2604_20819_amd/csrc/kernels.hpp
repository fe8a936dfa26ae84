// Host-visible kernel launch interface (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cqsa.h"
#include "records.hpp"

namespace cqsa {

// Epilogue of the inner forward kernel.
enum FwdMode : int {
  kModeStats = 0,  // write task-local (acc_i, m_i, l_i, lt_i) for recomposition
  kModeFinal = 1,  // single task covering all tokens: write O = acc/lt and LSE
};

// One launch of the inner forward kernel over `ntask` tasks (a launch group).
// Staged inputs: task j's rows are [B, L_j, H, d] at q/k/v + j * in_stride
// elements.  Inputs read in place (in_place = 1): q/k/v are the caller's
// [B, Lg, H, d] tensors and task j's local token t is the global row its runs
// give (the block rows of DevTask::sum_off).  Task j's statistics are acc_j
// [B, L_j, H, d] at acc + j * acc_stride, m_j, l_j and lt_j [B, H, L_j] at
// m/l/lt + j * st_stride.  l sums the fp32 weights exp2(s - m) and gives the
// log-sum-exp; lt sums the same weights rounded to the input dtype, exactly
// the values the P.V product consumes, and normalises O (equal to l for fp32
// inputs).  In final mode the single task spans all L tokens: q/k/v are the
// caller's tensors, acc is O and m is LSE.
struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  int64_t in_stride;
  float* acc;
  float* m;             // log2 domain (stats) or natural-log LSE (final)
  float* l;             // stats only
  float* lt;            // stats only
  int64_t acc_stride, st_stride;
  const char* tab;      // packed plan image (DevTask offsets are relative to it)
  const DevTask* tasks; // the launch's tasks
  int32_t ntask;
  int32_t B, H;
  int32_t causal;
  float scale_log2;     // softmax scale * log2(e)
  int32_t in_place;     // 1: q/k/v are the caller's tensors, rows by the runs
  int64_t Lg;           // rows per batch element of q/k/v when in_place
  // when not null, each wave adds its tile decisions over the key tiles its
  // work group visits: [0] masked for the wave (skipped), [1] clear, [2]
  // mixed (16-bit kernels, launched as their counting instance; waves with
  // no query of the task add nothing)
  unsigned long long* tile_count;
};

// Gather-merge of one launch group's task statistics into the global
// accumulator (App. A.1, Eq. "merge"), fused with the finalisation
// O = acc / lt, LSE = m + log l when the group is the last one (l and lt are
// merged with the same factors; FwdArgs says what each sums).
struct CombineArgs {
  const DevSeg* segs;        // the group's segments, ascending blk0
  int32_t n_seg;
  const DevContrib* contribs;
  const DevTask* tasks;      // the group's tasks (for L_j)
  const float* acc_i;        // task j's statistics at + j * acc_stride / st_stride
  const float* m_i;
  const float* l_i;
  const float* lt_i;
  int64_t acc_stride, st_stride;
  float* acc;                // [B, L, H, d] running acc, or O when final
  float* m;                  // [B, H, L] running max (log2), or LSE when final
  float* l;                  // [B, H, L] running sum of the fp32 weights
  float* lt;                 // [B, H, L] running sum of the rounded weights
  int64_t L;
  int32_t B, H, d;
  int32_t final;
};

// Inner backward kernels over the tasks of one launch (App. A.1, Eq.
// "globallse").  Work groups take the tasks' strips in task order (task j's
// strips precede task j + 1's), and each reads its task's runs, summaries,
// block rows and strip order from the plan image through its DevTask record.
struct BwdArgs {
  const void* q;        // [B, L, H, d] staged rows of the launch's single task, or,
  const void* k;        // when in_place, the caller's [B, Lg, H, d] tensors with
  const void* v;        // local token t of a task at the global row its runs give
  const void* dO;
  int32_t in_place;
  const char* tab;      // packed plan image (DevTask offsets are relative to it)
  const DevTask* tasks; // the launch's tasks
  int32_t ntask;
  int32_t B, H;
  int32_t causal;
  float scale_log2;     // softmax scale * log2(e)
  float scale;          // softmax scale (dQ = scale dS K, dK = scale dS^T Q)
  const float* lse;     // [B, H, Lg] global natural-log LSE from the forward
  const float* D;       // [B, H, Lg] global rowsum(dO * O)
  int64_t Lg;           // global sequence length
  int32_t local_out;    // 0: dq/dk/dv are the global [B, Lg, H, d] fp32 gradients and
                        //    the (single) task's rows are added at their global rows;
                        // 1: task j's own [B, L_j, H, d] fp32 buffers sit at
                        //    dq/dk/dv + j * out_stride and its rows are stored at
                        //    their local rows
  int64_t out_stride;   // elements
  float* dq;
  float* dk;
  float* dv;
  // when not null, the launches run their counting instances: each dQ wave
  // adds its tile decisions over the key tiles its work group visits to
  // [0] masked, [1] clear, [2] mixed, each dK/dV key group its decisions over
  // the query tiles its work group visits to [3], [4], [5]
  unsigned long long* tile_count;
};

// Gather-merge of one launch group's task-local gradients (task j's at
// + j * stride) into the global fp32 dQ, dK, dV: every token's rows are the
// sum of its contributions in task order, added to the running value when an
// earlier group touched the token.
struct GradMergeArgs {
  const DevSeg* segs;   // the group's segments, ascending blk0
  int32_t n_seg;
  const DevContrib* contribs;
  const DevTask* tasks; // the group's tasks (for L_j)
  const float* src[3];  // task-local dq, dk, dv of the group's first task
  int64_t stride;       // elements between consecutive tasks' buffers
  float* dst[3];        // global [B, L, H, d] dQ, dK, dV
  int64_t L;
  int32_t B, H, d;
};

// Copy the rows of a task's runs from up to four [B, Lg, H, d] tensors into
// task-local [B, Li, H, d] staging buffers (device to device).
struct StageArgs {
  const void* src[4];
  void* dst[4];
  int32_t n_tensors;
  int64_t row_bytes;    // H * d * elem
  int64_t Li, Lg;
  int32_t B;
  const void* runs;     // DevRun[n_runs]
  int32_t n_runs;
};

// `wgs` = total work groups: sum over the tasks of ceil(L_j / rows) * B * H with
// rows = fwd_rows_per_wg(dtype, d).
hipError_t launch_fwd(cqsa_dtype dt, int d, FwdMode mode, const FwdArgs& a, int64_t wgs,
                      hipStream_t s);
int fwd_rows_per_wg(cqsa_dtype dt, int d);
// `blocks` = combine work groups per batch element (the group's last segment's
// blk0 plus its block count).
hipError_t launch_combine(const CombineArgs& a, int64_t blocks, hipStream_t s);
hipError_t launch_stage(const StageArgs& a, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);
// dst[i] = src[i] rounded to the 16-bit dtype `dt` (nearest even), i < n.
hipError_t launch_cast_out(const float* src, void* dst, int64_t n, cqsa_dtype dt, hipStream_t s);
// Zeroes n 64-bit counters (a kernel, not a memset, so that the call stays
// free of memset nodes).
hipError_t launch_zero_u64(unsigned long long* p, int n, hipStream_t s);
// D[(b * H + h) * ld + g] = sum_d dO * O over rows g < L of B batch elements
// of [B, L, H, d] inputs (ld = L for whole tensors; a chunk of rows passes
// its first output and the full sequence length).
hipError_t launch_bwd_preprocess(const void* dO, const float* O, float* D, cqsa_dtype dt,
                                 int64_t B, int64_t L, int64_t H, int d, int64_t ld,
                                 hipStream_t s);
// `wgs` = total work groups: sum over the launch's tasks of
// ceil(L_j / rows) * B * H with rows = dkdv_rows_per_wg(d) (dK/dV) or
// dq_rows_per_wg(d) (dQ).
hipError_t launch_bwd_dkdv(cqsa_dtype dt, int d, const BwdArgs& a, int64_t wgs, hipStream_t s);
hipError_t launch_bwd_dq(cqsa_dtype dt, int d, const BwdArgs& a, int64_t wgs, hipStream_t s);
// `blocks` as for launch_combine.
hipError_t launch_grad_merge(const GradMergeArgs& a, int64_t blocks, hipStream_t s);

}  // namespace cqsa
