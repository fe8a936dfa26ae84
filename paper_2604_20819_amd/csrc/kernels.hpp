// Host-visible kernel launch interface (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cqsa.h"

namespace cqsa {

constexpr int kMaxRuns = 128;  // runs per task the kernels accept (l**depth bound)

// Epilogue of the inner forward kernel.
enum FwdMode : int {
  kModeStats = 0,  // write task-local (acc_i, m_i, l_i) for recomposition
  kModeFinal = 1,  // single task covering all tokens: write O = acc/l and LSE
};

struct FwdArgs {
  const void* q;        // [B, seq_rows, H, d] input rows (staged slot or caller tensor)
  const void* k;
  const void* v;
  int64_t seq_rows;     // rows per batch element in q/k/v
  int64_t row0;         // first row of the task in q/k/v
  int32_t L;            // task length
  int32_t B, H;
  int32_t causal;
  float scale_log2;     // softmax scale * log2(e)
  const void* runs;     // DevRun[n_runs], task-local
  int32_t n_runs;
  const uint32_t* blk_or;   // per 64-token block
  const uint32_t* blk_and;
  float* acc;           // stats: [B, L, H, d]; final: O [B, out_rows, H, d]
  float* m;             // stats: [B, H, L] (log2 domain); final: LSE [B, H, out_rows]
  float* l;             // stats: [B, H, L]; final: unused
  int64_t out_rows;
};

// Recompose one task's statistics into the global accumulator (device).
struct MergeArgs {
  const float* acc_i;   // [B, Li, H, d]
  const float* m_i;     // [B, H, Li] log2 domain
  const float* l_i;     // [B, H, Li]
  float* acc;           // [B, L, H, d]  (the O buffer)
  float* m;             // [B, H, L]     (the LSE buffer, log2 domain until finalize)
  float* l;             // [B, H, L]
  const void* runs;     // DevRun[n_runs]
  int32_t n_runs;
  int64_t Li, L;
  int32_t B, H, d;
};

// Inner backward kernels over one staged task (App. A.1, Eq. "globallse").
struct BwdArgs {
  const void* q;        // [B, L, H, d] staged task rows (seq_rows = L)
  const void* k;
  const void* v;
  const void* dO;
  int32_t L;            // task length
  int32_t B, H;
  int32_t causal;
  float scale_log2;     // softmax scale * log2(e)
  float scale;          // softmax scale (dQ = scale dS K, dK = scale dS^T Q)
  const void* runs;     // DevRun[n_runs]
  int32_t n_runs;
  const uint32_t* blk_or;
  const uint32_t* blk_and;
  const float* lse;     // [B, H, Lg] global natural-log LSE from the forward
  const float* D;       // [B, H, Lg] global rowsum(dO * O)
  int64_t Lg;           // global sequence length
  float* dq;            // [B, Lg, H, d] global fp32 gradients (scatter-added)
  float* dk;
  float* dv;
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

hipError_t launch_fwd(cqsa_dtype dt, int d, FwdMode mode, const FwdArgs& a, hipStream_t s);
hipError_t launch_acc_init(float* acc, float* m, float* l, int64_t n_acc, int64_t n_stat,
                           hipStream_t s);
hipError_t launch_recompose(const MergeArgs& a, hipStream_t s);
hipError_t launch_stage(const StageArgs& a, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);
hipError_t launch_bwd_preprocess(const void* dO, const float* O, float* D, cqsa_dtype dt,
                                 int64_t B, int64_t L, int64_t H, int d, hipStream_t s);
hipError_t launch_bwd_dkdv(cqsa_dtype dt, int d, const BwdArgs& a, hipStream_t s);
hipError_t launch_bwd_dq(cqsa_dtype dt, int d, const BwdArgs& a, hipStream_t s);
hipError_t launch_finalize(float* acc, float* m, const float* l, int64_t B, int64_t L, int64_t H,
                           int d, hipStream_t s);

}  // namespace cqsa
