// Recomposition kernels (App. A.1): initialise the global accumulator, merge
// one task's (acc_i, l_i, m_i) into it with the max-shifted rule of Eq.
// "merge", and finalise O = acc / l, LSE = m + log l.
//
// Statistics are kept in the log2 domain with integer-valued maxima (the
// inner kernels round running maxima up to integers), so both rescale factors
// e^{m-m'} and e^{m_i-m'} are exact powers of two.  A task row with no kept
// key carries m_i = -inf and is skipped as a null contribution.
//
// All passes are HBM-bound and walk rows of d contiguous floats with 16-byte
// accesses; each work group owns (batch, head, 32 consecutive local rows) and
// resolves local -> global rows through the task's runs.
#include <algorithm>

#include "hip_common.hpp"
#include "kernels.hpp"

namespace cqsa {

__global__ void __launch_bounds__(256) acc_init_kernel(float* acc, float* m, float* l,
                                                       int64_t n_acc4, int64_t n_stat) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_acc4; i += stride)
    ((f32x4*)acc)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n_stat; i += stride) {
    m[i] = -INFINITY;
    l[i] = 0.f;
  }
}

template <int D>
__global__ void __launch_bounds__(256) recompose_kernel(const MergeArgs a) {
  constexpr int ROWS = 32, TPR = 8, FPT = D / TPR;  // threads per row, floats per thread
  __shared__ DevRun runs_s[kMaxRuns];
  const int tid = threadIdx.x;
  for (int i = tid; i < a.n_runs; i += 256) runs_s[i] = ((const DevRun*)a.runs)[i];
  __syncthreads();
  const int64_t nchunk = (a.Li + ROWS - 1) / ROWS;
  const int64_t w = blockIdx.x;
  const int64_t chunk = w % nchunk;
  const int h = int((w / nchunk) % a.H);
  const int b = int(w / (nchunk * a.H));
  const int64_t r = chunk * ROWS + tid / TPR;
  if (r >= a.Li) return;
  int64_t g = -1;
  for (int i = 0; i < a.n_runs; ++i)
    if (r < runs_s[i].local_start + runs_s[i].length) {
      g = runs_s[i].global_start + (r - runs_s[i].local_start);
      break;
    }
  if (g < 0) return;
  const int64_t si = (int64_t(b) * a.H + h) * a.Li + r;
  const int64_t gi = (int64_t(b) * a.H + h) * a.L + g;
  const float mi = a.m_i[si];
  if (mi == -INFINITY) return;  // null contribution
  const float mo = a.m[gi];
  const float mn = fmaxf(mo, mi);
  const float fo = mo == -INFINITY ? 0.f : fast_exp2(mo - mn);
  const float fi = fast_exp2(mi - mn);
  const int64_t rs = int64_t(a.H) * D;
  const float* src = a.acc_i + (int64_t(b) * a.Li + r) * rs + int64_t(h) * D + (tid % TPR) * FPT;
  float* dst = a.acc + (int64_t(b) * a.L + g) * rs + int64_t(h) * D + (tid % TPR) * FPT;
#pragma unroll
  for (int i = 0; i < FPT; i += 4) {
    const f32x4 x = *(const f32x4*)(src + i);
    f32x4 y = *(const f32x4*)(dst + i);
    y = y * fo + x * fi;
    *(f32x4*)(dst + i) = y;
  }
  if (tid % TPR == 0) {
    a.l[gi] = a.l[gi] * fo + a.l_i[si] * fi;
    a.m[gi] = mn;
  }
}

template <int D>
__global__ void __launch_bounds__(256) finalize_kernel(float* acc, float* m, const float* l,
                                                       int64_t B, int64_t L, int64_t H) {
  constexpr int ROWS = 32, TPR = 8, FPT = D / TPR;
  const int tid = threadIdx.x;
  const int64_t nchunk = (L + ROWS - 1) / ROWS;
  const int64_t w = blockIdx.x;
  const int64_t chunk = w % nchunk;
  const int64_t h = (w / nchunk) % H;
  const int64_t b = w / (nchunk * H);
  const int64_t r = chunk * ROWS + tid / TPR;
  if (r >= L) return;
  const int64_t si = (b * H + h) * L + r;
  const float ll = l[si];
  const float inv = 1.f / ll;
  float* p = acc + (b * L + r) * H * D + h * D + (tid % TPR) * FPT;
#pragma unroll
  for (int i = 0; i < FPT; i += 4) {
    f32x4 y = *(f32x4*)(p + i);
    *(f32x4*)(p + i) = y * inv;
  }
  if (tid % TPR == 0) m[si] = (m[si] + __log2f(ll)) * 0.69314718055994530942f;
}

hipError_t launch_acc_init(float* acc, float* m, float* l, int64_t n_acc, int64_t n_stat,
                           hipStream_t s) {
  const int64_t n4 = n_acc / 4;
  int64_t blocks = (std::max(n4, n_stat) + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(acc_init_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, acc, m, l, n4,
                     n_stat);
  return hipGetLastError();
}

hipError_t launch_recompose(const MergeArgs& a, hipStream_t s) {
  if (a.n_runs > kMaxRuns) return hipErrorInvalidValue;
  const int64_t n = ((a.Li + 31) / 32) * int64_t(a.H) * a.B;
  if (n == 0) return hipSuccess;
  if (a.d == 128)
    hipLaunchKernelGGL(recompose_kernel<128>, dim3(unsigned(n)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(recompose_kernel<64>, dim3(unsigned(n)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_finalize(float* acc, float* m, const float* l, int64_t B, int64_t L, int64_t H,
                           int d, hipStream_t s) {
  const int64_t n = ((L + 31) / 32) * H * B;
  if (n == 0) return hipSuccess;
  if (d == 128)
    hipLaunchKernelGGL(finalize_kernel<128>, dim3(unsigned(n)), dim3(256), 0, s, acc, m, l, B, L, H);
  else
    hipLaunchKernelGGL(finalize_kernel<64>, dim3(unsigned(n)), dim3(256), 0, s, acc, m, l, B, L, H);
  return hipGetLastError();
}

}  // namespace cqsa
