// HBM-bound helper kernels: task staging (gather of a task's runs), zero
// fill, and the backward preprocess D = rowsum(dO * O).
#include "hip_common.hpp"
#include "kernels.hpp"

namespace cqsa {

// One (tensor, batch, run) span per blockIdx.y; blockIdx.x strides over its
// 16-byte chunks.  A run is contiguous in both the global tensor and the
// task-local buffer, so every span is a straight copy.
__global__ void __launch_bounds__(256) stage_kernel(const StageArgs a) {
  const int span = blockIdx.y;
  const int run = span % a.n_runs;
  const int b = (span / a.n_runs) % a.B;
  const int t = span / (a.n_runs * a.B);
  const DevRun r = ((const DevRun*)a.runs)[run];
  const char* src = (const char*)a.src[t] + (int64_t(b) * a.Lg + r.global_start) * a.row_bytes;
  char* dst = (char*)a.dst[t] + (int64_t(b) * a.Li + r.local_start) * a.row_bytes;
  const int64_t n16 = r.length * a.row_bytes / 16;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
    ((u32x4*)dst)[i] = ((const u32x4*)src)[i];
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float* p, int64_t n4) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n4; i += stride)
    ((f32x4*)p)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// D[b, h, g] = sum_d dO[b, g, h, d] * O[b, g, h, d]; 16 lanes per (b, g, h);
// output row stride ld.
template <typename T, int D>
__global__ void __launch_bounds__(256) preprocess_kernel(const T* dO, const float* O, float* Dout,
                                                         int64_t B, int64_t L, int64_t H,
                                                         int64_t ld) {
  constexpr int EPL = D / 16;  // elements per lane
  const int64_t row = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / 16;
  const int sub = threadIdx.x & 15;
  const bool ok = row < B * L * H;
  float acc = 0.f;
  if (ok) {
    const T* x = dO + row * D + sub * EPL;
    const float* y = O + row * D + sub * EPL;
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc += float(x[i]) * y[i];
  }
  acc += __shfl_xor(acc, 1);
  acc += __shfl_xor(acc, 2);
  acc += __shfl_xor(acc, 4);
  acc += __shfl_xor(acc, 8);
  if (ok && sub == 0) {
    const int64_t h = row % H, g = (row / H) % L, b = row / (H * L);
    Dout[(b * H + h) * ld + g] = acc;
  }
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s) {
  if (a.n_runs <= 0 || a.Li == 0) return hipSuccess;
  const unsigned ny = unsigned(a.n_tensors * a.B * a.n_runs);
  // enough blocks per span to cover the longest run in a few strides
  hipLaunchKernelGGL(stage_kernel, dim3(64, ny), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
  const int64_t n4 = n / 4;
  int64_t blocks = (n4 + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, p, n4);
  return hipGetLastError();
}

hipError_t launch_bwd_preprocess(const void* dO, const float* O, float* D, cqsa_dtype dt,
                                 int64_t B, int64_t L, int64_t H, int d, int64_t ld,
                                 hipStream_t s) {
  const int64_t rows = B * L * H;
  const unsigned blocks = unsigned((rows * 16 + 255) / 256);
  if (rows == 0) return hipSuccess;
  switch (d) {
#define CQSA_PRE_D(DD)                                                                   \
  case DD:                                                                               \
    if (dt == CQSA_BF16)                                                                 \
      hipLaunchKernelGGL((preprocess_kernel<__bf16, DD>), dim3(blocks), dim3(256), 0, s, \
                         (const __bf16*)dO, O, D, B, L, H, ld);                              \
    else if (dt == CQSA_F16)                                                             \
      hipLaunchKernelGGL((preprocess_kernel<_Float16, DD>), dim3(blocks), dim3(256), 0,  \
                         s, (const _Float16*)dO, O, D, B, L, H, ld);                         \
    else                                                                                 \
      return hipErrorInvalidValue;                                                       \
    break;
    CQSA_PRE_D(32)
    CQSA_PRE_D(64)
    CQSA_PRE_D(96)
    CQSA_PRE_D(128)
    CQSA_PRE_D(160)
    CQSA_PRE_D(192)
    CQSA_PRE_D(224)
    CQSA_PRE_D(256)
#undef CQSA_PRE_D
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace cqsa
