// Recomposition (App. A.1): the max-shifted merge of Eq. "merge" of a launch
// group's task statistics (acc_i, m_i, l_i, lt_i) into the global
// accumulator, fused with the finalisation O = acc / lt, LSE = m + log l
// after the last group (l sums the fp32 weights, lt the rounded weights the
// inner kernel's P.V product consumed; both merge with the same factors).
//
// Gather form: every work group owns kCombinePairs consecutive (token, head)
// pairs of one elementary segment and one batch element.  A segment lies
// inside one run of each task that holds it, so each contribution is a
// contiguous slab of the task's statistics; the work group reads every
// contribution (and the running global state when an earlier group touched
// these tokens), merges in registers and writes each output once.  Work
// groups own disjoint tokens, so the merge needs no atomics and no ordering
// between tasks of the group.
//
// Statistics are in the log2 domain with integer-valued maxima (the inner
// kernels round running maxima up to integers), so every factor
// 2^(m_i - m') is an exact power of two.  A task row with no kept key carries
// m_i = -inf and l_i = lt_i = 0: a null contribution with factor 0.
#include "hip_common.hpp"
#include "kernels.hpp"

namespace cqsa {

template <int D>
__global__ void __launch_bounds__(256) combine_kernel(const CombineArgs a) {
  constexpr int P = kCombinePairs;
  constexpr int F4 = D / 4;            // float4 per (token, head)
  constexpr int NF = P * F4 / 256;     // float4 per thread
  static_assert(P * F4 % 256 == 0, "combine tiling");
  __shared__ float fac_s[kMaxContrib + 1][P];
  __shared__ float inv_s[P];

  const int tid = threadIdx.x;
  const int b = blockIdx.y;
  const int64_t blk = blockIdx.x;
  // segment of this work group: the last one with blk0 <= blk
  int lo = 0, hi = a.n_seg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].blk0 <= blk) lo = mid; else hi = mid - 1;
  }
  const DevSeg sg = a.segs[lo];
  const int H = a.H;
  const int64_t pair0 = (blk - sg.blk0) * P;        // first pair within the segment
  const int64_t npair64 = sg.len * H - pair0;
  const int npair = npair64 < P ? int(npair64) : P;
  const int nc = sg.n_c < kMaxContrib ? sg.n_c : kMaxContrib;  // the planner caps n_c
  const bool glob = sg.has_global != 0;

  // merge factors of each pair (one thread per pair)
  if (tid < npair) {
    const int64_t pr = pair0 + tid;
    const int64_t r = pr / H;
    const int h = int(pr % H);
    const int64_t gi = (int64_t(b) * H + h) * a.L + sg.g0 + r;
    float mg = -INFINITY, lg = 0.f, ltg = 0.f;
    if (glob) {
      mg = a.m[gi];
      lg = a.l[gi];
      ltg = a.lt[gi];
    }
    float mx = mg;
    for (int k = 0; k < nc; ++k) {
      const DevContrib c = a.contribs[sg.c_off + k];
      const int64_t Lj = a.tasks[c.j].L_local;
      const float mk = a.m_i[c.j * a.st_stride + (int64_t(b) * H + h) * Lj + c.local_start + r];
      mx = fmaxf(mx, mk);
    }
    const float fg = mg == -INFINITY ? 0.f : fast_exp2(mg - mx);
    float lsum = lg * fg, ltsum = ltg * fg;
    fac_s[0][tid] = fg;
    for (int k = 0; k < nc; ++k) {
      const DevContrib c = a.contribs[sg.c_off + k];
      const int64_t Lj = a.tasks[c.j].L_local;
      const int64_t si = c.j * a.st_stride + (int64_t(b) * H + h) * Lj + c.local_start + r;
      const float mk = a.m_i[si];
      const float f = mk == -INFINITY ? 0.f : fast_exp2(mk - mx);
      lsum += a.l_i[si] * f;
      ltsum += a.lt_i[si] * f;
      fac_s[k + 1][tid] = f;
    }
    if (a.final) {
      inv_s[tid] = 1.f / ltsum;
      a.m[gi] = (mx + __log2f(lsum)) * 0.69314718055994530942f;
    } else {
      inv_s[tid] = 1.f;
      a.m[gi] = mx;
      a.l[gi] = lsum;
      a.lt[gi] = ltsum;
    }
  }
  __syncthreads();

  // stream the (token, head) rows: contiguous in the global tensor and in
  // every contribution, 16 bytes per thread per pass
  const int64_t row_g = (int64_t(b) * a.L + sg.g0) * H;  // pair index of token g0, head 0
  f32x4 acc[NF];
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    const int f = tid + 256 * i, p = f / F4;
    acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (glob && p < npair) {
      const f32x4 x = *(const f32x4*)(a.acc + (row_g + pair0 + p) * D + (f % F4) * 4);
      acc[i] = x * fac_s[0][p];
    }
  }
  for (int k = 0; k < nc; ++k) {
    const DevContrib c = a.contribs[sg.c_off + k];
    const int64_t Lj = a.tasks[c.j].L_local;
    const float* src = a.acc_i + c.j * a.acc_stride +
                       ((int64_t(b) * Lj + c.local_start) * H + pair0) * D;
    f32x4 x[NF];
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int f = tid + 256 * i, p = f / F4;
      x[i] = p < npair ? *(const f32x4*)(src + int64_t(p) * D + (f % F4) * 4)
                       : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int p = (tid + 256 * i) / F4;
      if (p < npair) acc[i] += x[i] * fac_s[k + 1][p];
    }
  }
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    const int f = tid + 256 * i, p = f / F4;
    if (p < npair)
      *(f32x4*)(a.acc + (row_g + pair0 + p) * D + (f % F4) * 4) = acc[i] * inv_s[p];
  }
}

// Gradient recomposition of a launch group: every (token, head) row of dQ,
// dK and dV is the sum of the group's task-local rows that hold the token, in
// task order, added to the running value when an earlier group touched the
// token (task gradients add: each kept pair belongs to one task).  Work
// groups own kCombinePairs consecutive (token, head) pairs of one segment and
// batch element, as in the combine; the rows are contiguous in every buffer,
// 16 bytes per thread per pass.
template <int D>
__global__ void __launch_bounds__(256) grad_merge_kernel(const GradMergeArgs a) {
  constexpr int P = kCombinePairs;
  constexpr int F4 = D / 4;
  constexpr int NF = P * F4 / 256;
  static_assert(P * F4 % 256 == 0, "merge tiling");
  const int tid = threadIdx.x;
  const int b = blockIdx.y;
  const int64_t blk = blockIdx.x;
  int lo = 0, hi = a.n_seg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].blk0 <= blk) lo = mid; else hi = mid - 1;
  }
  const DevSeg sg = a.segs[lo];
  const int H = a.H;
  const int64_t pair0 = (blk - sg.blk0) * P;
  const int64_t npair64 = sg.len * H - pair0;
  const int npair = npair64 < P ? int(npair64) : P;
  const int nc = sg.n_c < kMaxContrib ? sg.n_c : kMaxContrib;
  const bool glob = sg.has_global != 0;
  const int64_t row_g = (int64_t(b) * a.L + sg.g0) * H + pair0;  // first pair's row
#pragma unroll 1
  for (int t = 0; t < 3; ++t) {
    float* dst = a.dst[t] + row_g * D;
    f32x4 acc[NF];
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int f = tid + 256 * i, p = f / F4;
      acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (glob && p < npair) acc[i] = *(const f32x4*)(dst + int64_t(p) * D + (f % F4) * 4);
    }
    for (int k = 0; k < nc; ++k) {
      const DevContrib c = a.contribs[sg.c_off + k];
      const int64_t Lj = a.tasks[c.j].L_local;
      const float* src = a.src[t] + c.j * a.stride + ((int64_t(b) * Lj + c.local_start) * H + pair0) * D;
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int f = tid + 256 * i, p = f / F4;
        if (p < npair) acc[i] += *(const f32x4*)(src + int64_t(p) * D + (f % F4) * 4);
      }
    }
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int f = tid + 256 * i, p = f / F4;
      if (p < npair) *(f32x4*)(dst + int64_t(p) * D + (f % F4) * 4) = acc[i];
    }
  }
}

// fp32 result rounded to a 16-bit output dtype (nearest even): 8 elements
// per thread, one 32-byte read and one 16-byte write.
template <typename T>
__global__ void __launch_bounds__(256) cast_out_kernel(const float* __restrict__ src,
                                                       T* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i + 8 <= n) {
    const f32x4 x0 = *(const f32x4*)(src + i), x1 = *(const f32x4*)(src + i + 4);
    typedef __attribute__((__vector_size__(8 * sizeof(T)))) T t8;
    t8 y;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y[e] = (T)x0[e];
      y[4 + e] = (T)x1[e];
    }
    *(t8*)(dst + i) = y;
  } else {
    for (int64_t k = i; k < n; ++k) dst[k] = (T)src[k];
  }
}

hipError_t launch_cast_out(const float* src, void* dst, int64_t n, cqsa_dtype dt, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 2047) / 2048;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  if (dt == CQSA_BF16)
    hipLaunchKernelGGL(cast_out_kernel<__bf16>, dim3(unsigned(blocks)), dim3(256), 0, s, src,
                       (__bf16*)dst, n);
  else if (dt == CQSA_F16)
    hipLaunchKernelGGL(cast_out_kernel<_Float16>, dim3(unsigned(blocks)), dim3(256), 0, s, src,
                       (_Float16*)dst, n);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int64_t blocks, hipStream_t s) {
  if (blocks <= 0 || a.B <= 0) return hipSuccess;
  if (a.n_seg < 1 || blocks > 0x7fffffff || a.B > 65535) return hipErrorInvalidValue;
  const dim3 grid(unsigned(blocks), unsigned(a.B));
  switch (a.d) {
    case 32: hipLaunchKernelGGL(combine_kernel<32>, grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL(combine_kernel<64>, grid, dim3(256), 0, s, a); break;
    case 96: hipLaunchKernelGGL(combine_kernel<96>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(combine_kernel<128>, grid, dim3(256), 0, s, a); break;
    case 160: hipLaunchKernelGGL(combine_kernel<160>, grid, dim3(256), 0, s, a); break;
    case 192: hipLaunchKernelGGL(combine_kernel<192>, grid, dim3(256), 0, s, a); break;
    case 224: hipLaunchKernelGGL(combine_kernel<224>, grid, dim3(256), 0, s, a); break;
    case 256: hipLaunchKernelGGL(combine_kernel<256>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace cqsa

namespace cqsa {

hipError_t launch_grad_merge(const GradMergeArgs& a, int64_t blocks, hipStream_t s) {
  if (blocks <= 0 || a.B <= 0) return hipSuccess;
  if (a.n_seg < 1 || blocks > 0x7fffffff || a.B > 65535) return hipErrorInvalidValue;
  const dim3 grid(unsigned(blocks), unsigned(a.B));
  switch (a.d) {
    case 32: hipLaunchKernelGGL(grad_merge_kernel<32>, grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL(grad_merge_kernel<64>, grid, dim3(256), 0, s, a); break;
    case 96: hipLaunchKernelGGL(grad_merge_kernel<96>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(grad_merge_kernel<128>, grid, dim3(256), 0, s, a); break;
    case 160: hipLaunchKernelGGL(grad_merge_kernel<160>, grid, dim3(256), 0, s, a); break;
    case 192: hipLaunchKernelGGL(grad_merge_kernel<192>, grid, dim3(256), 0, s, a); break;
    case 224: hipLaunchKernelGGL(grad_merge_kernel<224>, grid, dim3(256), 0, s, a); break;
    case 256: hipLaunchKernelGGL(grad_merge_kernel<256>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

__global__ void __launch_bounds__(64) zero_u64_kernel(unsigned long long* p, int n) {
  const int i = threadIdx.x;
  if (i < n) p[i] = 0ull;
}

hipError_t launch_zero_u64(unsigned long long* p, int n, hipStream_t s) {
  if (n <= 0 || n > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(64), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace cqsa
