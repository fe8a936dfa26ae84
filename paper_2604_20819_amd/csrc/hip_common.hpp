// Device-side building blocks for the gfx950 (CDNA4) kernels.
//
// MFMA lane layouts used throughout (wave64, v_mfma_f32_32x32x16_{bf16,f16}):
//   A (M x K = 32 x 16): lane l holds row l%32, k = 8*(l/32) .. +8
//   B (K x N = 16 x 32): lane l holds column l%32, k = 8*(l/32) .. +8
//   C/D (32 x 32 fp32):  lane l holds column l%32; register r holds row
//                        8*(r/4) + 4*(l/32) + (r%4)
// ds_read_b64_tr_b16 (LDS transpose read), per group of 16 lanes: lane i of
// the group receives element (i%4) of the 4 x 16-bit words read by source
// lane 4*e + i/4, for e = 0..3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace cqsa {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void* lds_ptr;
// Words read through the constant address space: a load at a wave-uniform
// address is then a scalar load (tables that no kernel writes).
typedef const __attribute__((address_space(4))) uint32_t const_u32;

// Input element tags.
struct BF16 {
  typedef bf16x8 vec8;
};
struct F16 {
  typedef f16x8 vec8;
};

template <typename E>
__device__ __forceinline__ f32x16 mfma32(const typename E::vec8& a, const typename E::vec8& b,
                                         const f32x16& c);
template <>
__device__ __forceinline__ f32x16 mfma32<BF16>(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x16 mfma32<F16>(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Convert 8 fp32 values to a packed 16-bit operand (round to nearest even).
template <typename E>
__device__ __forceinline__ typename E::vec8 pack8(const float* x);
template <>
__device__ __forceinline__ bf16x8 pack8<BF16>(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)x[i];
  return r;
}
template <>
__device__ __forceinline__ f16x8 pack8<F16>(const float* x) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (_Float16)x[i];
  return r;
}

// Running sum of the 8 packed 16-bit values of an MFMA operand, as fp32:
// four dot products with (1, 1) (v_dot2c_f32_{bf16,f16}); the products are
// exact, so this adds exactly the rounded values the product consumes.
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
template <typename E>
__device__ __forceinline__ float sum8(const typename E::vec8& x, float acc);
template <>
__device__ __forceinline__ float sum8<BF16>(const bf16x8& x, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 p = {x[2 * i], x[2 * i + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(p, one, acc, false);
  }
  return acc;
}
template <>
__device__ __forceinline__ float sum8<F16>(const f16x8& x, float acc) {
  const f16x2 one = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f16x2 p = {x[2 * i], x[2 * i + 1]};
    acc = __builtin_amdgcn_fdot2(p, one, acc, false);
  }
  return acc;
}

template <typename V>
__device__ __forceinline__ V bitcast_u4(const u32x4& u) {
  return __builtin_bit_cast(V, u);
}

// Two LDS transpose reads forming one 8-element 16-bit MFMA operand.
template <typename E>
__device__ __forceinline__ typename E::vec8 lds_tr_pair(const char* p0, const char* p1) {
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
  u32x4 u;
  u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  u[0] = a[0];
  u[1] = a[1];
  u[2] = b[0];
  u[3] = b[1];
  return __builtin_bit_cast(typename E::vec8, u);
}

// LDS row of a K/V tile: d padded up to 64, 128 or 256 elements, so that a
// row holds at least 8 swizzle slots and a 1 KB direct load covers whole rows.
// The padding chunks are loaded (the neighbouring row's bytes, or zero past
// the buffer range) and never read by a product.
template <int D>
constexpr int lds_row_elems() {
  return D <= 64 ? 64 : (D <= 128 ? 128 : 256);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// a * b rounded to fp32 on its own: the opaque copy keeps the compiler from
// fusing the product into a following addition (an FMA rounds once), so a sum
// of such products is the same whichever code adds them.
__device__ __forceinline__ float mul_rounded(float a, float b) {
  float t = a * b;
  asm volatile("" : "+v"(t));
  return t;
}

// Value held by lane l^32 (the other half of the wave).
__device__ __forceinline__ float swap_halves(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                            __builtin_bit_cast(uint32_t, v), false, false);
  uint32_t lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  return __builtin_bit_cast(float, lane < 32 ? r[1] : r[0]);
}

// Raw buffer resource over `rows` rows of a [.., rows, H, d] tensor starting at
// `base` (row pitch `pitch_elems` 16-bit elements, `d` elements per row).  The
// range ends at the last element of row rows-1, so loads of later rows return
// zero (buffer range check) and every address is an SGPR base plus a 32-bit
// per-lane offset.  The last dword selects the raw (untyped) buffer format.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* base, int64_t rows,
                                                           int64_t pitch_bytes, int64_t row_bytes) {
  int64_t bytes = rows > 0 ? (rows - 1) * pitch_bytes + row_bytes : 0;
  if (bytes > 0x7fffffff) bytes = 0x7fffffff;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

// 16 bytes per lane from a buffer resource straight into LDS: lane i's bytes
// land at lds + 16 i (the wave fills 1 KB); out-of-range reads give zeros.
__device__ __forceinline__ void buf_load16_lds(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, 0,
                                           0, 0);
}

// Work-group barrier after this wave's own LDS reads and writes have
// completed (lgkmcnt(0)) that leaves LDS DMA loads (buffer_load ... lds,
// counted by vmcnt) in flight: the compiler's fences would wait for them.
// The caller waits (vmcnt) for the DMA loads the next phase reads.  The
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier_dma_in_flight() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Work-group barrier that orders LDS only.  __syncthreads() also orders
// global memory, which makes every wave wait for its in-flight global loads
// (the next tile's prefetch) at the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ int lane_id() {
  return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Group bits and global index of a task-local token (runs sorted by local start).
__device__ __forceinline__ uint32_t run_bits(const DevRun* runs, int n, int64_t local) {
  for (int i = 0; i < n; ++i)
    if (local < runs[i].local_start + runs[i].length) return runs[i].bits;
  return 0u;
}
__device__ __forceinline__ int64_t run_global(const DevRun* runs, int n, int64_t local) {
  for (int i = 0; i < n; ++i)
    if (local < runs[i].local_start + runs[i].length)
      return runs[i].global_start + (local - runs[i].local_start);
  return 0;
}

// Tensor row of local token r when the inputs are read in place: from the
// block row table when r's 64-token block lies in one run, else from the runs.
__device__ __forceinline__ int64_t in_place_row(const DevBlock* blks, const DevRun* runs, int n,
                                                int r) {
  const int32_t g = blks[r >> 6].row;
  return g != kNoRow ? int64_t(g) + (r & 63) : run_global(runs, n, r);
}

// Byte offset that every buffer load treats as out of range (resources span
// under 2^31 bytes): such lanes read zero.
constexpr uint32_t kOobOffset = 0x80000000u;

// Task of a work item in a launch over several tasks, whose work items are
// laid out task after task (ceil(L_j / rows) * per_row items for task j).
// Returns j and leaves the item's index within task j in `w`.
__device__ __forceinline__ int find_task(const DevTask* tasks, int ntask, int rows,
                                         int64_t per_row, int64_t& w) {
  int j = 0;
  for (; j < ntask - 1; ++j) {
    const int64_t n = ((tasks[j].L_local + rows - 1) / rows) * per_row;
    if (w < n) break;
    w -= n;
  }
  return j;
}

// Work-group id remapped so that consecutive work items land on the same XCD
// (the dispatcher deals work groups round-robin over the 8 XCDs, each with its
// own L2): work item w = xcd * per_xcd + slot.
__device__ __forceinline__ int64_t xcd_remap(int64_t id, int64_t n) {
  constexpr int64_t kXcd = 8;
  const int64_t per = n / kXcd, rem = n % kXcd;
  const int64_t xcd = id % kXcd, slot = id / kXcd;
  // the first `rem` XCDs own per+1 items
  const int64_t base = xcd * per + (xcd < rem ? xcd : rem);
  const int64_t cap = per + (xcd < rem ? 1 : 0);
  if (slot < cap) return base + slot;
  return id;  // unreachable when the grid has exactly n groups
}

}  // namespace cqsa
