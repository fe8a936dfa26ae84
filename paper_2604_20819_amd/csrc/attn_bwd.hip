// Inner backward kernels over one CQS task, in the global-LSE form of App. A.1
// (Eq. "globallse"): P[q,k] = exp(alpha s[q,k] - lse_global[q]) on the pairs the
// task keeps, D[q] = rowsum(dO * O), dS = P * (dP - D), and
//   dV = P^T dO,  dK = alpha dS^T Q  (key-parallel kernel, 4 products)
//   dQ = alpha dS K                  (query-parallel kernel, 3 products)
// The paper shows this equals Alg. 2; because every (query, key) pair is kept
// by exactly one task, task gradients add.  A launch of one task may add its
// rows straight into the global fp32 gradients (tasks are ordered on one
// stream and a task holds each token once, so no atomics are needed); a
// launch of several tasks stores each task's rows in its own buffer, and a
// gather-merge sums them in task order.
//
// Tile verdicts, masks and ascending-order causal tests follow the forward.
// Fully masked tiles are skipped before any load: a skipped tile leaves
// P = 0 and therefore dS = 0 (App. A.2, "Skipping fully-masked tiles").
//
// gfx950 layouts: the dQ kernel works on S^T (lane = query) like the forward
// and reads K^T operands with ds_read_b64_tr_b16; the dK/dV kernel works on S
// (lane = key), keeps the wave's K rows as register operands and the work
// group's V rows in LDS, and reads dO^T and Q^T operands from row-major LDS
// tiles with the transpose read.
#include "hip_common.hpp"
#include "kernels.hpp"

namespace cqsa {

constexpr float kLog2e = 1.4426950408889634f;

// Waves per dQ work group: 8 over a 256-query strip at d = 96, 128 and 160
// (at 96 and 128 the work group's single slot per CU leaves the LDS for a
// third K/V tile; at 160 the padded LDS rows leave one work group per CU and 4
// waves would run one wave per SIMD, where a 40 B spill costs less); 4 over a
// 128-query strip elsewhere (at 192 and up 8 waves spill more).
template <int D> constexpr int dq_waves() { return (D >= 96 && D <= 160) ? 8 : 4; }

// LOCAL (BwdArgs::local_out) is a template parameter: a run-time branch in
// the epilogue changes the register allocation of the whole kernel (the
// dK/dV kernel at d = 128 then spills).
// COUNT: the launch counts its tile decisions (BwdArgs::tile_count, [0..2]);
// a separate instance, so that the kernel without counting does no counting work
template <typename E, int D, bool LOCAL, bool COUNT>
__global__ void __launch_bounds__(64 * dq_waves<D>(), (lds_row_elems<D>() > 128 ? 1 : 2)) attn_bwd_dq(const BwdArgs a) {
  constexpr int WAVES = dq_waves<D>(), NT = 64 * WAVES;
  constexpr int BM = 32 * WAVES, BN = 64;
  // K and V tiles: rows of DP elements (d padded as in the forward) with the
  // forward's swizzle (chunk ch of row r in slot ch ^ swz(r)), free of bank
  // conflicts for the K and V row reads and the K transpose reads; filled by
  // direct buffer-to-LDS loads (lane i's 16 bytes at +16 i of a 1 KB block).
  constexpr int DP = lds_row_elems<D>();
  constexpr int RB = DP * 2;
  constexpr int KBYTES = BN * RB, VBYTES = BN * RB;
  constexpr int DK = D / 16, DB = D / 32, CHUNKS = DP / 8;
  constexpr int RPI = 64 / CHUNKS, NDMA = BN / RPI / WAVES;
  typedef typename E::vec8 vec8;
  auto swz = [](int r) { return 2 * (r & 3) + ((r >> 2) & 1); };

  // a ring of NBUF key tiles (K, V) filled NBUF - 1 tiles ahead of the
  // compute: three for the 8-wave work groups of unpadded rows, two elsewhere
  constexpr int NBUF = (WAVES == 8 && DP <= 128) ? 3 : 2, AHEAD = NBUF - 1;
  constexpr int TILE_OPS = 2 * NDMA;  // this wave's loads of one tile
  static_assert(NBUF == 2 || TILE_OPS < 16, "vmcnt immediate");
  // each buffer holds the K tile, then the V tile: the V rows lie a constant
  // offset from the K rows, so their reads share address registers
  __shared__ __attribute__((aligned(1024))) char kvst[NBUF][KBYTES + VBYTES];
  // d = 160 and 256: the 16-byte chunk offsets of the LDS reads split into a
  // swizzled low part and an immediate high part (below), which frees the
  // registers that these kernels otherwise spilled; elsewhere it measured
  // neutral or slower, so the plain offsets stay
  constexpr bool SPLIT_OFF = D == 160 || D == 256;
  __shared__ __attribute__((aligned(16))) uint32_t kbits_s[NBUF][BN];
  __shared__ DevRun runs_s[kMaxRuns];

  const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
  // uniform per wave, so per-wave loads and branches stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int64_t work = xcd_remap(blockIdx.x, gridDim.x);
  const int tj = find_task(a.tasks, a.ntask, BM, int64_t(a.H) * a.B, work);
  const DevTask tk = a.tasks[tj];
  const int L = int(tk.L_local);
  const int64_t nstrips = (L + BM - 1) / BM;
  // strips in the task's launch order (most live key tiles first; the plan
  // builds this table for BM-row strips, BM = dq_rows_per_wg)
  const int strip = ((const int32_t*)(a.tab + tk.dqorder_off))[work % nstrips];
  const int h = int((work / nstrips) % a.H);
  const int b = int(work / (nstrips * a.H));
  const int n_runs = tk.n_runs;
  const DevRun* runs_g = (const DevRun*)(a.tab + tk.runs_off);
  const DevBlock* blks = (const DevBlock*)(a.tab + tk.sum_off);
  const bool in_place = a.in_place != 0;
  for (int i = tid; i < n_runs; i += NT) runs_s[i] = runs_g[i];

  // token rows: consecutive when staged, the runs' global rows when the
  // caller's tensors are read in place (as in the forward)
  const int64_t rs = int64_t(a.H) * D;
  const int64_t seq = in_place ? a.Lg : int64_t(L);
  const int64_t base = int64_t(b) * seq * rs + int64_t(h) * D;
  const uint16_t* Qg = (const uint16_t*)a.q + base;
  const uint16_t* Kg = (const uint16_t*)a.k + base;
  const uint16_t* Vg = (const uint16_t*)a.v + base;
  const uint16_t* Og = (const uint16_t*)a.dO + base;
  const float c = a.scale_log2;
  const bool causal = a.causal != 0;

  const int q0w = strip * BM + wave * 32;
  const int myq = q0w + (lane & 31);
  const bool qvalid = myq < L;
  // the wave's 32 queries lie in one 64-token block, so the table lookup and
  // its branch are wave-uniform
  int64_t qrow = myq;
  if (in_place && q0w < L) {
    const int32_t br = blks[q0w >> 6].row;
    qrow = br != kNoRow ? int64_t(br) + (myq & 63) : (qvalid ? run_global(runs_g, n_runs, myq) : 0);
  }
  vec8 qf[DK], of[DK];
#pragma unroll
  for (int ks = 0; ks < DK; ++ks) {
    u32x4 u = {0u, 0u, 0u, 0u}, w = {0u, 0u, 0u, 0u};
    if (qvalid) {
      u = *(const u32x4*)(Qg + qrow * rs + ks * 16 + half * 8);
      w = *(const u32x4*)(Og + qrow * rs + ks * 16 + half * 8);
    }
    qf[ks] = bitcast_u4<vec8>(u);
    of[ks] = bitcast_u4<vec8>(w);
  }

  const int lastq_wg = (strip * BM + BM < L ? strip * BM + BM : L) - 1;
  const int qb0 = strip * (BM / 64), qb1 = lastq_wg / 64;
  uint32_t qor = 0u, qand = 0xFFFFFFFFu;
  for (int qb = qb0; qb <= qb1; ++qb) {
    qor |= blks[qb].bor;
    qand &= blks[qb].band;
  }
  const bool wave_live = q0w < L;
  const int wq1 = wave_live ? (q0w + 31 < L ? q0w + 31 : L - 1) : 0;
  const uint32_t wor = wave_live ? blks[q0w / 64].bor : 0u;
  const uint32_t wand = wave_live ? blks[q0w / 64].band : 0u;
  const int nkt = (L + BN - 1) / BN;
  // Tile skipping as in the forward: a window of 64 tiles' summaries (and
  // first rows, kNoRow across a run boundary) per vector load (lane i = tile
  // k0 + i) and a ballot for the first live one.
  struct Window {
    uint32_t an, on;
    int32_t row;
  };
  // The window's words stay as loaded until pick() uses them after the
  // tile's compute: arithmetic on them, or a default written over a
  // conditionally loaded register, would make the wave wait here for the
  // load (and, in order, for every tile load issued after it).  Lanes past
  // the last tile read the last tile's record; pick() ignores them.
  auto window = [&](int k0) {
    const int k = k0 + lane < nkt ? k0 + lane : nkt - 1;
    const u32x3 x = *(const u32x3*)(blks + k);
    return Window{x[1], x[0], int32_t(x[2])};
  };
  auto pick = [&](int k0, const Window& w, uint32_t& kor_out, uint32_t& kand_out,
                  int32_t& row_out) -> int {
    const int k = k0 + lane;
    const bool ok = k < nkt && !(causal && k * BN > lastq_wg) && (qand & w.an) == 0u;
    const uint64_t m = __builtin_amdgcn_ballot_w64(ok);
    if (m == 0ull) return -1;
    const int i = __builtin_ctzll(m);
    kand_out = __builtin_amdgcn_readlane(w.an, i);
    kor_out = __builtin_amdgcn_readlane(w.on, i);
    row_out = in_place ? __builtin_amdgcn_readlane(w.row, i) : (k0 + i) * BN;
    return k0 + i;
  };
  auto next_live = [&](int kt, uint32_t& kor_out, uint32_t& kand_out, int32_t& row_out) -> int {
    for (; kt < nkt; kt += 64) {
      if (causal && kt * BN > lastq_wg) return nkt;
      const int r = pick(kt, window(kt), kor_out, kand_out, row_out);
      if (r >= 0) return r;
    }
    return nkt;
  };

  // tile loads through per-tile buffer resources (rows past the task read as
  // zero) straight into LDS; lane i of load j of wave w carries slot
  // i % CHUNKS of row RPI * (NDMA * w + j) + i / CHUNKS
  uint32_t goff[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int row = RPI * (NDMA * wave + j) + lane / CHUNKS;
    goff[j] = uint32_t((row * rs + ((lane % CHUNKS) ^ swz(row)) * 8) * 2);
  }
  auto gload = [&](int buf, int kt, int32_t trow) {
    char* kb = kvst[buf];
    char* vb = kb + KBYTES;
    if (trow != kNoRow) {
      // consecutive rows from trow
      const int64_t rows = int64_t(L) - int64_t(kt) * BN;
      const __amdgpu_buffer_rsrc_t rk = row_rsrc(Kg + int64_t(trow) * rs, rows, rs * 2, D * 2);
      const __amdgpu_buffer_rsrc_t rv = row_rsrc(Vg + int64_t(trow) * rs, rows, rs * 2, D * 2);
#pragma unroll
      for (int j = 0; j < NDMA; ++j) {
        const int off = (NDMA * wave + j) * 1024;
        buf_load16_lds(rk, kb + off, goff[j]);
        buf_load16_lds(rv, vb + off, goff[j]);
      }
    } else {
      // across a run boundary: per-lane rows from the slice base
      const __amdgpu_buffer_rsrc_t rk = row_rsrc(Kg, seq, rs * 2, D * 2);
      const __amdgpu_buffer_rsrc_t rv = row_rsrc(Vg, seq, rs * 2, D * 2);
      // the lane index behind an opaque copy keeps the per-lane row math in
      // this rarely taken branch (not hoisted out of the tile loop)
      int ln = lane;
      asm volatile("" : "+v"(ln));
#pragma unroll
      for (int j = 0; j < NDMA; ++j) {
        const int row = RPI * (NDMA * wave + j) + ln / CHUNKS;
        const int key = kt * BN + row;
        const int ch = (ln % CHUNKS) ^ swz(row);
        const uint32_t vo =
            key < L ? uint32_t((run_global(runs_s, n_runs, key) * rs + ch * 8) * 2) : kOobOffset;
        const int off = (NDMA * wave + j) * 1024;
        buf_load16_lds(rk, kb + off, vo);
        buf_load16_lds(rv, vb + off, vo);
      }
      // this rare path's offsets are temporaries: wait here, so that the
      // compiler need not make every later iteration wait before reusing
      // their registers
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    }
  };
  auto sstore = [&](int buf, int kt, uint32_t kor_t) {
    if ((qor & kor_t) != 0u && tid < BN) {
      const int key = kt * BN + tid;
      kbits_s[buf][tid] = key < L ? run_bits(runs_s, n_runs, key) : 0u;
    }
  };

  f32x16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[db][r] = 0.f;

  __syncthreads();
  const uint32_t qbits = qvalid ? run_bits(runs_s, n_runs, myq) : 0u;
  const int64_t gq = qvalid ? run_global(runs_s, n_runs, myq) : 0;
  const int64_t si = (int64_t(b) * a.H + h) * a.Lg + gq;
  const float lse2 = qvalid ? a.lse[si] * kLog2e : 0.f;
  const float Dq = qvalid ? a.D[si] : 0.f;

  // tl[0] is the tile being computed, tl[1 .. AHEAD] the next live ones
  // (nkt: none); tor, tand, trw hold their block summaries and first rows
  int tl[NBUF];
  uint32_t tor[NBUF], tand[NBUF];
  int32_t trw[NBUF];
  tl[0] = next_live(0, tor[0], tand[0], trw[0]);
#pragma unroll
  for (int k = 1; k < NBUF; ++k) {
    tor[k] = tand[k] = 0u;
    trw[k] = 0;
    tl[k] = tl[k - 1] < nkt ? next_live(tl[k - 1] + 1, tor[k], tand[k], trw[k]) : nkt;
  }
#pragma unroll
  for (int k = 0; k < AHEAD; ++k)
    if (tl[k] < nkt) {
      gload(k, tl[k], trw[k]);
      sstore(k, tl[k], tor[k]);
    }
  int buf = 0;
  // this wave's tile decisions (wave-uniform): masked for the wave, clear, mixed
  uint32_t n_masked = 0u, n_clear = 0u, n_mixed = 0u;
  while (tl[0] < nkt) {
    const int kt = tl[0];
    // this wave's loads of tile kt have landed: only those of the tile after
    // it may still be in flight.  After the barrier every wave's have, and
    // every wave is done with the buffer refilled next; the barrier leaves
    // the DMA loads in flight.
    if (AHEAD == 2 && tl[1] < nkt)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (TILE_OPS & 15));  // vmcnt(2 NDMA)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    lds_barrier_dma_in_flight();
    // the loads of the last tile ahead
    const int kc = tl[AHEAD] + 1;
    const int bl = (buf + AHEAD) % NBUF;
    if (tl[AHEAD] < nkt) gload(bl, tl[AHEAD], trw[AHEAD]);
    const uint32_t kor = tor[0], kand = tand[0];
    const int k0 = kt * BN, k1 = (k0 + BN - 1 < L ? k0 + BN - 1 : L - 1);
    const bool wfull = !wave_live || (wand & kand) != 0u || (causal && k0 > wq1);
    if (COUNT) n_masked += wfull ? 1u : 0u;
    if (!wfull) {
      const bool wclear = (wor & kor) == 0u && (!causal || k1 <= q0w) && (k0 + BN <= L);
      if (COUNT) {
        n_clear += wclear ? 1u : 0u;
        n_mixed += wclear ? 0u : 1u;
      }
      const bool use_bits = (qor & kor) != 0u;
      const char* Kb = kvst[buf];
      const char* Vb = Kb + KBYTES;
      // one 32-key block at a time: S^T, dP^T, dS^T, then its dQ^T products
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] = 0.f;
          dp[r] = 0.f;
        }
        const int row = 32 * kb + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < DK; ++ks) {
          // 16-byte chunk 2 ks + half of the row: the swizzle changes only
          // the chunk's low 3 bits, so ks >> 2 may be a separate 128-byte step
          const int slot = SPLIT_OFF ? (((2 * (ks & 3) + half) ^ swz(row)) << 4) + 128 * (ks >> 2)
                                     : ((2 * ks + half) ^ swz(row)) << 4;
          const u32x4 ka = *(const u32x4*)(Kb + row * RB + slot);
          s = mfma32<E>(bitcast_u4<vec8>(ka), qf[ks], s);
          const u32x4 va = *(const u32x4*)(Vb + row * RB + slot);
          dp = mfma32<E>(bitcast_u4<vec8>(va), of[ks], dp);
        }
        if (!wclear) {
          // mixed tile: masked scores become -inf (so P = 0); the key bits
          // arrive four keys per 16-byte LDS read and the test is a select
          const uint32_t qmask = use_bits ? qbits : 0u;
          u32x4 kbv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) kbv[i] = *(const u32x4*)(&kbits_s[buf][32 * kb + 8 * i + 4 * half]);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
            const bool keep = (key < L) & (!causal | (key <= myq)) & ((kbv[r >> 2][r & 3] & qmask) == 0u);
            s[r] = keep ? s[r] : -INFINITY;
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(s[r], c, -lse2));
          s[r] = p * (dp[r] - Dq);  // dS^T
        }
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          float pv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) pv[e] = s[8 * sub + e];
          const vec8 bs = pack8<E>(pv);
          const int trow = 32 * kb + 16 * sub + 4 * half + ((lane & 15) >> 2);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            // column 32 db + 16 ((lane >> 4) & 1) + 4 (lane & 3) lies in chunk
            // 4 db + xl; as for the row reads, db >> 1 may be a 128-byte step
            const int col = 32 * db + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
            const int xl = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
            const int tcol = SPLIT_OFF ? (((4 * (db & 1) + xl) ^ swz(trow)) << 4) + 128 * (db >> 1) + 8 * (lane & 1)
                                       : (((col >> 3) ^ swz(trow)) << 4) + (col & 7) * 2;
            const char* p0 = Kb + trow * RB + tcol;
            dq[db] = mfma32<E>(lds_tr_pair<E>(p0, p0 + 8 * RB), bs, dq[db]);
          }
        }
      }
    }
    int kc2 = nkt;
    uint32_t or2 = 0u, and2 = 0u;
    int32_t row2 = 0;
    if (tl[AHEAD] < nkt) {
      sstore(bl, tl[AHEAD], tor[AHEAD]);
      if (kc < nkt && !(causal && kc * BN > lastq_wg)) {
        // when live, from one scalar load of its block's record; else the
        // vector scan, after which this wave waits for its loads (as in the
        // forward)
        const const_u32* bw = (const_u32*)(uintptr_t)(blks + kc);
        const uint32_t bor = bw[0], band = bw[1];
        const int32_t brow = int32_t(bw[2]);
        if ((qand & band) == 0u) {
          kc2 = kc;
          or2 = bor;
          and2 = band;
          row2 = in_place ? brow : kc * BN;
        } else {
          kc2 = next_live(kc + 1, or2, and2, row2);
          __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        }
      }
    }
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) {
      tl[k] = tl[k + 1];
      tor[k] = tor[k + 1];
      tand[k] = tand[k + 1];
      trw[k] = trw[k + 1];
    }
    tl[AHEAD] = kc2;
    tor[AHEAD] = or2;
    tand[AHEAD] = and2;
    trw[AHEAD] = row2;
    buf = buf + 1 == NBUF ? 0 : buf + 1;
  }
  if (COUNT && wave_live && lane == 0) {
    atomicAdd(a.tile_count + 0, (unsigned long long)n_masked);
    atomicAdd(a.tile_count + 1, (unsigned long long)n_clear);
    atomicAdd(a.tile_count + 2, (unsigned long long)n_mixed);
  }
  if (!qvalid) return;
  // global rows accumulate (a single task holds a token once and the dQ
  // launches of a call are ordered on one stream); a task-local buffer is
  // stored.  The scaled value is rounded before the addition (no fused
  // multiply-add), so accumulating here and summing task-local buffers later
  // in task order give the same bits.
  float* dst = (LOCAL ? a.dq + tj * a.out_stride + (int64_t(b) * L + myq) * rs
                      : a.dq + (int64_t(b) * a.Lg + gq) * rs) + int64_t(h) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4* p = (f32x4*)(dst + 32 * db + 8 * i + 4 * half);
      f32x4 v = LOCAL ? f32x4{0.f, 0.f, 0.f, 0.f} : *p;
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] += mul_rounded(a.scale, dq[db][4 * i + j]);
      *p = v;
    }
}

// From d = 160 the LDS rows are padded to 256 elements, which leaves one
// work group per CU, and above 160 the dK/dV accumulators of a whole row
// (2 x d/32 blocks) and the wave's K rows do not fit in registers.  There the
// columns of dK and dV are split over two halves of an 8-wave work group
// (waves w and w + 4 own the same 32 keys; the first half takes the extra
// block of an odd d/32), each half recomputing S and dP over the full d and
// accumulating its columns; the halves share the work group's Q/dO tiles and
// V rows, and the 8 waves run two per SIMD.
template <int D> constexpr int dkdv_splits() { return D >= 160 ? 2 : 1; }
// Groups of 32 keys per work group.  At d = 96 and 128 a work group of 8
// waves owns a 256-key strip: each query tile it loads (Q and dO rows) then
// feeds twice the products, which halves the tile traffic per product; the
// LDS (a 64 KB V strip and the tiles) leaves one work group per CU, two waves
// per SIMD as before.  Elsewhere 4 groups (a 128-key strip).
template <int D> constexpr int dkdv_key_waves() { return (D == 96 || D == 128) ? 8 : 4; }
// Query rows per tile: 64 (one summary block) at d = 96, 32 (two tiles per
// block) elsewhere.  A 64-query tile halves the barriers, tile probes and
// statistics loads per product, and its two halves are computed in turn.  At
// d = 128 it would need a few registers more than the 256 two waves per SIMD
// allow, and the compiler's spill code for that kernel was wrong: it saved a
// live register under a branch's partial exec mask (waves that skip the
// branch lost the value).  So d = 128 keeps 32-query tiles, which need no
// spill.
template <int D> constexpr int dkdv_qtile() { return D == 96 ? 64 : 32; }
template <int D> constexpr int dkdv_waves() { return dkdv_key_waves<D>() * dkdv_splits<D>(); }
// Minimum waves per SIMD the compiler must allow for (the second launch
// bound): two, which caps the registers at 256, except where one work group
// of the padded rows holds a CU.
template <int D> constexpr int dkdv_min_waves() { return lds_row_elems<D>() > 128 ? 1 : 2; }

// COUNT: as for the dQ kernel, into BwdArgs::tile_count[3..5]; one count per
// 32-key group (the first of the waves that share one when the columns split)
template <typename E, int D, bool LOCAL, bool COUNT>
__global__ void __launch_bounds__(64 * dkdv_waves<D>(), dkdv_min_waves<D>()) attn_bwd_dkdv(const BwdArgs a) {
  constexpr int KW = dkdv_key_waves<D>();
  constexpr int BK = 32 * KW, BQ = dkdv_qtile<D>();
  constexpr int TSH = BQ == 32 ? 1 : 0;  // query tile t lies in summary block t >> TSH
  // Q and dO tiles: rows of DP elements (d padded as in the forward) with
  // the forward's swizzle (chunk ch of row r in slot ch ^ swz(r)),
  // conflict-free for the row reads and the transpose reads; filled by
  // direct buffer-to-LDS loads
  constexpr int DP = lds_row_elems<D>();
  constexpr int P2 = DP * 2;
  constexpr int DK = D / 16, DB = D / 32, CHUNKS = DP / 8;
  constexpr int NSPLIT = dkdv_splits<D>(), DBO = (DB + NSPLIT - 1) / NSPLIT;
  constexpr int WAVES = KW * NSPLIT, NT = 64 * WAVES;
  constexpr int RPI = 64 / CHUNKS, NDMA = BQ / RPI / WAVES;
  static_assert(NDMA >= 1 && NDMA * RPI * WAVES == BQ, "tile loads");
  typedef typename E::vec8 vec8;
  auto swz = [](int r) { return 2 * (r & 3) + ((r >> 2) & 1); };

  // a ring of NBUF query tiles (Q, dO) with their per-query statistics,
  // filled NBUF - 1 tiles ahead of the compute: three 32-query buffers for the
  // 256-key strips of d = 128 (two tiles' compute for a tile's loads to land
  // in), else two (a 64-query tile's loads land during the previous 64-query
  // tile; a third 64-query buffer would not fit beside the 256-key V strip)
  constexpr int NBUF = (KW == 8 && BQ == 32) ? 3 : 2, AHEAD = NBUF - 1;
  static_assert(NBUF == 2 || 2 * NDMA < 16, "vmcnt immediate");
  // each buffer holds the Q tile, then the dO tile: the dO rows lie a
  // constant offset from the Q rows, so their reads share address registers
  __shared__ __attribute__((aligned(1024))) char qos[NBUF][2 * BQ * P2];
  __shared__ __attribute__((aligned(1024))) char vs[BK * P2];   // the strip's V rows, swizzled
  __shared__ __attribute__((aligned(16))) float lse_s[NBUF][BQ];  // natural-log LSE
  __shared__ __attribute__((aligned(16))) float d_s[NBUF][BQ];
  __shared__ __attribute__((aligned(16))) uint32_t qbits_s[NBUF][BQ];
  __shared__ DevRun runs_s[kMaxRuns];

  const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
  // uniform per wave, so per-wave loads and branches stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int64_t work = xcd_remap(blockIdx.x, gridDim.x);
  const int tj = find_task(a.tasks, a.ntask, BK, int64_t(a.H) * a.B, work);
  const DevTask tk = a.tasks[tj];
  const int L = int(tk.L_local);
  const int64_t nstrips = (L + BK - 1) / BK;
  // the wave's 32 keys are the kw-th of the strip; it owns dK, dV columns
  // from 32-column block db0 (both fixed at 4 waves, no split)
  const int kw = NSPLIT > 1 ? (wave & 3) : wave;
  const int db0 = NSPLIT > 1 ? (wave >> 2) * DBO : 0;
  // key strips in the task's launch order (most live query tiles first; the
  // plan builds this table for BK-row strips, BK = dkdv_rows_per_wg)
  const int strip = ((const int32_t*)(a.tab + tk.korder_off))[work % nstrips];
  const int h = int((work / nstrips) % a.H);
  const int b = int(work / (nstrips * a.H));
  const int n_runs = tk.n_runs;
  const DevRun* runs_g = (const DevRun*)(a.tab + tk.runs_off);
  const DevBlock* blks = (const DevBlock*)(a.tab + tk.sum_off);
  const bool in_place = a.in_place != 0;
  for (int i = tid; i < n_runs; i += NT) runs_s[i] = runs_g[i];

  // token rows: consecutive when staged, the runs' global rows when the
  // caller's tensors are read in place
  const int64_t rs = int64_t(a.H) * D;
  const int64_t seq = in_place ? a.Lg : int64_t(L);
  const int64_t base = int64_t(b) * seq * rs + int64_t(h) * D;
  const uint16_t* Qg = (const uint16_t*)a.q + base;
  const uint16_t* Kg = (const uint16_t*)a.k + base;
  const uint16_t* Vg = (const uint16_t*)a.v + base;
  const uint16_t* Og = (const uint16_t*)a.dO + base;
  const float c = a.scale_log2;
  const bool causal = a.causal != 0;

  const int k0w = strip * BK + kw * 32;
  const int mykey = k0w + (lane & 31);
  const bool kvalid = mykey < L;
  // the wave's 32 keys lie in one 64-token block, so the table lookup and
  // its branch are wave-uniform
  int64_t krow = mykey;
  if (in_place && k0w < L) {
    const int32_t br = blks[k0w >> 6].row;
    krow = br != kNoRow ? int64_t(br) + (mykey & 63) : (kvalid ? run_global(runs_g, n_runs, mykey) : 0);
  }
  // the wave's K rows stay in registers (B operands of S = Q K^T); the
  // strip's V rows (B operands of dP = dO V^T) go to LDS once
  // every lane loads (keys past the task read row 0, then take zeros): a
  // select rather than a branch around the loads
  vec8 kf[DK];
  const int64_t kr = kvalid ? krow : 0;
#pragma unroll
  for (int ks = 0; ks < DK; ++ks) {
    u32x4 u = *(const u32x4*)(Kg + kr * rs + ks * 16 + half * 8);
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = kvalid ? u[e] : 0u;
    kf[ks] = bitcast_u4<vec8>(u);
  }
  {
    // the strip's rows are consecutive from vrow unless, read in place, one
    // of its blocks crosses a run boundary or they lie in different runs
    const int vb0 = strip * (BK / 64), vb1 = ((strip * BK + BK < L ? strip * BK + BK : L) - 1) >> 6;
    int32_t vrow = strip * BK;
    if (in_place) {
      const int32_t r0 = blks[vb0].row;
      bool one = r0 != kNoRow;
      for (int vb = vb0 + 1; vb <= vb1; ++vb) one = one && blks[vb].row == r0 + 64 * (vb - vb0);
      vrow = one ? r0 : kNoRow;
    }
    const int64_t vrows = int64_t(L) - int64_t(strip) * BK;
    const __amdgpu_buffer_rsrc_t rv =
        vrow != kNoRow ? row_rsrc(Vg + int64_t(vrow) * rs, vrows, rs * 2, D * 2)
                       : row_rsrc(Vg, seq, rs * 2, D * 2);
    constexpr int NV = BK / RPI / WAVES;  // 1 KB loads per wave
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int row = RPI * (NV * wave + j) + lane / CHUNKS;
      const int ch = (lane % CHUNKS) ^ swz(row);
      uint32_t vo = uint32_t((row * rs + ch * 8) * 2);
      if (vrow == kNoRow) {
        // per-lane rows from the slice base (the runs in global memory: the
        // LDS copy is not visible yet); tokens past the task end read zero
        const int key = strip * BK + row;
        vo = key < L ? uint32_t((run_global(runs_g, n_runs, key) * rs + ch * 8) * 2) : kOobOffset;
      }
      buf_load16_lds(rv, vs + (NV * wave + j) * 1024, vo);
    }
  }

  const int lastk_wg = (strip * BK + BK < L ? strip * BK + BK : L) - 1;
  const int kb0 = strip * (BK / 64), kb1 = lastk_wg / 64;
  uint32_t kor = 0u, kand = 0xFFFFFFFFu;
  for (int kb = kb0; kb <= kb1; ++kb) {
    kor |= blks[kb].bor;
    kand &= blks[kb].band;
  }
  const bool wave_live = k0w < L;
  const int wk1 = wave_live ? (k0w + 31 < L ? k0w + 31 : L - 1) : 0;
  const uint32_t wor = wave_live ? blks[k0w / 64].bor : 0u;
  const uint32_t wand = wave_live ? blks[k0w / 64].band : 0u;
  const int nqt = (L + BQ - 1) / BQ;
  const int first_key = strip * BK;
  const int64_t stat_base = (int64_t(b) * a.H + h) * a.Lg;

  // Query-tile skipping as in the forward (a tile is dead when fully masked
  // or, causally, entirely before the strip's first key): a window of 64
  // tiles' summaries and first rows (kNoRow when the tile's block crosses a
  // run boundary) per vector load and a ballot for the first live one.
  struct Window {
    uint32_t an, on;
    int32_t row;
  };
  // raw words until pick(), as in the dQ kernel
  auto window = [&](int t0) {
    const int t = t0 + lane < nqt ? t0 + lane : nqt - 1;
    const u32x3 x = *(const u32x3*)(blks + (t >> TSH));
    return Window{x[1], x[0], int32_t(x[2])};
  };
  // row_out: the tile's first row in the Q and dO the kernel reads (local
  // when staged); grow_out: its first global row when its queries lie in one
  // run (for the statistics), else kNoRow
  auto pick = [&](int t0, const Window& w, uint32_t& qor_out, uint32_t& qand_out,
                  int32_t& row_out, int32_t& grow_out) -> int {
    const int t = t0 + lane;
    const bool ok = t < nqt && !(causal && t * BQ + BQ - 1 < first_key) && (kand & w.an) == 0u;
    const uint64_t m = __builtin_amdgcn_ballot_w64(ok);
    if (m == 0ull) return -1;
    const int i = __builtin_ctzll(m);
    qand_out = __builtin_amdgcn_readlane(w.an, i);
    qor_out = __builtin_amdgcn_readlane(w.on, i);
    const int32_t r = __builtin_amdgcn_readlane(w.row, i);
    const int32_t grow = r != kNoRow ? r + (TSH ? ((t0 + i) & 1) * BQ : 0) : kNoRow;
    row_out = in_place ? grow : (t0 + i) * BQ;
    grow_out = grow;
    return t0 + i;
  };
  auto next_live = [&](int t, uint32_t& qor_out, uint32_t& qand_out, int32_t& row_out,
                       int32_t& grow_out) -> int {
    for (; t < nqt; t += 64) {
      const int r = pick(t, window(t), qor_out, qand_out, row_out, grow_out);
      if (r >= 0) return r;
    }
    return nqt;
  };

  // Query-tile loads, issued right after a tile barrier, all straight into
  // LDS with no register results, so nothing waits for them before the
  // barrier of the iteration that computes the tile: first, for the first BQ
  // threads, the queries' global LSE and D (rows past the task read zero:
  // their Q and dO rows are zero, so they add nothing), then the Q and dO
  // rows through per-tile buffer resources (rows past the task read zero).
  // per-lane DMA offsets kept in registers across the tile loop (a register
  // a DMA load addressed must not be rewritten while the load is in flight,
  // so per-tile temporaries would make the wave wait for it)
  uint32_t goff[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int row = RPI * (NDMA * wave + j) + lane / CHUNKS;
    goff[j] = uint32_t((row * rs + ((lane % CHUNKS) ^ swz(row)) * 8) * 2);
  }
  const uint32_t soff = uint32_t(lane) * 4;
  // the threads that load and store a tile's per-query statistics: wave 0
  // for a 64-query tile (a wave-uniform branch), its first half for 32
  const bool stat_lanes = BQ == 64 ? wave == 0 : tid < BQ;
  auto gload = [&](int buf, int qt, int32_t trow, int32_t grow) {
    if (stat_lanes) {
      lds_ptr lse_d = (lds_ptr)lse_s[buf], d_d = (lds_ptr)d_s[buf];
      if (grow != kNoRow) {
        // the tile's queries are consecutive global rows from grow
        const int64_t n = int64_t(L) - int64_t(qt) * BQ;
        const __amdgpu_buffer_rsrc_t rl = row_rsrc(a.lse + stat_base + grow, 1, 0, (n < BQ ? n : BQ) * 4);
        const __amdgpu_buffer_rsrc_t rd = row_rsrc(a.D + stat_base + grow, 1, 0, (n < BQ ? n : BQ) * 4);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, lse_d, 4, soff, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, d_d, 4, soff, 0, 0, 0);
      } else {
        const __amdgpu_buffer_rsrc_t rl = row_rsrc(a.lse + stat_base, 1, 0, a.Lg * 4);
        const __amdgpu_buffer_rsrc_t rd = row_rsrc(a.D + stat_base, 1, 0, a.Lg * 4);
        const int q = qt * BQ + tid;
        const uint32_t so = q < L ? uint32_t(run_global(runs_s, n_runs, q) * 4) : kOobOffset;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, lse_d, 4, so, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, d_d, 4, so, 0, 0, 0);
        // this rare path's offsets are temporaries: wait here, so that the
        // compiler need not make every later iteration wait before reusing
        // their registers
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
      }
    }
    if (trow != kNoRow) {
      // consecutive rows from trow
      const int64_t rows = int64_t(L) - int64_t(qt) * BQ;
      const __amdgpu_buffer_rsrc_t rq = row_rsrc(Qg + int64_t(trow) * rs, rows, rs * 2, D * 2);
      const __amdgpu_buffer_rsrc_t ro = row_rsrc(Og + int64_t(trow) * rs, rows, rs * 2, D * 2);
#pragma unroll
      for (int j = 0; j < NDMA; ++j) {
        const int off = (NDMA * wave + j) * 1024;
        buf_load16_lds(rq, qos[buf] + off, goff[j]);
        buf_load16_lds(ro, qos[buf] + BQ * P2 + off, goff[j]);
      }
    } else {
      // across a run boundary: per-lane rows from the slice base
      const __amdgpu_buffer_rsrc_t rq = row_rsrc(Qg, seq, rs * 2, D * 2);
      const __amdgpu_buffer_rsrc_t ro = row_rsrc(Og, seq, rs * 2, D * 2);
      // the lane index behind an opaque copy keeps the per-lane row math in
      // this rarely taken branch (not hoisted out of the tile loop)
      int ln = lane;
      asm volatile("" : "+v"(ln));
#pragma unroll
      for (int j = 0; j < NDMA; ++j) {
        const int row = RPI * (NDMA * wave + j) + ln / CHUNKS;
        const int q = qt * BQ + row;
        const int ch = (ln % CHUNKS) ^ swz(row);
        const uint32_t vo =
            q < L ? uint32_t((run_global(runs_s, n_runs, q) * rs + ch * 8) * 2) : kOobOffset;
        const int off = (NDMA * wave + j) * 1024;
        buf_load16_lds(rq, qos[buf] + off, vo);
        buf_load16_lds(ro, qos[buf] + BQ * P2 + off, vo);
      }
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), as for the statistics
    }
  };
  // the group bits come from the runs in LDS
  auto sstore = [&](int buf, int qt) {
    if (stat_lanes) {
      const int q = qt * BQ + tid;
      qbits_s[buf][tid] = q < L ? run_bits(runs_s, n_runs, q) : 0u;
    }
  };

  f32x16 dk[DBO], dv[DBO];
#pragma unroll
  for (int db = 0; db < DBO; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[db][r] = 0.f;
      dv[db][r] = 0.f;
    }

  __syncthreads();  // runs_s visible
  const uint32_t kbits = kvalid ? run_bits(runs_s, n_runs, mykey) : 0u;

  // tl[0] is the tile being computed, tl[1 .. AHEAD] the next live ones
  // (nqt: none); tor, tand, trw hold their block summaries and first rows
  int tl[NBUF];
  uint32_t tor[NBUF], tand[NBUF];
  int32_t trw[NBUF], tgr[NBUF];
  tl[0] = next_live(causal ? first_key / BQ : 0, tor[0], tand[0], trw[0], tgr[0]);
#pragma unroll
  for (int k = 1; k < NBUF; ++k) {
    tor[k] = tand[k] = 0u;
    trw[k] = tgr[k] = 0;
    tl[k] = tl[k - 1] < nqt ? next_live(tl[k - 1] + 1, tor[k], tand[k], trw[k], tgr[k]) : nqt;
  }
#pragma unroll
  for (int k = 0; k < AHEAD; ++k)
    if (tl[k] < nqt) {
      gload(k, tl[k], trw[k], tgr[k]);
      sstore(k, tl[k]);
    }
  int buf = 0;
  // this wave's tile decisions (wave-uniform): masked for the wave, clear, mixed
  uint32_t n_masked = 0u, n_clear = 0u, n_mixed = 0u;
  while (tl[0] < nqt) {
    const int qt = tl[0];
    // this wave's loads of tile qt have landed: only the loads of the tiles
    // after it, 2 NDMA per tile (those of wave 0 follow its two statistics
    // loads, which are older), may still be in flight.  After the barrier
    // every wave's have, and every wave is done with the buffer refilled next.
    if (AHEAD == 2 && tl[1] < nqt)
      __builtin_amdgcn_s_waitcnt(0x0F70 | ((2 * NDMA) & 15));  // vmcnt(2 NDMA)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    lds_barrier_dma_in_flight();
    // the loads of the last tile ahead
    const int qc = tl[AHEAD] + 1;
    const int bl = (buf + AHEAD) % NBUF;
    if (tl[AHEAD] < nqt) gload(bl, tl[AHEAD], trw[AHEAD], tgr[AHEAD]);
    const int q0 = qt * BQ;
    const uint32_t qor = tor[0], qand = tand[0];
    const bool wfull = !wave_live || (wand & qand) != 0u || (causal && q0 + BQ - 1 < k0w);
    if (COUNT) n_masked += wfull ? 1u : 0u;
    if (!wfull) {
      const bool wclear = (wor & qor) == 0u && (!causal || q0 >= wk1);
      if (COUNT) {
        n_clear += wclear ? 1u : 0u;
        n_mixed += wclear ? 0u : 1u;
      }
      const bool use_bits = (kor & qor) != 0u;
      const uint32_t kmask = use_bits ? kbits : 0u;
      const char* qsb = qos[buf];
      const char* osb = qsb + BQ * P2;
#pragma unroll 1
      for (int qb = 0; qb < BQ / 32; ++qb) {
        f32x16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] = 0.f;
          dp[r] = 0.f;
        }
        const int row = 32 * qb + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < DK; ++ks) {
          // 16-byte chunk 2 ks + half of the row: the swizzle changes only
          // the chunk's low 3 bits, so writing ks >> 2 as a separate 128-byte
          // step leaves four distinct per-lane offsets (the rest immediate)
          const int slot = (((2 * (ks & 3) + half) ^ swz(row)) << 4) + 128 * (ks >> 2);
          const u32x4 qa = *(const u32x4*)(qsb + row * P2 + slot);
          s = mfma32<E>(bitcast_u4<vec8>(qa), kf[ks], s);
          const u32x4 oa = *(const u32x4*)(osb + row * P2 + slot);
          const int vr = kw * 32 + (lane & 31);
          const u32x4 vb = *(const u32x4*)(vs + vr * P2 + (((2 * (ks & 3) + half) ^ swz(vr)) << 4) +
                                           128 * (ks >> 2));
          dp = mfma32<E>(bitcast_u4<vec8>(oa), bitcast_u4<vec8>(vb), dp);
        }
        // 16 queries at a time: P and dS = P (dP - D), packed for dV and dK
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          float pv[8], dsv[8];
#pragma unroll
          for (int ii = 0; ii < 2; ++ii) {
            const int ql = 32 * qb + 8 * (2 * sub + ii) + 4 * half;
            const f32x4 l4 = *(const f32x4*)(&lse_s[buf][ql]) * kLog2e;
            const f32x4 d4 = *(const f32x4*)(&d_s[buf][ql]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int r = 8 * sub + 4 * ii + j;
              pv[4 * ii + j] = fast_exp2(fmaf(s[r], c, -l4[j]));
            }
            if (!wclear) {
              // mixed tile: the query bits of these four queries come in one
              // 16-byte LDS read and the test is a select
              const u32x4 qb4 = *(const u32x4*)(&qbits_s[buf][ql]);
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const bool keep = (!causal | (mykey <= q0 + ql + j)) & ((qb4[j] & kmask) == 0u);
                pv[4 * ii + j] = keep ? pv[4 * ii + j] : 0.f;
              }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) dsv[4 * ii + j] = pv[4 * ii + j] * (dp[8 * sub + 4 * ii + j] - d4[j]);
          }
          const vec8 bp = pack8<E>(pv);
          const vec8 bs = pack8<E>(dsv);
          const int trow = 32 * qb + 16 * sub + 4 * half + ((lane & 15) >> 2);
#pragma unroll
          for (int db = 0; db < DBO; ++db) {
            if (NSPLIT > 1 && db0 + db >= DB) break;  // the last half of an odd d/32
            // column 32 g + 16 ((lane >> 4) & 1) + 4 (lane & 3) of block g
            // lies in chunk 4 g + xl; as for the row reads, g >> 1 is a
            // separate 128-byte step
            const int g = db0 + db;
            const int xl = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
            const int tcol = (((4 * (g & 1) + xl) ^ swz(trow)) << 4) + 128 * (g >> 1) + 8 * (lane & 1);
            const char* po = osb + trow * P2 + tcol;
            dv[db] = mfma32<E>(lds_tr_pair<E>(po, po + 8 * P2), bp, dv[db]);
            const char* pq = qsb + trow * P2 + tcol;
            dk[db] = mfma32<E>(lds_tr_pair<E>(pq, pq + 8 * P2), bs, dk[db]);
          }
        }
      }
    }
    int qc2 = nqt;
    uint32_t or2 = 0u, and2 = 0u;
    int32_t row2 = 0, grow2 = 0;
    if (tl[AHEAD] < nqt) {
      sstore(bl, tl[AHEAD]);
      if (qc < nqt) {
        // the tile after it, when live, from one scalar load of its block's
        // record (scalar loads are counted apart from the tile loads, so
        // nothing here waits for those); else the vector scan, after which
        // this wave waits for its loads (the scan's registers are reused by
        // the next iteration, and the compiler would otherwise wait for them,
        // and for the tile loads, on every iteration)
        const const_u32* bw = (const_u32*)(uintptr_t)(blks + (qc >> TSH));
        const uint32_t bor = bw[0], band = bw[1];
        const int32_t brow = int32_t(bw[2]);
        if (!(causal && qc * BQ + BQ - 1 < first_key) && (kand & band) == 0u) {
          qc2 = qc;
          or2 = bor;
          and2 = band;
          grow2 = brow != kNoRow ? brow + (TSH ? (qc & 1) * BQ : 0) : kNoRow;
          row2 = in_place ? grow2 : qc * BQ;
        } else {
          qc2 = next_live(qc + 1, or2, and2, row2, grow2);
          __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        }
      }
    }
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) {
      tl[k] = tl[k + 1];
      tor[k] = tor[k + 1];
      tand[k] = tand[k + 1];
      trw[k] = trw[k + 1];
      tgr[k] = tgr[k + 1];
    }
    tl[AHEAD] = qc2;
    tor[AHEAD] = or2;
    tand[AHEAD] = and2;
    trw[AHEAD] = row2;
    tgr[AHEAD] = grow2;
    buf = buf + 1 == NBUF ? 0 : buf + 1;
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // the V fill has landed even when no tile was live
  if (COUNT && wave_live && db0 == 0 && lane == 0) {
    atomicAdd(a.tile_count + 3, (unsigned long long)n_masked);
    atomicAdd(a.tile_count + 4, (unsigned long long)n_clear);
    atomicAdd(a.tile_count + 5, (unsigned long long)n_mixed);
  }
  if (!kvalid) return;
  // global rows accumulate; a task-local buffer is stored (as for dQ, the
  // scaled dK is rounded before the addition)
  const int64_t orow = LOCAL ? tj * a.out_stride + (int64_t(b) * L + mykey) * rs
                             : (int64_t(b) * a.Lg + run_global(runs_s, n_runs, mykey)) * rs;
  float* dkp = a.dk + orow + int64_t(h) * D;
  float* dvp = a.dv + orow + int64_t(h) * D;
#pragma unroll
  for (int db = 0; db < DBO; ++db) {
    if (NSPLIT > 1 && db0 + db >= DB) break;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int off = 32 * (db0 + db) + 8 * i + 4 * half;
      f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f}, y = x;
      if (!LOCAL) {
        x = *(f32x4*)(dkp + off);
        y = *(f32x4*)(dvp + off);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] += mul_rounded(a.scale, dk[db][4 * i + j]);
        y[j] += dv[db][4 * i + j];
      }
      *(f32x4*)(dkp + off) = x;
      *(f32x4*)(dvp + off) = y;
    }
  }
}

template <typename E, int D, bool LOCAL>
static void launch_dq_l(const BwdArgs& a, int64_t n, hipStream_t s) {
  if (a.tile_count)
    hipLaunchKernelGGL((attn_bwd_dq<E, D, LOCAL, true>), dim3(unsigned(n)), dim3(64 * dq_waves<D>()), 0, s, a);
  else
    hipLaunchKernelGGL((attn_bwd_dq<E, D, LOCAL, false>), dim3(unsigned(n)), dim3(64 * dq_waves<D>()), 0, s, a);
}

template <typename E, int D>
static hipError_t launch_dq_t(const BwdArgs& a, int64_t n, hipStream_t s) {
  if (a.local_out)
    launch_dq_l<E, D, true>(a, n, s);
  else
    launch_dq_l<E, D, false>(a, n, s);
  return hipGetLastError();
}

template <typename E, int D, bool LOCAL>
static void launch_dkdv_l(const BwdArgs& a, int64_t n, hipStream_t s) {
  if (a.tile_count)
    hipLaunchKernelGGL((attn_bwd_dkdv<E, D, LOCAL, true>), dim3(unsigned(n)), dim3(64 * dkdv_waves<D>()), 0, s, a);
  else
    hipLaunchKernelGGL((attn_bwd_dkdv<E, D, LOCAL, false>), dim3(unsigned(n)), dim3(64 * dkdv_waves<D>()), 0, s, a);
}

template <typename E, int D>
static hipError_t launch_dkdv_t(const BwdArgs& a, int64_t n, hipStream_t s) {
  if (a.local_out)
    launch_dkdv_l<E, D, true>(a, n, s);
  else
    launch_dkdv_l<E, D, false>(a, n, s);
  return hipGetLastError();
}

#define CQSA_BWD_SWITCH(LAUNCH)                                        \
  switch (d) {                                                         \
    case 32: return dt == CQSA_BF16 ? LAUNCH<BF16, 32>(a, wgs, s) : LAUNCH<F16, 32>(a, wgs, s);    \
    case 64: return dt == CQSA_BF16 ? LAUNCH<BF16, 64>(a, wgs, s) : LAUNCH<F16, 64>(a, wgs, s);    \
    case 96: return dt == CQSA_BF16 ? LAUNCH<BF16, 96>(a, wgs, s) : LAUNCH<F16, 96>(a, wgs, s);    \
    case 128: return dt == CQSA_BF16 ? LAUNCH<BF16, 128>(a, wgs, s) : LAUNCH<F16, 128>(a, wgs, s); \
    case 160: return dt == CQSA_BF16 ? LAUNCH<BF16, 160>(a, wgs, s) : LAUNCH<F16, 160>(a, wgs, s); \
    case 192: return dt == CQSA_BF16 ? LAUNCH<BF16, 192>(a, wgs, s) : LAUNCH<F16, 192>(a, wgs, s); \
    case 224: return dt == CQSA_BF16 ? LAUNCH<BF16, 224>(a, wgs, s) : LAUNCH<F16, 224>(a, wgs, s); \
    case 256: return dt == CQSA_BF16 ? LAUNCH<BF16, 256>(a, wgs, s) : LAUNCH<F16, 256>(a, wgs, s); \
  }                                                                    \
  return hipErrorInvalidValue;

int dkdv_qtile_rows(int d) {
  switch (d) {
#define CQSA_KV_QTILE(DD) \
  case DD:                \
    return dkdv_qtile<DD>();
    CQSA_KV_QTILE(32)
    CQSA_KV_QTILE(64)
    CQSA_KV_QTILE(96)
    CQSA_KV_QTILE(128)
    CQSA_KV_QTILE(160)
    CQSA_KV_QTILE(192)
    CQSA_KV_QTILE(224)
    CQSA_KV_QTILE(256)
#undef CQSA_KV_QTILE
  }
  return 32;
}

int dkdv_rows_per_wg(int d) {
  switch (d) {
#define CQSA_KV_ROWS(DD) \
  case DD:               \
    return 32 * dkdv_key_waves<DD>();
    CQSA_KV_ROWS(32)
    CQSA_KV_ROWS(64)
    CQSA_KV_ROWS(96)
    CQSA_KV_ROWS(128)
    CQSA_KV_ROWS(160)
    CQSA_KV_ROWS(192)
    CQSA_KV_ROWS(224)
    CQSA_KV_ROWS(256)
#undef CQSA_KV_ROWS
  }
  return 128;
}

int dq_rows_per_wg(int d) {
  switch (d) {
#define CQSA_DQ_ROWS(DD) \
  case DD:               \
    return 32 * dq_waves<DD>();
    CQSA_DQ_ROWS(32)
    CQSA_DQ_ROWS(64)
    CQSA_DQ_ROWS(96)
    CQSA_DQ_ROWS(128)
    CQSA_DQ_ROWS(160)
    CQSA_DQ_ROWS(192)
    CQSA_DQ_ROWS(224)
    CQSA_DQ_ROWS(256)
#undef CQSA_DQ_ROWS
  }
  return 128;
}

// Launch checks: a task table, a grid that fits, and global accumulation
// only for a single task (tasks of one launch may share tokens).
static bool bwd_launch_ok(cqsa_dtype dt, const BwdArgs& a, int64_t wgs) {
  if (dt != CQSA_BF16 && dt != CQSA_F16) return false;
  if (a.ntask < 1 || !a.tasks || !a.tab || wgs > 0x7fffffff) return false;
  return a.local_out != 0 || a.ntask == 1;
}

hipError_t launch_bwd_dq(cqsa_dtype dt, int d, const BwdArgs& a, int64_t wgs, hipStream_t s) {
  if (wgs == 0) return hipSuccess;
  if (!bwd_launch_ok(dt, a, wgs)) return hipErrorInvalidValue;
  CQSA_BWD_SWITCH(launch_dq_t)
}

hipError_t launch_bwd_dkdv(cqsa_dtype dt, int d, const BwdArgs& a, int64_t wgs, hipStream_t s) {
  if (wgs == 0) return hipSuccess;
  if (!bwd_launch_ok(dt, a, wgs)) return hipErrorInvalidValue;
  CQSA_BWD_SWITCH(launch_dkdv_t)
}
#undef CQSA_BWD_SWITCH

}  // namespace cqsa
