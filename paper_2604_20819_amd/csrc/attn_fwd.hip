// Inner forward kernels: masked flash-style attention over one CQS task.
//
// One launch covers the tasks of a launch group.  Each work group owns a
// 128- or 256-query strip of one (task, batch, head) and walks the task's
// 64-key tiles with an online softmax, emitting the local statistics (unnormalised
// acc, row max m, row sum l) that the max-shifted merge of App. A.1
// (Eq. "merge") recomposes across tasks.
//
// Tile verdicts (App. A.2): from the 64-token block summaries a (strip, key
// tile) pair is fully masked (AND(rows) & AND(cols) != 0, or causally empty),
// clear (OR(rows) & OR(cols) == 0 and causally full) or mixed; fully masked
// tiles are never loaded, clear tiles run without any mask work, and only
// mixed tiles apply the per-element test bits[q] & bits[k] == 0.  Because
// tokens are gathered in ascending order, the causal test is on local indices.
//
// gfx950 design: S^T = K Q^T on v_mfma_f32_32x32x16 so each lane owns one
// query column and its row statistics stay in-lane (one permlane32 swap per
// tile); P^T feeds O^T = V^T P^T directly from registers, and V^T operands come
// from row-major LDS through ds_read_b64_tr_b16.  K/V tiles rotate through two
// or three LDS buffers, filled by direct buffer-to-LDS loads issued right
// after each tile barrier, so they cost no registers and no LDS store
// instructions.  Each row's shift (the running maximum in the log2 domain) is
// an integer, so every rescale is an exact power of two and 16-bit P is
// rounded identically whichever task, or the undecomposed call, produced it;
// a tile keeps the row's shift while the weights it gives stay bounded, and
// takes the exact maximum, rounded up, otherwise.
//
// Two row sums: l adds the fp32 weights (it gives the log-sum-exp), lt adds
// the 16-bit weights the P.V product actually consumes.  Both are task
// statistics merged with the same power-of-two factors, and O = acc / lt is
// the exactly normalised average of V rows under the rounded weights (a
// one-hot row returns its V row) whatever the decomposition: every task
// rounds the same weights to the same values.
#include "hip_common.hpp"
#include "kernels.hpp"

namespace cqsa {

// Waves per work group: 8 (256-query strips) for d = 96 ... 192, where two
// waves per SIMD is the occupancy either way and the kernel fits the 256
// registers per lane that leaves: the K/V tiles a work group loads serve
// twice the queries, and d = 160, 192 (one work group per CU for LDS) still
// run two waves per SIMD.  4 (128-query strips) for d = 32, 64, whose 4-wave
// work groups fit three to a CU, and for d = 224, 256, which would spill.
template <int D> constexpr int fwd_waves() { return (D >= 96 && D <= 192) ? 8 : 4; }

// COUNT: the launch counts its tile decisions (FwdArgs::tile_count); a
// separate instance, so that the kernel without counting does no counting work
template <typename E, int D, int MODE, bool COUNT>
__global__ void __launch_bounds__(64 * fwd_waves<D>(), (lds_row_elems<D>() > 128 ? 1 : 2)) attn_fwd_mfma(const FwdArgs a) {
  constexpr int WAVES = fwd_waves<D>(), NT = 64 * WAVES;
  constexpr int BM = 32 * WAVES, BN = 64;
  // K and V tiles: unpadded rows of 2D bytes; 16-byte chunk ch of row r sits
  // in slot ch ^ swz(r), which keeps the K row reads and the V transpose
  // reads free of bank conflicts.  Tiles arrive by direct global-to-LDS
  // loads: one wave instruction fills 1 KB, lane i its i-th 16 bytes.
  constexpr int DP = lds_row_elems<D>(); // LDS row elements (d padded)
  constexpr int RB = DP * 2;             // LDS row bytes
  constexpr int KBYTES = BN * RB, VBYTES = BN * RB;
  constexpr int DK = D / 16;             // k-steps of S^T = K Q^T
  constexpr int DB = D / 32;             // 32-wide d blocks of O^T
  constexpr int CHUNKS = DP / 8;         // 16-byte chunks per LDS row
  constexpr int RPI = 64 / CHUNKS;       // rows per 1 KB load instruction
  constexpr int NDMA = BN / RPI / WAVES; // load instructions per wave per tensor
  static_assert(NDMA >= 1, "tile loads");
  typedef typename E::vec8 vec8;
  auto swz = [](int r) { return 2 * (r & 3) + ((r >> 2) & 1); };

  // a ring of NBUF key tiles (K, V), filled NBUF - 1 tiles ahead of the
  // compute: three at d = 96 and 128, whose 8-wave work group per CU leaves
  // the LDS for a third tile, two elsewhere
  constexpr int NBUF = (WAVES == 8 && DP <= 128) ? 3 : 2, AHEAD = NBUF - 1;
  // loads of one tile per wave (the vmcnt that leaves them in flight)
  constexpr int TILE_OPS = 2 * NDMA;
  static_assert(NBUF == 2 || TILE_OPS < 16, "vmcnt immediate");
  __shared__ __attribute__((aligned(1024))) char kst[NBUF][KBYTES];
  __shared__ __attribute__((aligned(1024))) char vst[NBUF][VBYTES];
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
  // builds this table for BM-row strips, BM = fwd_rows_per_wg)
  const int strip = ((const int32_t*)(a.tab + tk.qorder_off))[work % nstrips];
  const int h = int((work / nstrips) % a.H);
  const int b = int(work / (nstrips * a.H));
  const int n_runs = tk.n_runs;
  const DevBlock* blks = (const DevBlock*)(a.tab + tk.sum_off);
  const DevRun* runs_g = (const DevRun*)(a.tab + tk.runs_off);
  const bool in_place = a.in_place != 0;

  for (int i = tid; i < n_runs; i += NT) runs_s[i] = runs_g[i];

  // Staged inputs hold the task's tokens as consecutive rows; inputs read in
  // place are the caller's tensors, where local token t sits at the global
  // row its run gives (the block row table answers for whole blocks).
  const int64_t rs = int64_t(a.H) * D;  // elements between consecutive tokens
  const int64_t seq = in_place ? a.Lg : int64_t(L);  // rows per batch element
  const int64_t base = int64_t(b) * seq * rs + int64_t(h) * D + tj * a.in_stride;
  const uint16_t* Qg = (const uint16_t*)a.q + base;
  const uint16_t* Kg = (const uint16_t*)a.k + base;
  const uint16_t* Vg = (const uint16_t*)a.v + base;
  const float c = a.scale_log2;
  const bool causal = a.causal != 0;

  const int q0w = strip * BM + wave * 32;  // first query of this wave
  const int myq = q0w + (lane & 31);
  const bool qvalid = myq < L;
  // the wave's 32 queries lie in one 64-token block, so the table lookup and
  // its branch are wave-uniform
  int64_t qrow = myq;
  if (in_place && q0w < L) {
    const int32_t br = blks[q0w >> 6].row;
    qrow = br != kNoRow ? int64_t(br) + (myq & 63) : (qvalid ? run_global(runs_g, n_runs, myq) : 0);
  }

  vec8 qf[DK];
#pragma unroll
  for (int ks = 0; ks < DK; ++ks) {
    u32x4 u = {0u, 0u, 0u, 0u};
    if (qvalid) u = *(const u32x4*)(Qg + qrow * rs + ks * 16 + half * 8);
    qf[ks] = bitcast_u4<vec8>(u);
  }

  // block summaries of the strip and of this wave's queries
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
  // Tile skipping (App. A.2): a key tile is live for the strip unless it is
  // fully masked (AND of the strip's and the tile's group bits non-zero) or
  // causally empty.  Each wave reads a window of 64 tiles' block summaries
  // with one vector load (lane i holds tile k0 + i); a ballot then names the
  // first live tile.  The main loop issues the window for the tile after the
  // next one before its prefetch and consumes it after the compute, so these
  // loads never stall a tile.  The window also carries each tile's first
  // row in the inputs (kNoRow for a tile that crosses a run boundary).
  struct Window {
    uint32_t an, on;  // this lane's tile summaries (AND, OR)
    int32_t row;
  };
  // The window's words stay as loaded until pick() uses them after the
  // tile's compute: arithmetic on them, or a default written over a
  // conditionally loaded register, would make the wave wait for the load
  // (and, in order, for every tile load issued after it).  Lanes past the
  // last tile read the last tile's record; pick() ignores them.
  auto window = [&](int k0) {
    const int k = k0 + lane < nkt ? k0 + lane : nkt - 1;
    const u32x3 x = *(const u32x3*)(blks + k);
    return Window{x[1], x[0], int32_t(x[2])};
  };
  // First live tile in [k0, k0 + 64), or -1; its summaries in kor_out/kand_out
  // and its first row in row_out.
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
  // First live tile at or after kt (blocking; walks windows).
  auto next_live = [&](int kt, uint32_t& kor_out, uint32_t& kand_out, int32_t& row_out) -> int {
    for (; kt < nkt; kt += 64) {
      if (causal && kt * BN > lastq_wg) return nkt;
      const int r = pick(kt, window(kt), kor_out, kand_out, row_out);
      if (r >= 0) return r;
    }
    return nkt;
  };

  // Tile loads: per-tile buffer resources (SGPR base, fixed per-lane 32-bit
  // offsets; rows past the task end read as zero) feeding LDS directly.
  // Instruction j of wave w fills rows RPI*(NDMA*w + j) ...; lane i carries
  // slot i % CHUNKS of its row, i.e. global chunk (i % CHUNKS) ^ swz(row).
  uint32_t goff[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int row = RPI * (NDMA * wave + j) + lane / CHUNKS;
    const int ch = (lane % CHUNKS) ^ swz(row);
    goff[j] = uint32_t((row * rs + ch * 8) * 2);
  }
  auto gload = [&](int buf, int kt, int32_t trow) {
    char* kb = kst[buf];
    char* vb = vst[buf];
    if (trow != kNoRow) {
      // the tile's tokens are consecutive rows from trow
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
      // a tile crossing a run boundary (inputs read in place): each lane
      // addresses its token's row from the slice base; tokens past the task
      // end read as zero
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
    // group bits of the tile's keys, only when the CQS mask can bite here
    if ((qor & kor_t) != 0u && tid < BN) {
      const int key = kt * BN + tid;
      kbits_s[buf][tid] = key < L ? run_bits(runs_s, n_runs, key) : 0u;
    }
  };

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f, lt_run = 0.f;

  __syncthreads();  // runs_s visible
  const uint32_t qbits = qvalid ? run_bits(runs_s, n_runs, myq) : 0u;

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
    // it (2 NDMA) may still be in flight.  After the barrier every wave's
    // have, and every wave is done with the buffer refilled next; the
    // barrier itself leaves the DMA loads in flight.
    if (AHEAD == 2 && tl[1] < nkt)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (TILE_OPS & 15));  // vmcnt(2 NDMA)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    lds_barrier_dma_in_flight();
    // the loads of the last tile ahead
    const int kc = tl[AHEAD] + 1;
    const int bl = (buf + AHEAD) % NBUF;
    if (tl[AHEAD] < nkt) gload(bl, tl[AHEAD], trw[AHEAD]);

    // ---- compute on tile kt (wave-uniform verdict) ----
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
      const char* Kb = kst[buf];
      const char* Vb = vst[buf];
      // S^T of the tile, the mixed tile's masked scores -inf; the two 32-key
      // blocks' accumulation chains alternate, so consecutive products never
      // depend on each other
      auto scores = [&](f32x16(&s)[2]) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
        // K operands read two steps ahead of their products.  Up to d = 192
        // the 16-byte chunk 2 ks + half is addressed as a swizzled low part
        // (the swizzle changes only the chunk's low 3 bits) plus ks >> 2 as
        // an immediate 128-byte step, which needs four per-lane offsets
        // instead of eight and frees registers; at 224 and 256 (one wave per
        // SIMD, registers to spare) that measured slower
        constexpr bool SPLIT_OFF = D <= 192;
        auto kread = [&](int ks, int kb) {
          const int kr = 32 * kb + (lane & 31);
          const int slot = SPLIT_OFF ? (((2 * (ks & 3) + half) ^ swz(kr)) << 4) + 128 * (ks >> 2)
                                     : ((2 * ks + half) ^ swz(kr)) << 4;
          return *(const u32x4*)(Kb + kr * RB + slot);
        };
        u32x4 ka[3][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          ka[0][kb] = kread(0, kb);
          ka[1][kb] = kread(1, kb);
        }
#pragma unroll
        for (int ks = 0; ks < DK; ++ks) {
          if (ks + 2 < DK) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) ka[(ks + 2) % 3][kb] = kread(ks + 2, kb);
          }
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) s[kb] = mfma32<E>(bitcast_u4<vec8>(ka[ks % 3][kb]), qf[ks], s[kb]);
        }
        // keep the reads two steps ahead of the products they feed
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int ks = 0; ks < DK; ++ks) {
          if (ks + 2 < DK) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        }
        if (!wclear) {
          // mixed tile: the group bits of this lane's 32 keys arrive four
          // consecutive keys per 16-byte LDS read, all issued before any is
          // used, and the per-element test is a select (no branch, no
          // short-circuit); with use_bits false the bits drop out of the test
          const uint32_t qmask = use_bits ? qbits : 0u;
          u32x4 kbv[2][4];
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              kbv[kb][i] = *(const u32x4*)(&kbits_s[buf][32 * kb + 8 * i + 4 * half]);
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = k0 + 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
              const bool keep = (key < L) & (!causal | (key <= myq)) &
                                ((kbv[kb][r >> 2][r & 3] & qmask) == 0u);
              s[kb][r] = keep ? s[kb][r] : -INFINITY;
            }
        }
      };
      f32x16 s[2];
      scores(s);
      // The running maximum is an integer (log2) and rarely rises, so the
      // tile first keeps it: a lane's sum of weights bounds each of them, and
      // a sum <= 2^16 leaves P, acc, l and lt far inside fp32 (another integer
      // shift scales them by a power of two, undone by the final division or
      // the merge).  While some lane has no maximum yet, or when a sum exceeds
      // the bound, the tile takes the exact maximum, with its scores
      // recomputed if the first try overwrote them.
      float psum = 0.f;
      bool kept = false;
      {
        if (__builtin_amdgcn_ballot_w64(m_run == -INFINITY) == 0ull) {
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float p = fast_exp2(fmaf(s[kb][r], c, -m_run));
              s[kb][r] = p;
              psum += p;
            }
          kept = __builtin_amdgcn_ballot_w64(!(psum <= 65536.f)) == 0ull;
          if (!kept) scores(s);
        }
      }
      if (!kept) {
        float smax = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) smax = fmaxf(smax, s[kb][r]);
        smax = fmaxf(smax, swap_halves(smax));
        const float mnew = fmaxf(m_run, ceilf(smax * c));
        const float msafe = mnew == -INFINITY ? 0.f : mnew;
        const float alpha = fast_exp2(m_run - msafe);
        m_run = mnew;
        // integer maxima change rarely: rescale only when some lane's did
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0ull) {
          l_run *= alpha;
          lt_run *= alpha;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        }
        psum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = fast_exp2(fmaf(s[kb][r], c, -msafe));
            s[kb][r] = p;
            psum += p;
          }
      }
      l_run += psum;
#pragma unroll
      for (int ks2 = 0; ks2 < 4; ++ks2) {
        const int kb = ks2 >> 1, sub = ks2 & 1;
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[e] = s[kb][8 * sub + e];
        const vec8 pb = pack8<E>(pv);
        lt_run = sum8<E>(pb, lt_run);
        const int row = 32 * kb + 16 * sub + 4 * half + ((lane & 15) >> 2);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int col = 32 * db + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
          // column col lies in chunk 4 db + xl: as for the K reads, db >> 1
          // may be a separate 128-byte step
          const int xl = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
          const int vcol = D <= 192 ? (((4 * (db & 1) + xl) ^ swz(row)) << 4) + 128 * (db >> 1) + 8 * (lane & 1)
                                    : (((col >> 3) ^ swz(row)) << 4) + (col & 7) * 2;
          const char* p0 = Vb + row * RB + vcol;
          const vec8 va = lds_tr_pair<E>(p0, p0 + 8 * RB);
          o[db] = mfma32<E>(va, pb, o[db]);
        }
      }
    }
    // ---- group bits of the last tile ahead, the live tile after it ----
    int kc2 = nkt;
    uint32_t or2 = 0u, and2 = 0u;
    int32_t row2 = 0;
    if (tl[AHEAD] < nkt) {
      sstore(bl, tl[AHEAD], tor[AHEAD]);
      if (kc < nkt && !(causal && kc * BN > lastq_wg)) {
        // when live, from one scalar load of its block's record (scalar
        // loads are counted apart from the tile loads, so nothing here waits
        // for those); else the vector scan, after which this wave waits for
        // its loads (the scan's registers are reused by the next iteration,
        // and the compiler would otherwise wait for them, and for the tile
        // loads, on every iteration)
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

  const float l_tot = l_run + swap_halves(l_run);
  const float lt_tot = lt_run + swap_halves(lt_run);
  if (COUNT && wave_live && lane == 0) {
    atomicAdd(a.tile_count + 0, (unsigned long long)n_masked);
    atomicAdd(a.tile_count + 1, (unsigned long long)n_clear);
    atomicAdd(a.tile_count + 2, (unsigned long long)n_mixed);
  }
  if (!qvalid) return;
  if (MODE == kModeStats) {
    float* accp = a.acc + tj * a.acc_stride + (int64_t(b) * L + myq) * rs + int64_t(h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v = {o[db][4 * i], o[db][4 * i + 1], o[db][4 * i + 2], o[db][4 * i + 3]};
        *(f32x4*)(accp + 32 * db + 8 * i + 4 * half) = v;
      }
    if (half == 0) {
      const int64_t si = tj * a.st_stride + (int64_t(b) * a.H + h) * L + myq;
      a.m[si] = m_run;
      a.l[si] = l_tot;
      a.lt[si] = lt_tot;
    }
  } else {
    const float inv = 1.f / lt_tot;
    float* op = a.acc + (int64_t(b) * L + myq) * rs + int64_t(h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v = {o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv,
                   o[db][4 * i + 3] * inv};
        *(f32x4*)(op + 32 * db + 8 * i + 4 * half) = v;
      }
    if (half == 0) {
      const int64_t si = (int64_t(b) * a.H + h) * L + myq;
      a.m[si] = (m_run + __log2f(l_tot)) * 0.69314718055994530942f;
    }
  }
}

// fp32 inputs: plain VALU flash loop (8 threads per query, d/8 dims each).
// Same statistics convention as the MFMA kernel (log2 domain, integer max).
template <int D, int MODE>
__global__ void __launch_bounds__(256) attn_fwd_f32(const FwdArgs a) {
  constexpr int QPB = 32, BN = 32, SL = D / 8;
  __shared__ float ks_[BN][D + 1];
  __shared__ float vs_[BN][D + 1];
  __shared__ uint32_t kbits_s[BN];
  __shared__ int64_t krow_s[BN];
  __shared__ DevRun runs_s[kMaxRuns];
  const int tid = threadIdx.x, sub = tid & 7, ql = tid >> 3;
  int64_t work = blockIdx.x;
  const int tj = find_task(a.tasks, a.ntask, QPB, int64_t(a.H) * a.B, work);
  const DevTask tk = a.tasks[tj];
  const int L = int(tk.L_local);
  const int64_t nstrips = (L + QPB - 1) / QPB;
  const int strip = int(work % nstrips);
  const int h = int((work / nstrips) % a.H);
  const int b = int(work / (nstrips * a.H));
  const int n_runs = tk.n_runs;
  const DevRun* runs_g = (const DevRun*)(a.tab + tk.runs_off);
  const DevBlock* blks = (const DevBlock*)(a.tab + tk.sum_off);
  const bool in_place = a.in_place != 0;
  for (int i = tid; i < n_runs; i += 256) runs_s[i] = runs_g[i];
  // token rows as in the MFMA kernel: consecutive when staged, the runs'
  // global rows when read in place
  const int64_t rs = int64_t(a.H) * D;
  const int64_t seq = in_place ? a.Lg : int64_t(L);
  const int64_t base = int64_t(b) * seq * rs + int64_t(h) * D + tj * a.in_stride;
  const float* Qg = (const float*)a.q + base;
  const float* Kg = (const float*)a.k + base;
  const float* Vg = (const float*)a.v + base;
  const float c = a.scale_log2;
  const int myq = strip * QPB + ql;
  const bool qvalid = myq < L;
  const int64_t qrow = !qvalid ? 0 : in_place ? in_place_row(blks, runs_g, n_runs, myq) : myq;
  float q[SL], o[SL];
#pragma unroll
  for (int i = 0; i < SL; ++i) {
    q[i] = qvalid ? Qg[qrow * rs + sub * SL + i] : 0.f;
    o[i] = 0.f;
  }
  __syncthreads();
  const uint32_t qbits = qvalid ? run_bits(runs_s, n_runs, myq) : 0u;
  float m_run = -INFINITY, l_run = 0.f;
  const int nkt = (L + BN - 1) / BN;
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    if (tid < BN) {
      const int key = kt * BN + tid;
      kbits_s[tid] = key < L ? run_bits(runs_s, n_runs, key) : 0xFFFFFFFFu;
      krow_s[tid] = key >= L ? 0 : in_place ? run_global(runs_s, n_runs, key) : key;
    }
    __syncthreads();
    for (int i = tid; i < BN * D; i += 256) {
      const int r = i / D, dd = i % D, key = kt * BN + r;
      ks_[r][dd] = key < L ? Kg[krow_s[r] * rs + dd] : 0.f;
      vs_[r][dd] = key < L ? Vg[krow_s[r] * rs + dd] : 0.f;
    }
    __syncthreads();
    float s[BN];
    float smax = -INFINITY;
#pragma unroll
    for (int j = 0; j < BN; ++j) {
      float part = 0.f;
#pragma unroll
      for (int i = 0; i < SL; ++i) part = fmaf(q[i], ks_[j][sub * SL + i], part);
      part += __shfl_xor(part, 1);
      part += __shfl_xor(part, 2);
      part += __shfl_xor(part, 4);
      const int key = kt * BN + j;
      const bool keep = key < L && (!a.causal || key <= myq) && (kbits_s[j] & qbits) == 0u;
      s[j] = keep ? part : -INFINITY;
      smax = fmaxf(smax, s[j]);
    }
    const float mnew = fmaxf(m_run, ceilf(smax * c));
    const float msafe = mnew == -INFINITY ? 0.f : mnew;
    const float alpha = exp2f(m_run - msafe);
    m_run = mnew;
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < SL; ++i) o[i] *= alpha;
#pragma unroll
    for (int j = 0; j < BN; ++j) {
      const float p = exp2f(fmaf(s[j], c, -msafe));
      l_run += p;
#pragma unroll
      for (int i = 0; i < SL; ++i) o[i] = fmaf(p, vs_[j][sub * SL + i], o[i]);
    }
  }
  if (!qvalid) return;
  if (MODE == kModeStats) {
    float* accp = a.acc + tj * a.acc_stride + (int64_t(b) * L + myq) * rs + int64_t(h) * D + sub * SL;
#pragma unroll
    for (int i = 0; i < SL; ++i) accp[i] = o[i];
    if (sub == 0) {
      const int64_t si = tj * a.st_stride + (int64_t(b) * a.H + h) * L + myq;
      a.m[si] = m_run;
      a.l[si] = l_run;
      a.lt[si] = l_run;  // fp32 weights are not rounded
    }
  } else {
    const float inv = 1.f / l_run;
    float* op = a.acc + (int64_t(b) * L + myq) * rs + int64_t(h) * D + sub * SL;
#pragma unroll
    for (int i = 0; i < SL; ++i) op[i] = o[i] * inv;
    if (sub == 0) {
      const int64_t si = (int64_t(b) * a.H + h) * L + myq;
      a.m[si] = (m_run + log2f(l_run)) * 0.69314718055994530942f;
    }
  }
}

template <typename E, int D, int MODE>
static void launch_mfma_mode(const FwdArgs& a, int64_t n, hipStream_t s) {
  if (a.tile_count)
    hipLaunchKernelGGL((attn_fwd_mfma<E, D, MODE, true>), dim3(unsigned(n)), dim3(64 * fwd_waves<D>()), 0, s, a);
  else
    hipLaunchKernelGGL((attn_fwd_mfma<E, D, MODE, false>), dim3(unsigned(n)), dim3(64 * fwd_waves<D>()), 0, s, a);
}

template <typename E, int D>
static hipError_t launch_mfma(FwdMode mode, const FwdArgs& a, int64_t n, hipStream_t s) {
  if (mode == kModeStats)
    launch_mfma_mode<E, D, kModeStats>(a, n, s);
  else
    launch_mfma_mode<E, D, kModeFinal>(a, n, s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_f32(FwdMode mode, const FwdArgs& a, int64_t n, hipStream_t s) {
  if (mode == kModeStats)
    hipLaunchKernelGGL((attn_fwd_f32<D, kModeStats>), dim3(unsigned(n)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attn_fwd_f32<D, kModeFinal>), dim3(unsigned(n)), dim3(256), 0, s, a);
  return hipGetLastError();
}

int fwd_rows_per_wg(cqsa_dtype dt, int d) {
  if (dt == CQSA_F32) return 32;
  switch (d) {
#define CQSA_FWD_ROWS(DD) \
  case DD:                \
    return 32 * fwd_waves<DD>();
    CQSA_FWD_ROWS(32)
    CQSA_FWD_ROWS(64)
    CQSA_FWD_ROWS(96)
    CQSA_FWD_ROWS(128)
    CQSA_FWD_ROWS(160)
    CQSA_FWD_ROWS(192)
    CQSA_FWD_ROWS(224)
    CQSA_FWD_ROWS(256)
#undef CQSA_FWD_ROWS
  }
  return 128;
}

hipError_t launch_fwd(cqsa_dtype dt, int d, FwdMode mode, const FwdArgs& a, int64_t wgs,
                      hipStream_t s) {
  if (wgs <= 0) return hipSuccess;
  if (wgs > 0x7fffffff || a.ntask < 1) return hipErrorInvalidValue;
  switch (d) {
#define CQSA_FWD_D(DD)                                                   \
  case DD:                                                               \
    if (dt == CQSA_BF16) return launch_mfma<BF16, DD>(mode, a, wgs, s);  \
    if (dt == CQSA_F16) return launch_mfma<F16, DD>(mode, a, wgs, s);    \
    return launch_f32<DD>(mode, a, wgs, s);
    CQSA_FWD_D(32)
    CQSA_FWD_D(64)
    CQSA_FWD_D(96)
    CQSA_FWD_D(128)
    CQSA_FWD_D(160)
    CQSA_FWD_D(192)
    CQSA_FWD_D(224)
    CQSA_FWD_D(256)
#undef CQSA_FWD_D
  }
  return hipErrorInvalidValue;
}

}  // namespace cqsa
