// CQS task planner (host only).
//
// Builds the c**depth subsequence tasks of BuildSubseq (Alg. 3) as run lists,
// derives the per-token group bits of the CQS mask (Section 3.3; App. A.2),
// the 64-token block summaries (App. A.2), the 128x128 tile census, and the
// modelled device footprint used by the depth rule of Section 3.4.
//
// Readings fixed here (the paper leaves them open):
//  * BalancedChunkLayout(L, c) gives the first L mod c chunks one extra token.
//  * A task's chunks are gathered in ascending chunk order, so local order is
//    global order and causal masking composes by conjunction (App. A.3).
//  * At level t (0-based here) the chunk (q + I[j]) mod c, j >= 1, carries bit
//    t*(l-1) + (j-1); the owner chunk q (offset I[0] = 0) carries none.
#include <algorithm>
#include <cstring>
#include <string>

#include "plan.hpp"

namespace cqsa {

size_t dtype_size(cqsa_dtype t) {
  switch (t) {
    case CQSA_F32: return 4;
    case CQSA_F16: return 2;
    case CQSA_BF16: return 2;
  }
  return 0;
}

bool is_perfect_difference_set(const int32_t* I, int32_t l, int32_t c) {
  if (c <= 0 || l <= 0) return false;
  std::vector<int32_t> hits(c, 0);
  for (int32_t a = 0; a < l; ++a)
    for (int32_t b = 0; b < l; ++b) {
      if (a == b) continue;
      int32_t diff = ((I[a] - I[b]) % c + c) % c;
      hits[diff]++;
    }
  if (hits[0] != 0) return false;
  for (int32_t r = 1; r < c; ++r)
    if (hits[r] != 1) return false;
  return true;
}

static int64_t ipow(int64_t b, int32_t e) {
  int64_t r = 1;
  for (int32_t i = 0; i < e; ++i) {
    r *= b;
    if (r > (int64_t(1) << 40)) return r;
  }
  return r;
}

cqsa_status validate_plan_args(int64_t L, int32_t H, int32_t d, const cqsa_plan_opts& o,
                               std::string* err) {
  auto bad = [&](cqsa_status s, const std::string& m) {
    *err = m;
    return s;
  };
  if (L < 1) return bad(CQSA_ERR_INVALID_ARG, "L must be >= 1");
  if (L > (int64_t(1) << 31) - 1) return bad(CQSA_ERR_UNSUPPORTED, "L must be < 2^31");
  if (H < 1) return bad(CQSA_ERR_INVALID_ARG, "H must be >= 1");
  if (d < 1) return bad(CQSA_ERR_INVALID_ARG, "d must be >= 1");
  if (d != 64 && d != 128) return bad(CQSA_ERR_UNSUPPORTED, "head dim must be 64 or 128");
  if (o.B < 1) return bad(CQSA_ERR_INVALID_ARG, "B must be >= 1");
  if (dtype_size(o.dtype) == 0) return bad(CQSA_ERR_INVALID_ARG, "unknown dtype");
  if (o.l < 1 || o.l > CQSA_MAX_INTEREST) return bad(CQSA_ERR_INVALID_ARG, "l must be in [1, 16]");
  if (o.c != o.l * (o.l - 1) + 1) return bad(CQSA_ERR_INVALID_ARG, "c must equal l(l-1)+1");
  if (o.interest[0] != 0) return bad(CQSA_ERR_INVALID_ARG, "interest set must start with 0");
  for (int32_t j = 0; j < o.l; ++j)
    if (o.interest[j] < 0 || o.interest[j] >= o.c)
      return bad(CQSA_ERR_INVALID_ARG, "interest offsets must lie in [0, c)");
  if (!is_perfect_difference_set(o.interest, o.l, o.c))
    return bad(CQSA_ERR_INVALID_ARG, "interest set is not a perfect (c,l,1) difference set");
  if (o.depth < -1) return bad(CQSA_ERR_INVALID_ARG, "depth must be -1 (auto) or >= 0");
  if (o.min_depth < 0 || o.max_depth < o.min_depth)
    return bad(CQSA_ERR_INVALID_ARG, "need 0 <= min_depth <= max_depth");
  int32_t top = o.depth >= 0 ? o.depth : o.max_depth;
  if (int64_t(top) * (o.l - 1) > 32)
    return bad(CQSA_ERR_UNSUPPORTED, "depth*(l-1) group bits exceed 32");
  if (ipow(o.c, top) > (int64_t(1) << 20))
    return bad(CQSA_ERR_UNSUPPORTED, "more than 2^20 tasks");
  if (o.n_slots < 1) return bad(CQSA_ERR_INVALID_ARG, "n_slots must be >= 1");
  if (o.inputs_on_device != 0 && o.inputs_on_device != 1)
    return bad(CQSA_ERR_INVALID_ARG, "inputs_on_device must be 0 or 1");
  if (o.acc_on_device != 0 && o.acc_on_device != 1)
    return bad(CQSA_ERR_INVALID_ARG, "acc_on_device must be 0 or 1");
  if (o.with_backward && (!o.inputs_on_device || !o.acc_on_device))
    return bad(CQSA_ERR_UNSUPPORTED, "the backward supports device-resident tensors only");
  if (o.with_backward && o.dtype == CQSA_F32)
    return bad(CQSA_ERR_UNSUPPORTED, "the backward supports fp16 and bf16 inputs only");
  return CQSA_OK;
}

// Append the part of `cur` covering local [a, b) to `out`, relabelled to start
// at local `at`, with `bit` OR-ed into every token.
static void slice_runs(const std::vector<Run>& cur, int64_t a, int64_t b, int64_t at,
                       uint32_t bit, std::vector<Run>& out) {
  for (const Run& r : cur) {
    int64_t rs = r.local_start, re = r.local_start + r.length;
    int64_t lo = std::max(a, rs), hi = std::min(b, re);
    if (lo >= hi) continue;
    Run n;
    n.local_start = at + (lo - a);
    n.global_start = r.global_start + (lo - rs);
    n.length = hi - lo;
    n.bits = r.bits | bit;
    // coalesce with the previous run when globally contiguous with equal bits
    if (!out.empty()) {
      Run& p = out.back();
      if (p.global_start + p.length == n.global_start && p.bits == n.bits &&
          p.local_start + p.length == n.local_start) {
        p.length += n.length;
        continue;
      }
    }
    out.push_back(n);
  }
}

static void finish_task(Task& t) {
  t.abi_runs.clear();
  for (const Run& r : t.runs) t.abi_runs.push_back(cqsa_run{r.global_start, r.length, r.bits});
  int64_t nb = (t.L_local + kBlock - 1) / kBlock;
  t.blk_or.assign(nb, 0u);
  t.blk_and.assign(nb, 0xFFFFFFFFu);
  for (const Run& r : t.runs) {
    int64_t s = r.local_start, e = r.local_start + r.length;
    for (int64_t b = s / kBlock; b * kBlock < e; ++b) {
      t.blk_or[b] |= r.bits;
      t.blk_and[b] &= r.bits;
    }
  }
}

static void descend(const std::vector<Run>& cur, int64_t Lcur, int32_t level, int32_t depth,
                    const cqsa_plan_opts& o, std::vector<int32_t>& quorum,
                    std::vector<Task>& out) {
  if (level == depth) {
    Task t;
    t.quorum = quorum;
    t.L_local = Lcur;
    t.runs = cur;
    finish_task(t);
    out.push_back(std::move(t));
    return;
  }
  const int64_t base = Lcur / o.c, extra = Lcur % o.c;
  auto chunk_start = [&](int64_t u) { return u * base + std::min<int64_t>(u, extra); };
  struct Pick {
    int32_t chunk;
    uint32_t bit;
  };
  for (int32_t q = 0; q < o.c; ++q) {
    std::vector<Pick> picks;
    for (int32_t j = 0; j < o.l; ++j) {
      int32_t chunk = (q + o.interest[j]) % o.c;
      uint32_t bit = j == 0 ? 0u : (1u << (level * (o.l - 1) + (j - 1)));
      picks.push_back({chunk, bit});
    }
    std::sort(picks.begin(), picks.end(),
              [](const Pick& x, const Pick& y) { return x.chunk < y.chunk; });
    std::vector<Run> next;
    int64_t at = 0;
    for (const Pick& p : picks) {
      int64_t a = chunk_start(p.chunk), b = chunk_start(p.chunk + 1);
      slice_runs(cur, a, b, at, p.bit, next);
      at += b - a;
    }
    quorum.push_back(q);
    descend(next, at, level + 1, depth, o, quorum, out);
    quorum.pop_back();
  }
}

std::vector<Task> build_tasks(int64_t L, const cqsa_plan_opts& o, int32_t depth) {
  std::vector<Task> out;
  std::vector<Run> root{Run{0, 0, L, 0u}};
  std::vector<int32_t> quorum;
  descend(root, L, 0, depth, o, quorum, out);
  return out;
}

uint64_t fwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged,
                        bool stats) {
  const uint64_t rows = uint64_t(o.B) * uint64_t(Lmax) * uint64_t(g.H);
  uint64_t s = 0;
  if (staged) s += 3 * align_up(rows * g.d * dtype_size(o.dtype));
  if (stats) s += align_up(rows * g.d * 4) + 2 * align_up(rows * 4);
  return s;
}

uint64_t bwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged) {
  const uint64_t rows = uint64_t(o.B) * uint64_t(Lmax) * uint64_t(g.H);
  return staged ? 4 * align_up(rows * g.d * dtype_size(o.dtype)) : 0;
}

// Per task on the device: runs (32 bytes each) and two 32-bit words per block.
uint64_t table_bytes(const std::vector<Task>& tasks) {
  uint64_t s = 0;
  for (const Task& t : tasks)
    s += align_up(t.runs.size() * 32) + 2 * align_up(t.blk_or.size() * 4);
  return s;
}

void pack_tables(const std::vector<Task>& tasks, std::vector<uint8_t>* image,
                 std::vector<TableOffsets>* offs) {
  image->assign(table_bytes(tasks), 0);
  offs->clear();
  uint64_t at = 0;
  for (const Task& t : tasks) {
    TableOffsets o;
    o.runs = at;
    for (size_t i = 0; i < t.runs.size(); ++i) {
      int64_t rec[4] = {t.runs[i].local_start, t.runs[i].global_start, t.runs[i].length,
                        int64_t(t.runs[i].bits)};
      std::memcpy(image->data() + at + 32 * i, rec, 32);
    }
    at += align_up(t.runs.size() * 32);
    o.blk_or = at;
    std::memcpy(image->data() + at, t.blk_or.data(), t.blk_or.size() * 4);
    at += align_up(t.blk_or.size() * 4);
    o.blk_and = at;
    std::memcpy(image->data() + at, t.blk_and.data(), t.blk_and.size() * 4);
    at += align_up(t.blk_and.size() * 4);
    offs->push_back(o);
  }
}

Footprint footprint(const Geometry& g, const cqsa_plan_opts& o, int32_t depth,
                    const std::vector<Task>& tasks) {
  Footprint f;
  int64_t Lmax = 0;
  for (const Task& t : tasks) Lmax = std::max(Lmax, t.L_local);
  const uint64_t tok = uint64_t(o.B) * uint64_t(g.L) * uint64_t(g.H);
  const uint64_t in_bytes = align_up(tok * g.d * dtype_size(o.dtype));
  const uint64_t f32_full = align_up(tok * g.d * 4);
  const uint64_t stat_full = align_up(tok * 4);
  f.resident_fwd = (o.inputs_on_device ? 3 * in_bytes : 0) +
                   (o.acc_on_device ? f32_full + stat_full : 0);
  f.resident_bwd = 4 * in_bytes + f32_full + stat_full + 3 * f32_full;
  const bool staged_fwd = depth > 0 || !o.inputs_on_device;
  const bool stats_fwd = depth > 0 || !o.acc_on_device;
  f.slot_fwd = fwd_slot_bytes(g, o, Lmax, staged_fwd, stats_fwd);
  f.slot_bwd = bwd_slot_bytes(g, o, Lmax, depth > 0);
  f.global_fwd = (o.acc_on_device && depth > 0) ? stat_full : 0;   // global row sums l
  f.global_bwd = stat_full;                                         // D = rowsum(dO * O)
  f.tables = table_bytes(tasks);
  const uint64_t slots = uint64_t(std::min<int64_t>(o.n_slots, int64_t(tasks.size())));
  uint64_t peak_fwd = f.resident_fwd + slots * f.slot_fwd + f.global_fwd + f.tables;
  uint64_t peak_bwd = o.with_backward
                          ? f.resident_bwd + slots * f.slot_bwd + f.global_bwd + f.tables
                          : 0;
  f.peak = std::max(peak_fwd, peak_bwd);
  return f;
}

void tile_census(const std::vector<Task>& tasks, int64_t out[3]) {
  const int per = kTile / kBlock;
  int64_t full = 0, clear = 0, mixed = 0;
  for (const Task& t : tasks) {
    const int64_t nb = int64_t(t.blk_or.size());
    const int64_t nt = (nb + per - 1) / per;
    std::vector<uint32_t> tor(nt, 0u), tand(nt, 0xFFFFFFFFu);
    for (int64_t b = 0; b < nb; ++b) {
      tor[b / per] |= t.blk_or[b];
      tand[b / per] &= t.blk_and[b];
    }
    for (int64_t r = 0; r < nt; ++r)
      for (int64_t s = 0; s <= r; ++s) {
        if (tand[r] & tand[s])
          ++full;
        else if ((tor[r] & tor[s]) == 0)
          ++clear;
        else
          ++mixed;
      }
  }
  out[0] = full;
  out[1] = clear;
  out[2] = mixed;
}

}  // namespace cqsa
