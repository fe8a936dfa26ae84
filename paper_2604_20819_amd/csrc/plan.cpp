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
//  * At level t (0-based here) with set (c_t, l_t, I_t) the chunk
//    (q + I_t[j]) mod c_t, j >= 1, carries bit s_t + (j-1), s_t being the sum
//    of (l_u - 1) over the levels above; the owner chunk q (offset I_t[0] = 0)
//    carries none.  Section 3.3 lets each depth use its own valid set.
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

LevelSet level_set(const cqsa_plan_opts& o, int32_t level) {
  if (o.n_level_sets <= 0) return LevelSet{o.c, o.l, o.interest};
  const cqsa_interest_set& s = o.level_sets[std::min(level, o.n_level_sets - 1)];
  return LevelSet{s.c, s.l, s.interest};
}

static std::string check_set(int32_t c, int32_t l, const int32_t* I) {
  if (l < 1 || l > CQSA_MAX_INTEREST) return "l must be in [1, 16]";
  if (c != l * (l - 1) + 1) return "c must equal l(l-1)+1";
  if (I[0] != 0) return "interest set must start with 0";
  for (int32_t j = 0; j < l; ++j)
    if (I[j] < 0 || I[j] >= c) return "interest offsets must lie in [0, c)";
  if (!is_perfect_difference_set(I, l, c)) return "interest set is not a perfect (c,l,1) difference set";
  return "";
}

bool in_place_fits(int64_t L, int32_t H, int32_t d, const cqsa_plan_opts& o) {
  return uint64_t(L) * uint64_t(H) * uint64_t(d) * dtype_size(o.dtype) <= 0x7fffffffull;
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
  if (d % 32 != 0 || d > 256)
    return bad(CQSA_ERR_UNSUPPORTED, "head dim must be one of 32, 64, ..., 256");
  if (o.B < 1) return bad(CQSA_ERR_INVALID_ARG, "B must be >= 1");
  if (dtype_size(o.dtype) == 0) return bad(CQSA_ERR_INVALID_ARG, "unknown dtype");
  if (o.n_level_sets < 0 || o.n_level_sets > CQSA_MAX_LEVEL_SETS)
    return bad(CQSA_ERR_INVALID_ARG, "n_level_sets must be in [0, 4]");
  if (o.n_level_sets == 0) {
    const std::string e = check_set(o.c, o.l, o.interest);
    if (!e.empty()) return bad(CQSA_ERR_INVALID_ARG, e);
  }
  for (int32_t i = 0; i < o.n_level_sets; ++i) {
    const cqsa_interest_set& ls = o.level_sets[i];
    const std::string e = check_set(ls.c, ls.l, ls.interest);
    if (!e.empty()) return bad(CQSA_ERR_INVALID_ARG, "level set " + std::to_string(i) + ": " + e);
  }
  if (o.depth < -1) return bad(CQSA_ERR_INVALID_ARG, "depth must be -1 (auto) or >= 0");
  if (o.min_depth < 0 || o.max_depth < o.min_depth)
    return bad(CQSA_ERR_INVALID_ARG, "need 0 <= min_depth <= max_depth");
  const int32_t top = o.depth >= 0 ? o.depth : o.max_depth;
  int64_t bits = 0, ntask = 1;
  for (int32_t t = 0; t < top; ++t) {
    const LevelSet ls = level_set(o, t);
    bits += ls.l - 1;
    ntask = std::min<int64_t>(ntask * ls.c, int64_t(1) << 40);
  }
  if (bits > 32) return bad(CQSA_ERR_UNSUPPORTED, "the levels' group bits exceed 32");
  if (ntask > (int64_t(1) << 20)) return bad(CQSA_ERR_UNSUPPORTED, "more than 2^20 tasks");
  if (o.n_slots < 1) return bad(CQSA_ERR_INVALID_ARG, "n_slots must be >= 1");
  if (o.inputs_on_device != 0 && o.inputs_on_device != 1)
    return bad(CQSA_ERR_INVALID_ARG, "inputs_on_device must be 0 or 1");
  if (o.acc_on_device < -1 || o.acc_on_device > 1)
    return bad(CQSA_ERR_INVALID_ARG, "acc_on_device must be -1 (auto), 0 or 1");
  if (o.tasks_per_slot < 0 || o.tasks_per_slot > kMaxContrib)
    return bad(CQSA_ERR_INVALID_ARG, "tasks_per_slot must be in [0, 32]");
  if (o.tasks_per_slot > 1 && o.acc_on_device != 1)
    return bad(CQSA_ERR_UNSUPPORTED, "tasks_per_slot > 1 needs the accumulator on the device");
  if (o.bwd_tasks_per_launch < 0 || o.bwd_tasks_per_launch > kMaxContrib)
    return bad(CQSA_ERR_INVALID_ARG, "bwd_tasks_per_launch must be in [0, 32]");
  if (o.bwd_tasks_per_launch > 1 &&
      (o.inputs_on_device != 1 || o.read_in_place == 0 || o.acc_on_device == 0))
    return bad(CQSA_ERR_UNSUPPORTED,
               "bwd_tasks_per_launch > 1 needs device-resident inputs read in place and "
               "device-resident outputs");
  if (o.read_in_place < -1 || o.read_in_place > 1)
    return bad(CQSA_ERR_INVALID_ARG, "read_in_place must be -1 (auto), 0 or 1");
  if (o.read_in_place == 1 && !o.inputs_on_device)
    return bad(CQSA_ERR_UNSUPPORTED, "read_in_place = 1 needs device-resident inputs");
  if (o.read_in_place == 1 && !in_place_fits(L, H, d, o))
    return bad(CQSA_ERR_UNSUPPORTED, "read_in_place = 1 needs L * H * d * elem < 2^31 bytes");
  if (o.with_backward && o.dtype == CQSA_F32)
    return bad(CQSA_ERR_UNSUPPORTED, "the backward supports fp16 and bf16 inputs only");
  if (o.out16 != 0 && o.out16 != 1) return bad(CQSA_ERR_INVALID_ARG, "out16 must be 0 or 1");
  if (o.out16 && o.dtype == CQSA_F32)
    return bad(CQSA_ERR_INVALID_ARG, "out16 = 1 needs fp16 or bf16 inputs");
  if (o.out16 && o.acc_on_device != 1)
    return bad(CQSA_ERR_UNSUPPORTED, "out16 = 1 needs acc_on_device = 1");
  if (o.out16 && o.with_backward)
    return bad(CQSA_ERR_UNSUPPORTED, "out16 = 1 is forward only: the backward reads the fp32 O");
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
                    uint32_t bit0, const cqsa_plan_opts& o, std::vector<int32_t>& quorum,
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
  const LevelSet ls = level_set(o, level);
  const int64_t base = Lcur / ls.c, extra = Lcur % ls.c;
  auto chunk_start = [&](int64_t u) { return u * base + std::min<int64_t>(u, extra); };
  struct Pick {
    int32_t chunk;
    uint32_t bit;
  };
  for (int32_t q = 0; q < ls.c; ++q) {
    std::vector<Pick> picks;
    for (int32_t j = 0; j < ls.l; ++j) {
      int32_t chunk = (q + ls.interest[j]) % ls.c;
      uint32_t bit = j == 0 ? 0u : (1u << (bit0 + uint32_t(j - 1)));
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
    descend(next, at, level + 1, depth, bit0 + uint32_t(ls.l - 1), o, quorum, out);
    quorum.pop_back();
  }
}

std::vector<Task> build_tasks(int64_t L, const cqsa_plan_opts& o, int32_t depth) {
  std::vector<Task> out;
  std::vector<Run> root{Run{0, 0, L, 0u}};
  std::vector<int32_t> quorum;
  descend(root, L, 0, depth, 0u, o, quorum, out);
  return out;
}

uint64_t fwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged,
                        bool stats) {
  const uint64_t rows = uint64_t(o.B) * uint64_t(Lmax) * uint64_t(g.H);
  uint64_t s = 0;
  if (staged) s += 3 * align_up(rows * g.d * dtype_size(o.dtype));
  if (stats) s += align_up(rows * g.d * 4) + 3 * align_up(rows * 4);  // acc, m, l, lt
  return s;
}

uint64_t bwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged) {
  const uint64_t rows = uint64_t(o.B) * uint64_t(Lmax) * uint64_t(g.H);
  // staged Q, K, V, dO; with host-resident gradients the task's own fp32
  // dQ, dK, dV, copied back to the host and scatter-added there
  uint64_t s = staged ? 4 * align_up(rows * g.d * dtype_size(o.dtype)) : 0;
  if (o.acc_on_device != 1) s += 3 * align_up(rows * g.d * 4);
  return s;
}

bool bwd_staged(const cqsa_plan_opts& o, int32_t depth) {
  return !o.inputs_on_device || (depth > 0 && o.read_in_place != 1);
}

bool direct_forward(const cqsa_plan_opts& o, int32_t depth) {
  return depth == 0 && o.inputs_on_device && o.acc_on_device;
}

SegmentCover segment_cover(int64_t L, const std::vector<Task>& tasks) {
  SegmentCover sc;
  sc.bounds.push_back(0);
  sc.bounds.push_back(L);
  for (const Task& t : tasks)
    for (const Run& r : t.runs) {
      sc.bounds.push_back(r.global_start);
      sc.bounds.push_back(r.global_start + r.length);
    }
  std::sort(sc.bounds.begin(), sc.bounds.end());
  sc.bounds.erase(std::unique(sc.bounds.begin(), sc.bounds.end()), sc.bounds.end());
  sc.cover.assign(sc.bounds.size() - 1, {});
  for (size_t t = 0; t < tasks.size(); ++t)
    for (const Run& r : tasks[t].runs) {
      size_t s = size_t(std::lower_bound(sc.bounds.begin(), sc.bounds.end(), r.global_start) -
                        sc.bounds.begin());
      for (; s + 1 < sc.bounds.size() && sc.bounds[s] < r.global_start + r.length; ++s)
        sc.cover[s].push_back({int32_t(t), r.local_start + (sc.bounds[s] - r.global_start)});
    }
  return sc;
}

std::vector<int64_t> fwd_slot_tasks(int64_t ntask, int32_t group_size, int32_t n_slots) {
  const int64_t g = std::max<int64_t>(1, group_size);
  const int64_t ngroup = std::max<int64_t>(1, (ntask + g - 1) / g);
  const int64_t ns = std::min<int64_t>(std::max(1, n_slots), ngroup);
  std::vector<int64_t> cap(ns, 0);
  for (int64_t k = 0; k < ngroup; ++k)
    cap[k % ns] = std::max(cap[k % ns], std::min(g, std::max<int64_t>(0, ntask - k * g)));
  for (int64_t& c : cap) c = std::max<int64_t>(1, c);
  return cap;
}

int64_t fwd_subslots(int64_t ntask, int32_t group_size, int32_t n_slots) {
  int64_t n = 0;
  for (int64_t c : fwd_slot_tasks(ntask, group_size, n_slots)) n += c;
  return n;
}

std::vector<Group> make_groups(int64_t ntask, int32_t group_size) {
  std::vector<Group> gs;
  const int64_t g = std::max<int64_t>(1, group_size);
  for (int64_t t0 = 0; t0 < std::max<int64_t>(1, ntask); t0 += g) {
    Group gr;
    gr.task0 = t0;
    gr.count = std::min<int64_t>(g, ntask - t0);
    gs.push_back(gr);
  }
  gs.back().final = true;
  return gs;
}

namespace {

// Stable permutation of 0..n-1 by descending count.
std::vector<int32_t> longest_first(const std::vector<int64_t>& count) {
  std::vector<int32_t> ord(count.size());
  for (size_t i = 0; i < ord.size(); ++i) ord[i] = int32_t(i);
  std::stable_sort(ord.begin(), ord.end(),
                   [&](int32_t a, int32_t b) { return count[size_t(a)] > count[size_t(b)]; });
  return ord;
}

}  // namespace

// Prefix counts of each distinct value of `vals` (a task's block ANDs take a
// few values: the group-bit patterns of its runs and of blocks that straddle
// runs).  count(i, p) = positions before p holding value v[i].
struct ValuePrefix {
  std::vector<uint32_t> v;
  std::vector<std::vector<int32_t>> pre;
  explicit ValuePrefix(const std::vector<uint32_t>& vals) {
    for (uint32_t x : vals)
      if (std::find(v.begin(), v.end(), x) == v.end()) v.push_back(x);
    pre.assign(v.size(), std::vector<int32_t>(vals.size() + 1, 0));
    for (size_t i = 0; i < v.size(); ++i)
      for (size_t p = 0; p < vals.size(); ++p) pre[i][p + 1] = pre[i][p] + (vals[p] == v[i] ? 1 : 0);
  }
  // positions in [lo, hi) whose value shares no bit with m
  int64_t disjoint(uint32_t m, int64_t lo, int64_t hi) const {
    int64_t n = 0;
    if (hi <= lo) return 0;
    for (size_t i = 0; i < v.size(); ++i)
      if ((v[i] & m) == 0u) n += pre[i][size_t(hi)] - pre[i][size_t(lo)];
    return n;
  }
};

std::vector<int32_t> query_strip_order(const Task& t, bool causal, int32_t rows) {
  const int64_t L = t.L_local, nb = int64_t(t.blk_and.size());
  const int64_t ns = (L + rows - 1) / rows;
  const ValuePrefix vp(t.blk_and);  // 64-key tile k is block k
  std::vector<int64_t> live(size_t(ns), 0);
  for (int64_t s = 0; s < ns; ++s) {
    const int64_t last = std::min(L, (s + 1) * rows) - 1;
    uint32_t qand = 0xFFFFFFFFu;  // AND over the strip's blocks
    for (int64_t b = s * rows / kBlock; b <= last / kBlock; ++b) qand &= t.blk_and[size_t(b)];
    live[size_t(s)] = vp.disjoint(qand, 0, causal ? last / kBlock + 1 : nb);
  }
  return longest_first(live);
}

std::vector<int32_t> key_strip_order(const Task& t, bool causal, int32_t rows) {
  const int64_t L = t.L_local, nq = (L + 31) / 32;
  const int64_t ns = (L + rows - 1) / rows;
  std::vector<uint32_t> tile_and(static_cast<size_t>(nq));  // 32-query tile q lies in block q / 2
  for (int64_t q = 0; q < nq; ++q) tile_and[size_t(q)] = t.blk_and[size_t(q / 2)];
  const ValuePrefix vp(tile_and);
  std::vector<int64_t> live(size_t(ns), 0);
  for (int64_t s = 0; s < ns; ++s) {
    const int64_t first = s * rows, last = std::min<int64_t>(L, (s + 1) * rows) - 1;
    uint32_t kand = 0xFFFFFFFFu;  // AND over the strip's blocks
    for (int64_t b = first / kBlock; b <= last / kBlock; ++b) kand &= t.blk_and[size_t(b)];
    // causally, tile q is dead when its last query, 32 q + 31, precedes the
    // strip's first key (a multiple of 32): the first live tile is first / 32
    const int64_t q0 = causal ? first / 32 : 0;
    live[size_t(s)] = vp.disjoint(kand, q0, nq);
  }
  return longest_first(live);
}

void fwd_tile_decisions(const Task& t, bool causal, int32_t rows, int64_t out[3]) {
  const int64_t L = t.L_local, nkt = (L + kBlock - 1) / kBlock;
  const int64_t ns = (L + rows - 1) / rows;
  std::vector<int64_t> visited;
  for (int64_t s = 0; s < ns; ++s) {
    const int64_t first = s * rows, last = std::min(L, first + rows) - 1;
    uint32_t qand = 0xFFFFFFFFu;  // AND over the work group's blocks
    for (int64_t b = first / kBlock; b <= last / kBlock; ++b) qand &= t.blk_and[size_t(b)];
    // key tile k is block k: live for the work group unless causally past its
    // last query or sharing a bit of the AND with it
    visited.clear();
    for (int64_t k = 0; k < nkt; ++k)
      if (!(causal && k * kBlock > last) && (qand & t.blk_and[size_t(k)]) == 0u) visited.push_back(k);
    for (int64_t q0 = first; q0 <= last; q0 += 32) {
      const int64_t q1 = std::min(q0 + 31, L - 1);
      const uint32_t wor = t.blk_or[size_t(q0 / kBlock)], wand = t.blk_and[size_t(q0 / kBlock)];
      for (int64_t k : visited) {
        const int64_t k0 = k * kBlock, k1 = std::min(k0 + kBlock - 1, L - 1);
        if ((wand & t.blk_and[size_t(k)]) != 0u || (causal && k0 > q1))
          ++out[0];
        else if ((wor & t.blk_or[size_t(k)]) == 0u && (!causal || k1 <= q0) && k0 + kBlock <= L)
          ++out[1];
        else
          ++out[2];
      }
    }
  }
}

void kv_tile_decisions(const Task& t, bool causal, int32_t rows, int32_t qtile, int64_t out[3]) {
  const int64_t L = t.L_local, nqt = (L + qtile - 1) / qtile;
  const int64_t per_block = kBlock / qtile;  // query tiles per summary block
  const int64_t ns = (L + rows - 1) / rows;
  std::vector<int64_t> visited;
  for (int64_t s = 0; s < ns; ++s) {
    const int64_t first = s * rows, last = std::min(L, first + rows) - 1;
    uint32_t kand = 0xFFFFFFFFu;  // AND over the work group's blocks
    for (int64_t b = first / kBlock; b <= last / kBlock; ++b) kand &= t.blk_and[size_t(b)];
    // query tile q: live for the work group unless causally wholly before its
    // first key or sharing a bit of the AND with it
    visited.clear();
    for (int64_t q = 0; q < nqt; ++q)
      if (!(causal && q * qtile + qtile - 1 < first) && (kand & t.blk_and[size_t(q / per_block)]) == 0u)
        visited.push_back(q);
    for (int64_t k0 = first; k0 <= last; k0 += 32) {
      const int64_t k1 = std::min(k0 + 31, L - 1);
      const uint32_t wor = t.blk_or[size_t(k0 / kBlock)], wand = t.blk_and[size_t(k0 / kBlock)];
      for (int64_t q : visited) {
        const int64_t q0 = q * qtile;
        const uint32_t qor = t.blk_or[size_t(q / per_block)], qand = t.blk_and[size_t(q / per_block)];
        if ((wand & qand) != 0u || (causal && q0 + qtile - 1 < k0))
          ++out[0];
        else if ((wor & qor) == 0u && (!causal || q0 >= k1))
          ++out[1];
        else
          ++out[2];
      }
    }
  }
}

void pack_image(const std::vector<Task>& tasks, const SegmentCover& sc, int32_t H, bool causal,
                int32_t fwd_rows, int32_t dq_rows, int32_t kv_rows, std::vector<Group>* groups,
                std::vector<uint8_t>* image, std::vector<TableOffsets>* offs) {
  std::vector<uint8_t>& im = *image;
  im.clear();
  offs->clear();
  auto reserve = [&](uint64_t bytes) {
    const uint64_t at = im.size();
    im.resize(align_up(at + bytes), 0);
    return at;
  };
  const uint64_t hdr = reserve(tasks.size() * sizeof(DevTask));
  for (size_t t = 0; t < tasks.size(); ++t) {
    const Task& k = tasks[t];
    TableOffsets o;
    o.runs = reserve(k.runs.size() * sizeof(DevRun));
    for (size_t i = 0; i < k.runs.size(); ++i) {
      DevRun r{k.runs[i].local_start, k.runs[i].global_start, k.runs[i].length, k.runs[i].bits, 0u};
      std::memcpy(im.data() + o.runs + i * sizeof(DevRun), &r, sizeof(r));
    }
    // block records: summaries and the block row table for kernels that
    // read the caller's tensors in place
    const size_t nb = k.blk_or.size();
    o.blocks = reserve(nb * sizeof(DevBlock));
    size_t ri = 0;
    for (size_t i = 0; i < nb; ++i) {
      const int64_t t0 = int64_t(i) * kBlock;
      const int64_t t1 = std::min<int64_t>(t0 + kBlock, k.L_local);  // one past the last
      while (k.runs[ri].local_start + k.runs[ri].length <= t0) ++ri;
      const Run& r = k.runs[ri];
      const int32_t row = t1 <= r.local_start + r.length
                              ? int32_t(r.global_start + (t0 - r.local_start))
                              : kNoRow;
      const DevBlock x{k.blk_or[i], k.blk_and[i], row, 0u};
      std::memcpy(im.data() + o.blocks + i * sizeof(DevBlock), &x, sizeof(x));
    }
    // strip launch orders, longest first: the forward's strips, dQ's and dK/dV's
    auto put = [&](const std::vector<int32_t>& v) {
      const uint64_t at = reserve(v.size() * 4);
      if (!v.empty()) std::memcpy(im.data() + at, v.data(), v.size() * 4);
      return at;
    };
    o.qorder = put(query_strip_order(k, causal, fwd_rows));
    o.dqorder = put(query_strip_order(k, causal, dq_rows));
    o.korder = put(key_strip_order(k, causal, kv_rows));
    DevTask d{k.L_local, int64_t(o.runs), int64_t(o.qorder), int64_t(o.dqorder),
              int64_t(o.korder), int64_t(o.blocks), int32_t(k.runs.size()), 0};
    std::memcpy(im.data() + hdr + t * sizeof(DevTask), &d, sizeof(d));
    offs->push_back(o);
  }
  pack_groups(sc, H, groups, image);
}

void pack_groups(const SegmentCover& sc, int32_t H, std::vector<Group>* groups,
                 std::vector<uint8_t>* image) {
  std::vector<uint8_t>& im = *image;
  auto reserve = [&](uint64_t bytes) {
    const uint64_t at = im.size();
    im.resize(align_up(at + bytes), 0);
    return at;
  };
  const size_t nseg = sc.cover.size();
  for (Group& g : *groups) {
    const int32_t t0 = int32_t(g.task0), t1 = int32_t(g.task0 + g.count);
    std::vector<DevSeg> segs;
    std::vector<DevContrib> cons;
    int64_t blk = 0;
    for (size_t s = 0; s < nseg; ++s) {
      const auto& cv = sc.cover[s];
      const int32_t c_off = int32_t(cons.size());
      bool earlier = false;
      for (const auto& e : cv) {
        if (e.first < t0) earlier = true;
        if (e.first >= t0 && e.first < t1) cons.push_back(DevContrib{e.second, e.first - t0, 0});
      }
      const int32_t n_c = int32_t(cons.size()) - c_off;
      if (n_c == 0 && !g.final) continue;
      const int64_t len = sc.bounds[s + 1] - sc.bounds[s];
      segs.push_back(DevSeg{sc.bounds[s], len, blk, c_off, n_c, earlier ? 1 : 0, 0});
      blk += (len * H + kCombinePairs - 1) / kCombinePairs;
    }
    g.n_seg = int32_t(segs.size());
    g.blocks = blk;
    g.seg_off = reserve(segs.size() * sizeof(DevSeg));
    if (!segs.empty()) std::memcpy(im.data() + g.seg_off, segs.data(), segs.size() * sizeof(DevSeg));
    g.contrib_off = reserve(cons.size() * sizeof(DevContrib));
    if (!cons.empty())
      std::memcpy(im.data() + g.contrib_off, cons.data(), cons.size() * sizeof(DevContrib));
  }
}

bool bwd_batchable(const cqsa_plan_opts& o, int32_t depth) {
  return depth > 0 && o.inputs_on_device && o.read_in_place == 1 && o.acc_on_device == 1;
}

uint64_t bwd_local_task_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax) {
  return 3 * align_up(uint64_t(o.B) * uint64_t(Lmax) * uint64_t(g.H) * uint64_t(g.d) * 4);
}

Footprint footprint(const Geometry& g, const cqsa_plan_opts& o, int32_t depth,
                    const std::vector<Task>& tasks, int32_t group_size, uint64_t image_bytes,
                    int32_t bwd_group) {
  Footprint f;
  int64_t Lmax = 0;
  for (const Task& t : tasks) Lmax = std::max(Lmax, t.L_local);
  const int64_t ntask = int64_t(tasks.size());
  f.group_size = std::max<int32_t>(1, group_size);
  f.groups = (ntask + f.group_size - 1) / f.group_size;
  const uint64_t tok = uint64_t(o.B) * uint64_t(g.L) * uint64_t(g.H);
  const uint64_t in_bytes = align_up(tok * g.d * dtype_size(o.dtype));
  const uint64_t f32_full = align_up(tok * g.d * 4);
  const uint64_t stat_full = align_up(tok * 4);
  const bool direct = direct_forward(o, depth);
  // caller's O and LSE; with out16 the caller's O is 16-bit and the fp32
  // result sits in the workspace
  f.resident_fwd = (o.inputs_on_device ? 3 * in_bytes : 0) +
                   (o.acc_on_device ? f32_full + stat_full + (o.out16 ? in_bytes : 0) : 0);
  // backward: Q, K, V, dO follow the inputs' residency; O, LSE, dQ, dK, dV
  // the accumulator's
  f.resident_bwd = (o.inputs_on_device ? 4 * in_bytes : 0) +
                   (o.acc_on_device == 1 ? f32_full + stat_full + 3 * f32_full : 0);
  // slot i holds as many task sub-slots (each sized for the longest task) as
  // the largest group that uses it (groups k with k % n_slots == i)
  const bool staged = o.read_in_place != 1;
  f.slot_fwd = direct ? 0 : fwd_slot_bytes(g, o, Lmax, staged, true);
  f.slot_bwd = bwd_slot_bytes(g, o, Lmax, bwd_staged(o, depth));
  // running row sums l and lt, needed while more than one group merges on device
  f.global_fwd = (o.acc_on_device && !direct && f.groups > 1) ? 2 * stat_full : 0;
  // D = rowsum(dO * O), and a device copy of a host-resident LSE
  f.global_bwd = stat_full + (o.acc_on_device == 1 ? 0 : stat_full);
  // task-local gradients of one backward launch group of several tasks
  f.bwd_group_size = std::max<int32_t>(1, bwd_group);
  f.bwd_local = f.bwd_group_size > 1 ? uint64_t(f.bwd_group_size) * bwd_local_task_bytes(g, o, Lmax)
                                     : 0;
  f.tables = align_up(image_bytes);
  const uint64_t subslots_fwd = uint64_t(fwd_subslots(ntask, f.group_size, o.n_slots));
  const uint64_t slots_bwd = uint64_t(std::min<int64_t>(o.n_slots, ntask));
  uint64_t peak_fwd = f.resident_fwd + subslots_fwd * f.slot_fwd + f.global_fwd + f.tables;
  uint64_t peak_bwd = o.with_backward
                          ? f.resident_bwd + slots_bwd * f.slot_bwd + f.global_bwd + f.bwd_local +
                                f.tables
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
