// Internal plan representation shared by the planner, the runtime and the
// C-ABI layer.  Not part of the public ABI (see include/cqsa.h).
#pragma once

#include <cstdint>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "cqsa.h"
#include "records.hpp"

namespace cqsa {

constexpr int kBlock = 64;   // tokens per block summary (App. A.2)
constexpr int kTile = 128;   // census tile edge (App. A.2)
// 128-query strips one forward launch should offer: two waves of the
// MI355X's resident 4-wave inner-kernel work groups (256 CUs x 2).
constexpr int64_t kLaunchWgs = 1024;

// One maximal run of a task: local tokens [local_start, local_start+length)
// are global tokens [global_start, global_start+length), all with `bits`.
struct Run {
  int64_t local_start;
  int64_t global_start;
  int64_t length;
  uint32_t bits;
};

struct Task {
  std::vector<int32_t> quorum;  // q_1..q_depth
  int64_t L_local = 0;
  std::vector<Run> runs;         // ascending local == ascending global
  std::vector<cqsa_run> abi_runs;
  // per 64-token local block
  std::vector<uint32_t> blk_or, blk_and;
};

// Offsets of one task's tables inside the packed table image (bytes).
struct TableOffsets {
  uint64_t runs = 0;    // DevRun[n_runs]: {local_start, global_start, length, bits, pad}
  uint64_t qorder = 0;  // int32[n_strips] forward query strips, longest first
  uint64_t dqorder = 0; // int32[n_strips] dQ query strips, longest first
  uint64_t korder = 0;  // int32[n_strips] key strips, longest first
  uint64_t blocks = 0;  // DevBlock[n_blocks]: block OR, AND and row (records.hpp, kNoRow)
};

// A launch group: tasks [task0, task0 + count) are staged into one slot,
// run by one inner-kernel launch and merged by one combine launch.
struct Group {
  int64_t task0 = 0, count = 0;
  uint64_t seg_off = 0;      // DevSeg[n_seg] in the packed image
  uint64_t contrib_off = 0;  // DevContrib[..] in the packed image
  int32_t n_seg = 0;
  int64_t blocks = 0;        // combine work groups per batch element
  bool final = false;        // last group: the combine writes O and LSE
};

// Elementary global segments: the cuts of every task's runs.  cover[s] lists
// (task, local token of the segment's first token) in ascending task order.
struct SegmentCover {
  std::vector<int64_t> bounds;  // segment s is [bounds[s], bounds[s + 1])
  std::vector<std::vector<std::pair<int32_t, int64_t>>> cover;
};

// Everything the runtime allocates for one call, in bytes.
struct Footprint {
  uint64_t resident_fwd = 0;   // caller tensors on device during the forward
  uint64_t resident_bwd = 0;   // caller tensors on device during the backward
  uint64_t slot_fwd = 0;       // one forward task sub-slot (staged inputs + statistics)
  uint64_t slot_bwd = 0;       // one backward staging slot (inputs)
  uint64_t global_fwd = 0;     // forward device workspace independent of slots
  uint64_t global_bwd = 0;     // backward device workspace independent of slots
  uint64_t tables = 0;         // packed plan image (task and merge tables)
  uint64_t peak = 0;           // modelled peak device bytes
  int32_t group_size = 1;      // tasks per forward staging slot
  int64_t groups = 1;          // forward launch groups
  int32_t bwd_group_size = 1;  // backward tasks per dQ and dK/dV launch
  uint64_t bwd_local = 0;      // task-local gradients of one backward launch group
};

struct Geometry {
  int64_t L;
  int32_t H, d, causal;
};

}  // namespace cqsa

struct cqsa_plan_s {
  cqsa::Geometry g;
  uint64_t budget;
  cqsa_plan_opts opts;
  int32_t depth;
  int64_t max_L_local;
  std::vector<cqsa::Task> tasks;
  cqsa::Footprint fp;
  // packed plan image, uploaded to the device by every call: DevTask[ntask]
  // at offset 0, then every task's tables, then every group's merge tables
  std::vector<uint8_t> packed;
  std::vector<cqsa::TableOffsets> table_off;
  std::vector<cqsa::Group> groups;
  // backward launch groups (bwd_batched plans only; merge tables in `packed`)
  std::vector<cqsa::Group> bwd_groups;
  // lazily computed census
  mutable std::once_flag census_once;
  mutable int64_t census[3] = {0, 0, 0};
  // OOM guardrail (Sec. 3.4): the fallback plans that last succeeded after
  // an allocation failure under an automatic depth, reused by later calls.
  // Shared, so a call keeps its fallback alive while another call on the
  // same plan replaces the cached one.
  mutable std::mutex guard_mu;
  mutable std::shared_ptr<const cqsa_plan_s> guard_fwd, guard_bwd;
};

namespace cqsa {

size_t dtype_size(cqsa_dtype t);

// True when a [L, H, d] slice of the inputs spans under 2^31 bytes, so the
// kernels can address the caller's tensors in place with 32-bit offsets.
bool in_place_fits(int64_t L, int32_t H, int32_t d, const cqsa_plan_opts& o);

// Validates options and geometry; returns CQSA_OK or sets the error text.
cqsa_status validate_plan_args(int64_t L, int32_t H, int32_t d, const cqsa_plan_opts& o,
                               std::string* err);

// Builds the c**depth tasks of BuildSubseq with ascending chunk order.
// Interest set of level `level` (0-based): (c, l, interest), or the opts'
// per-level set (the last one repeating below the given levels).
struct LevelSet {
  int32_t c, l;
  const int32_t* interest;
};
LevelSet level_set(const cqsa_plan_opts& o, int32_t level);
std::vector<Task> build_tasks(int64_t L, const cqsa_plan_opts& o, int32_t depth);

// Footprint of running `tasks` under `o` with `group_size` tasks per forward
// slot, `bwd_group` tasks per backward launch and a plan image of
// `image_bytes` (mirrors the runtime's allocations).
Footprint footprint(const Geometry& g, const cqsa_plan_opts& o, int32_t depth,
                    const std::vector<Task>& tasks, int32_t group_size, uint64_t image_bytes,
                    int32_t bwd_group = 1);

// Whether the backward can run several tasks per launch with task-local
// gradients and a gather-merge: inputs read in place, device-resident
// outputs and gradients, depth >= 1.
bool bwd_batchable(const cqsa_plan_opts& o, int32_t depth);
// Bytes of one backward task's local dQ, dK, dV (each sized for the longest task).
uint64_t bwd_local_task_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax);

// True when the forward writes O directly from one undecomposed launch.
bool direct_forward(const cqsa_plan_opts& o, int32_t depth);

SegmentCover segment_cover(int64_t L, const std::vector<Task>& tasks);

// Task sub-slots of each forward staging slot: slot i serves the groups
// k with k % S == i (S = min(n_slots, groups)) and holds the largest of them.
std::vector<int64_t> fwd_slot_tasks(int64_t ntask, int32_t group_size, int32_t n_slots);
int64_t fwd_subslots(int64_t ntask, int32_t group_size, int32_t n_slots);

// Consecutive groups of `group_size` tasks (the last one may be shorter).
std::vector<Group> make_groups(int64_t ntask, int32_t group_size);

void tile_census(const std::vector<Task>& tasks, int64_t out[3]);

bool is_perfect_difference_set(const int32_t* I, int32_t l, int32_t c);

// Runtime workspace layout helpers (bytes), shared with the footprint model.
uint64_t fwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged,
                        bool stats);
uint64_t bwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged);
// Whether the backward gathers each task's Q, K, V, dO into a staging slot
// (host-resident inputs always; device-resident ones unless read in place or
// undecomposed).
bool bwd_staged(const cqsa_plan_opts& o, int32_t depth);
// Packs the plan image: the DevTask records, every task's runs and block
// summaries, and every group's segments and contributions (filling the
// groups' offsets and combine block counts for H heads).
// `fwd_rows` and `dq_rows` are the forward and dQ kernels' query-strip
// heights (fwd_rows_per_wg, dq_rows_per_wg).
void pack_image(const std::vector<Task>& tasks, const SegmentCover& sc, int32_t H, bool causal,
                int32_t fwd_rows, int32_t dq_rows, int32_t kv_rows, std::vector<Group>* groups,
                std::vector<uint8_t>* image, std::vector<TableOffsets>* offs);
// Appends the segments and contributions of `groups` to the image (filling
// their offsets and block counts for H heads).
void pack_groups(const SegmentCover& sc, int32_t H, std::vector<Group>* groups,
                 std::vector<uint8_t>* image);

// Query rows per work group of the inner forward and dQ kernels, and key
// rows per work group of the dK/dV kernel.
int fwd_rows_per_wg(cqsa_dtype dt, int d);
int dq_rows_per_wg(int d);
int dkdv_rows_per_wg(int d);
// Query rows per tile of the dK/dV kernel (64 or 32).
int dkdv_qtile_rows(int d);

// Strip orders of one task for its kernels' launch order (longest first):
// query strips of `rows` rows (a multiple of 64) by the 64-key tiles live for
// them, and key strips of `rows` rows (a multiple of 64) by the 32-query
// tiles live for them (both halves of a 64-token block share its summaries, so
// counting the dK/dV kernel's 64-query tiles instead, at d = 96, halves the
// counts up to the causal boundary tile and keeps the order), with the
// kernels' liveness rule (a tile is skipped
// when the AND of the strip's block summaries and of the tile's shares a
// bit, or when it lies causally past the strip).  Ties keep strip order.
std::vector<int32_t> query_strip_order(const Task& t, bool causal, int32_t rows);
std::vector<int32_t> key_strip_order(const Task& t, bool causal, int32_t rows);

// The inner forward's tile decisions on one (batch element, head) of task t
// (App. A.2), with the kernel's rules at `rows` query rows per work group
// and 32 per wave: out[0] masked for a wave, out[1] clear, out[2] mixed,
// over the 64-key tiles each work group visits and the waves holding a
// query.  O(tiles x waves) per task.
void fwd_tile_decisions(const Task& t, bool causal, int32_t rows, int64_t out[3]);
// The dK/dV kernel's tile decisions on one (batch element, head) of task t:
// key strips of `rows` rows, groups of 32 keys, query tiles of `qtile` rows
// (64: tile q's summaries are those of block q; 32: of block q / 2); out as
// for fwd_tile_decisions.
void kv_tile_decisions(const Task& t, bool causal, int32_t rows, int32_t qtile, int64_t out[3]);

inline uint64_t align_up(uint64_t x, uint64_t a = 256) { return (x + a - 1) / a * a; }

}  // namespace cqsa
