// Internal plan representation shared by the planner, the runtime and the
// C-ABI layer.  Not part of the public ABI (see include/cqsa.h).
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "cqsa.h"

namespace cqsa {

constexpr int kBlock = 64;   // tokens per block summary (App. A.2)
constexpr int kTile = 128;   // census tile edge (App. A.2)

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
  uint64_t blk_or = 0;  // uint32[n_blocks]
  uint64_t blk_and = 0; // uint32[n_blocks]
};

// Everything the runtime allocates for one call, in bytes.
struct Footprint {
  uint64_t resident_fwd = 0;   // caller tensors on device during the forward
  uint64_t resident_bwd = 0;   // caller tensors on device during the backward
  uint64_t slot_fwd = 0;       // one forward staging slot (inputs + task statistics)
  uint64_t slot_bwd = 0;       // one backward staging slot (inputs)
  uint64_t global_fwd = 0;     // forward device workspace independent of slots
  uint64_t global_bwd = 0;     // backward device workspace independent of slots
  uint64_t tables = 0;         // packed per-task tables
  uint64_t peak = 0;           // modelled peak device bytes
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
  // packed per-task tables, uploaded to the device by every call
  std::vector<uint8_t> packed;
  std::vector<cqsa::TableOffsets> table_off;
  // lazily computed census
  mutable std::once_flag census_once;
  mutable int64_t census[3] = {0, 0, 0};
};

namespace cqsa {

size_t dtype_size(cqsa_dtype t);

// Validates options and geometry; returns CQSA_OK or sets the error text.
cqsa_status validate_plan_args(int64_t L, int32_t H, int32_t d, const cqsa_plan_opts& o,
                               std::string* err);

// Builds the c**depth tasks of BuildSubseq with ascending chunk order.
std::vector<Task> build_tasks(int64_t L, const cqsa_plan_opts& o, int32_t depth);

// Footprint of running `tasks` under `o` (mirrors the runtime's allocations).
Footprint footprint(const Geometry& g, const cqsa_plan_opts& o, int32_t depth,
                    const std::vector<Task>& tasks);

void tile_census(const std::vector<Task>& tasks, int64_t out[3]);

bool is_perfect_difference_set(const int32_t* I, int32_t l, int32_t c);

// Runtime workspace layout helpers (bytes), shared with the footprint model.
uint64_t fwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged,
                        bool stats);
uint64_t bwd_slot_bytes(const Geometry& g, const cqsa_plan_opts& o, int64_t Lmax, bool staged);
uint64_t table_bytes(const std::vector<Task>& tasks);
// Packs every task's runs and block summaries into one image (layout of
// table_bytes; the DevRun record is 32 bytes).
void pack_tables(const std::vector<Task>& tasks, std::vector<uint8_t>* image,
                 std::vector<TableOffsets>* offs);

inline uint64_t align_up(uint64_t x, uint64_t a = 256) { return (x + a - 1) / a * a; }

}  // namespace cqsa
