// Records of the packed plan image that the kernels read (internal).
//
// The planner writes them on the host and every call uploads the image once;
// the layouts are plain C++ so host and device code share one definition.
#pragma once

#include <stdint.h>

namespace cqsa {

constexpr int kMaxRuns = 128;      // runs per task the kernels accept (l**depth bound)
constexpr int kMaxContrib = 32;    // tasks of one launch group that may share a token
constexpr int kCombinePairs = 64;  // (token, head) pairs per combine work group

// One maximal run of a task: local tokens [local_start, local_start + length)
// are global tokens [global_start, global_start + length), all with `bits`.
struct DevRun {
  int64_t local_start;
  int64_t global_start;
  int64_t length;
  uint32_t bits;
  uint32_t pad;
};

// One task: its length and where its tables sit in the image (byte offsets).
struct DevTask {
  int64_t L_local;
  int64_t runs_off;   // DevRun[n_runs]
  int64_t qorder_off; // int32[ceil(L_local / R)] forward query strips of R rows, R the
                      // forward's strip height (fwd_rows_per_wg), most live key tiles first
  int64_t dqorder_off;// int32[ceil(L_local / R)] dQ query strips of R rows, R the dQ
                      // kernel's strip height (dq_rows_per_wg), most live key tiles first
  int64_t korder_off; // int32[ceil(L_local / R)] dK/dV key strips of R rows, R the dK/dV
                      // kernel's strip height (dkdv_rows_per_wg), most live query tiles first
  int64_t sum_off;    // DevBlock[ceil(L_local / 64)]: each 64-token block's summaries and row
  int32_t n_runs;
  int32_t pad;
};

// One 64-token block: the OR and the AND of its tokens' group bits, and its
// row in the block row table (see kNoRow); a tile window reads one per lane.
struct DevBlock {
  uint32_t bor;
  uint32_t band;
  int32_t row;
  uint32_t pad;
};

// Strips of a (task, b, h) run in the order of the task's strip tables
// (forward, dQ, dK/dV), longest first, so a launch ends with its shortest
// strips.

// Block row table: entry i is the global row of local token 64 i when the
// tokens of block i (up to the task end) lie in one run, so they are
// consecutive rows of the caller's tensors; kNoRow when the block crosses a
// run boundary.
constexpr int32_t kNoRow = -1;

// Elementary global segment of a launch group's merge: tokens
// [g0, g0 + len) lie inside one run of every task that holds them.  The
// segment's contributions are DevContrib[c_off .. c_off + n_c); has_global
// says whether tasks of earlier groups already merged into these tokens.
// Combine work groups blk0 .. blk0 + ceil(len * H / kCombinePairs) - 1 own it.
struct DevSeg {
  int64_t g0;
  int64_t len;
  int64_t blk0;
  int32_t c_off;
  int32_t n_c;
  int32_t has_global;
  int32_t pad;
};

// Token g0 of a segment is local token `local_start` of the group's task j.
struct DevContrib {
  int64_t local_start;
  int32_t j;
  int32_t pad;
};

static_assert(sizeof(DevRun) == 32, "DevRun layout");
static_assert(sizeof(DevTask) == 56, "DevTask layout");
static_assert(sizeof(DevBlock) == 16, "DevBlock layout");
static_assert(sizeof(DevSeg) == 40, "DevSeg layout");
static_assert(sizeof(DevContrib) == 16, "DevContrib layout");

}  // namespace cqsa
