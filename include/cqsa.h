/*
 * cqsa.h -- C ABI of the Stream-CQSA hot path for AMD MI355X (gfx950).
 *
 * Stream-CQSA (arxiv 2604.20819) splits an exact attention call into c**itr
 * independent subsequence tasks by cyclic-quorum-set (CQS) decomposition
 * (Section 3, Eq. 1; Section 3.3), runs a masked flash-style inner kernel on
 * every task, and recomposes the per-task softmax statistics exactly in
 * full-token coordinates (App. A.1, Eq. "merge"); the backward recomputes the
 * probabilities from the global log-sum-exp (App. A.1, Eq. "globallse").
 * The depth is the smallest one whose modelled device footprint fits the
 * budget (Section 3.4).
 *
 * Conventions shared by every call
 *   - Every call returns cqsa_status: 0 on success, a negative code on error.
 *     No C++ exception or abort crosses this boundary.  On error the contents
 *     of outputs are unspecified and cqsa_last_error() describes the failure.
 *   - Tensors are dense row-major [B, L, H, d] (d fastest), with no stride
 *     arguments: a task's run of tokens is then one contiguous span per batch
 *     element, which staging copies in one transfer and the kernels address
 *     with one row offset.  The caller owns them.  LSE and the softmax
 *     statistics are [B, H, L] fp32.
 *   - Outputs O (unless the plan asks for a 16-bit O), dQ, dK, dV are fp32
 *     and LSE is the natural-log log-sum-exp of the scaled scores (Section 4.1: statistics, merge and output are
 *     fp32; App. A.1: lse = m + log l).
 *   - Inputs are fp32, fp16 or bf16.  Head dimension d: 32, 64, 96, ..., 256
 *     for the forward (the head dims the paper's forward covers, Sec. 5,
 *     kernel coverage) and for the backward (the paper's backward stops at
 *     64 and 128 and names the wider range as needed for production).
 *   - Calls on device-resident outputs are ordered on `hip_stream` (a
 *     hipStream_t; NULL = the null stream) and return without waiting;
 *     a call with any host-resident output blocks until it is complete.
 *   - The library is thread-safe for distinct plans and streams; a plan's
 *     decomposition is immutable after creation and the plan may be shared
 *     across threads (the only state a call may change is the OOM
 *     guardrail's cached fallback, which is guarded and reference-counted).
 */
#ifndef CQSA_H
#define CQSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CQSA_OK = 0,
  CQSA_ERR_INVALID_ARG = -1, /* bad pointer, shape, dtype or option; no device work done */
  CQSA_ERR_UNSUPPORTED = -2, /* valid but not built (e.g. d not a multiple of 32 in [32, 256],
                                fp32 inputs to the backward) */
  CQSA_ERR_BUDGET = -3,      /* no depth <= max_depth fits the device budget */
  CQSA_ERR_DEVICE_OOM = -4,  /* a device allocation failed */
  CQSA_ERR_HIP = -5,         /* a HIP runtime call failed (no device, launch error, ...) */
  CQSA_ERR_INTERNAL = -6
} cqsa_status;

typedef enum { CQSA_F32 = 0, CQSA_F16 = 1, CQSA_BF16 = 2 } cqsa_dtype;
typedef enum { CQSA_MEM_HOST = 0, CQSA_MEM_DEVICE = 1 } cqsa_mem;

/* A caller-owned tensor: `data` points at element [0,0,0,0] of a dense
 * row-major [B, L, H, d] array of `dtype`, in host memory (pinned memory is
 * recommended, pageable works) or device memory as `where` says.  `data`
 * must be 16-byte aligned (the kernels move rows in 16-byte vectors); a
 * misaligned tensor is rejected with CQSA_ERR_INVALID_ARG. */
typedef struct {
  void* data;
  cqsa_dtype dtype;
  cqsa_mem where;
  int64_t B, L, H, d;
} cqsa_tensor;

#define CQSA_MAX_INTEREST 16
#define CQSA_MAX_LEVEL_SETS 4

/* One level's interest set: a perfect (c, l, 1) cyclic difference set with
 * c = l(l-1)+1 and interest[0] = 0 (App. C, Table "interest_set"). */
typedef struct {
  int32_t c;
  int32_t l;
  int32_t interest[CQSA_MAX_INTEREST];
} cqsa_interest_set;

/* Planning options.  cqsa_plan_opts_default() fills the defaults noted here. */
typedef struct {
  int32_t B;                 /* batch size (1) */
  cqsa_dtype dtype;          /* input dtype (CQSA_BF16) */
  int32_t c;                 /* chunk count, c = l(l-1)+1 (7) */
  int32_t l;                 /* interest-set size (3) */
  int32_t interest[CQSA_MAX_INTEREST]; /* perfect (c,l,1) difference set ({0,1,3}); App. C */
  int32_t depth;             /* -1: automatic (smallest fitting depth >= min_depth); >= 0: forced (-1) */
  int32_t min_depth;         /* first depth the automatic search tries (1, the paper's auto*) */
  int32_t max_depth;         /* last depth the automatic search tries (4) */
  int32_t n_slots;           /* staging slots in flight, >= 1 (2) */
  int32_t inputs_on_device;  /* 1: Q, K, V (and dO) are device-resident; 0: host-resident (1) */
  int32_t acc_on_device;     /* 1: accumulator/outputs on device; 0: on host, merged by host
                                threads; -1: on the device when some depth in [min_depth,
                                max_depth] fits the budget there, else on the host (query
                                cqsa_plan_acc_on_device).  For the backward, O, LSE, dQ, dK
                                and dV follow this residency (1) */
  int32_t with_backward;     /* 1: the footprint must also fit cqsa_backward (0) */
  int32_t tasks_per_slot;    /* forward tasks staged, launched and merged together, in [0, 32]:
                                0 = automatic: with inputs read in place, every task up to 32
                                per launch; with staged inputs, enough tasks for 1024
                                inner-kernel work groups per launch (capped at 32 and at the
                                task count); either reduced until the budget fits, and 1 when
                                acc_on_device = 0; >= 1 forced; > 1 needs acc_on_device = 1 (0) */
  int32_t n_level_sets;      /* 0: every level uses (c, l, interest).  n in [1, 4]: level t
                                (1-based) uses level_sets[min(t, n) - 1], so the last set repeats
                                below level n, and (c, l, interest) are ignored.  Section 3.3
                                allows a different valid set at each depth, for finer control of
                                the task length (0) */
  cqsa_interest_set level_sets[CQSA_MAX_LEVEL_SETS];
  int32_t read_in_place;     /* how the inner kernels reach a task's tokens (App. A.3 gathers
                                them into contiguous buffers):
                                1: read in place -- the kernels address the runs inside the
                                caller's device tensors, so no per-task copy is made and no
                                task inputs are held in the workspace; needs
                                inputs_on_device = 1 and B-slices under 2 GiB
                                (L * H * d * elem < 2^31 bytes);
                                0: gather every task's runs into staging slots first;
                                -1: automatic -- 1 when its conditions hold, else 0 (query
                                cqsa_plan_reads_in_place) (-1) */
  int32_t out16;             /* 1: cqsa_forward writes O in the input dtype (bf16 or fp16), each
                                element the fp32 result rounded to nearest even; the fp32
                                result is kept in the workspace, and the footprint counts it.
                                Needs a 16-bit dtype, acc_on_device = 1 and with_backward = 0
                                (the backward reads the fp32 O).  0: O is fp32 (0) */
  int32_t bwd_tasks_per_launch; /* backward tasks run by one dQ and one dK/dV launch, in
                                [0, 32].  Applies when the inputs are read in place and O, LSE,
                                dQ, dK, dV are device-resident (acc_on_device = 1) at depth
                                >= 1: the tasks of a launch store their gradients in task-local
                                fp32 buffers in the workspace (3 x B x L_max x H x d x 4 bytes
                                per task) and one gather-merge per launch adds them into dQ, dK,
                                dV in task order.  0 = automatic: every task up to 32 when
                                with_backward = 1, reduced until the budget fits, over
                                balanced splits only (49 tasks: 25 per launch), else 1;
                                >= 1 forced (> 1 needs inputs_on_device = 1 and neither
                                read_in_place nor acc_on_device set to 0; where the
                                conditions above do not hold, 1 applies).  With 1, each
                                task's launches add its rows into the gradients directly, tasks
                                one after another.  Every setting gives the same bits (0) */
} cqsa_plan_opts;

/* One contiguous run of a task's tokens: global tokens
 * [global_start, global_start + length) all carrying group `bits`. */
typedef struct {
  int64_t global_start;
  int64_t length;
  uint32_t bits;
} cqsa_run;

/* Read-only view of one task (Alg. 3 entry).  Pointers stay valid until the
 * plan is destroyed.  Local token order equals global order (App. A.3).
 * Group bit numbering: at level t (1-based) with set (c_t, l_t, I_t), the chunk
 * (q_t + I_t[j]) mod c_t, j = 1..l_t-1, carries bit s_t + (j-1), where s_t is
 * the sum of (l_u - 1) over the levels u < t ((t-1)*(l-1) when every level
 * uses the same set); the owner chunk q_t carries none.
 * A local pair (q, k) is kept iff (bits[q] & bits[k]) == 0 (App. A.2), and, when
 * causal, global(k) <= global(q). */
typedef struct {
  int64_t index;             /* position in the plan's task list (lexicographic quorum order) */
  int32_t depth;
  const int32_t* quorum;     /* `depth` entries q_1..q_depth */
  int64_t L_local;           /* tokens in the task */
  int32_t n_runs;
  const cqsa_run* runs;      /* ascending global order */
  int64_t n_blocks;          /* ceil(L_local / 64) */
  const uint32_t* block_or;  /* per 64-token local block: OR of the bits (App. A.2) */
  const uint32_t* block_and; /* per 64-token local block: AND of the bits */
} cqsa_task;

typedef struct cqsa_plan_s cqsa_plan_t;

/* Per-call statistics (cqsa_last_stats).  Stage times are filled only when
 * timing is enabled (cqsa_set_timing); they come from HIP events recorded on
 * the stream each stage runs on. */
typedef struct {
  int32_t depth;
  int64_t num_tasks;
  uint64_t modelled_device_bytes;   /* the plan's footprint model */
  uint64_t workspace_bytes;         /* device bytes the library held for the call */
  uint64_t h2d_bytes, d2h_bytes, d2d_bytes; /* bytes staged across the host link / on device */
  int64_t inner_launches;           /* inner-kernel launches (forward or backward) */
  double ms_wall;                   /* first enqueue to completion, device clock */
  double ms_stage;                  /* sum of staging copy spans */
  double ms_inner;                  /* sum of inner forward (or backward) kernel spans */
  double ms_merge;                  /* forward: sum of merge-launch spans (device; the last one
                                       also finalises) or host-merge time; backward: zero-fill of
                                       dQ, dK, dV (the scatter-adds are fused into the kernels) */
  double ms_finalize;               /* forward: host finalisation time (acc on host);
                                       backward: preprocess span (D = rowsum(dO * O)) */
  double ms_d2h;                    /* sum of statistics device-to-host spans */
  int64_t tiles_full, tiles_clear, tiles_mixed; /* 128x128 tile census of the plan */
  int64_t merge_launches;           /* device merge launches (forward merges, or the backward's
                                       gradient merges) */
  double ms_inner_busy;             /* time at least one inner kernel ran (union of its spans) */
  int64_t guard_steps;              /* OOM guardrail fallbacks this call took (0: the plan ran) */
  int64_t resident_tasks;           /* task working sets held at once (forward sub-slots,
                                       backward staging slots, or the backward tasks per launch
                                       whose local gradients the workspace holds; 0 for the
                                       undecomposed path and for one in-place task per launch) */
  /* The kernels' own tile decisions (App. A.2), counted on the device when
   * tile counting is enabled (cqsa_set_tile_counting), else -1.  Forward
   * (16-bit inputs) and the backward's dQ kernel: one wave of 32 consecutive
   * local queries (every wave holding a query of its task) against one 64-key
   * tile its work group visits, summed over tasks, batch elements and heads:
   * masked (every pair masked for the wave: skipped), clear (no pair masked:
   * no mask work), mixed (per-pair tests).  cqsa_plan_fwd_tile_decisions
   * and cqsa_plan_bwd_tile_decisions give the counts the block summaries
   * predict. */
  int64_t kernel_tiles_masked, kernel_tiles_clear, kernel_tiles_mixed;
  /* Backward only: the dK/dV kernel's decisions, one group of 32 consecutive
   * local keys against one query tile its work group visits (64 queries at
   * d = 96, else 32). */
  int64_t kernel_kv_tiles_masked, kernel_kv_tiles_clear, kernel_kv_tiles_mixed;
} cqsa_run_stats;

/* Fill `o` with the defaults listed in cqsa_plan_opts. */
void cqsa_plan_opts_default(cqsa_plan_opts* o);

/* Plan a call on L tokens, H heads, head dim d (Section 3.4; Alg. 3).
 * device_budget_bytes = 0 means uncapped.  opts = NULL uses the defaults.
 * Validates every level's (c, l, interest) as a perfect difference set
 * (App. C); at most 32 group bits and 2^20 tasks in total.  With an
 * automatic depth, returns the smallest depth in [min_depth, max_depth] whose
 * modelled device footprint fits the budget, else CQSA_ERR_BUDGET; a forced
 * depth is planned even if it does not fit (the footprint is still reported).
 * Host only: no device work.  *out receives a plan the caller must destroy. */
cqsa_status cqsa_plan(int64_t L, int32_t H, int32_t d, int32_t causal,
                      uint64_t device_budget_bytes, const cqsa_plan_opts* opts,
                      cqsa_plan_t** out);
int32_t cqsa_plan_depth(const cqsa_plan_t* plan);          /* -1 if plan is NULL */
int64_t cqsa_plan_num_tasks(const cqsa_plan_t* plan);      /* -1 if plan is NULL */
/* Fill *out with task t's view; CQSA_ERR_INVALID_ARG if t is out of range. */
cqsa_status cqsa_plan_get_task(const cqsa_plan_t* plan, int64_t t, cqsa_task* out);
/* Modelled peak device bytes of a call under this plan: caller tensors that are
 * device-resident plus everything the library allocates. 0 if plan is NULL. */
uint64_t cqsa_plan_modelled_device_bytes(const cqsa_plan_t* plan);
/* Forward tasks per staging slot and launch group the plan chose; -1 if plan is NULL. */
int32_t cqsa_plan_tasks_per_slot(const cqsa_plan_t* plan);
/* Backward tasks per dQ and dK/dV launch the plan chose (bwd_tasks_per_launch);
 * -1 if plan is NULL. */
int32_t cqsa_plan_bwd_tasks_per_launch(const cqsa_plan_t* plan);
/* Where the plan keeps the accumulator and outputs: 1 device, 0 host (the choice of an
 * automatic acc_on_device = -1; App. A.3, residency); -1 if plan is NULL. */
int32_t cqsa_plan_acc_on_device(const cqsa_plan_t* plan);
/* Whether the plan's kernels read the caller's tensors in place: 1 yes, 0 they gather
 * each task's runs into staging slots (the choice of read_in_place = -1); -1 if plan is
 * NULL. */
int32_t cqsa_plan_reads_in_place(const cqsa_plan_t* plan);
/* Pooled 128x128 tile census over causal-retained tiles of every task (App. A.2). */
cqsa_status cqsa_plan_tile_census(const cqsa_plan_t* plan, int64_t* full, int64_t* clear,
                                  int64_t* mixed);
/* The inner forward's tile decisions this plan predicts, in the unit of
 * cqsa_run_stats.kernel_tiles_* (App. A.2 verdicts from the 64-token block
 * summaries, at the 16-bit kernel's work-group and wave shapes for the plan's
 * d): a work group of R query rows (R = 256 at d = 96 ... 192, else 128)
 * visits key tile t unless t is causally past its last query or the AND of
 * its blocks' summaries meets tile t's; a visited tile is masked for a wave
 * when the wave's block AND meets the tile's or it is causally past the
 * wave's last query, clear when the wave's block OR misses the tile's, the
 * tile lies causally below the wave's first query and holds 64 keys, mixed
 * otherwise.  Summed over tasks times B x H.  CQSA_ERR_UNSUPPORTED for fp32
 * plans (their kernel is not counted). */
cqsa_status cqsa_plan_fwd_tile_decisions(const cqsa_plan_t* plan, int64_t* masked,
                                         int64_t* clear, int64_t* mixed);
/* The backward kernels' tile decisions this plan predicts (16-bit plans).
 * dq[0..2]: the dQ kernel's masked, clear, mixed counts, by the rules of
 * cqsa_plan_fwd_tile_decisions at its work-group height (256 query rows at
 * d = 96 ... 160, else 128).  kv[0..2]: the dK/dV kernel's, for key strips of
 * R rows (256 at d = 96, 128, else 128), groups of 32 keys and query tiles
 * of T rows (64 at d = 96, one summary block; else 32, half a block):
 * a work group visits query tile t unless t lies causally wholly
 * before its first key or the AND of its blocks' summaries meets the
 * summaries of t's block; a visited tile is masked for a key group when the
 * group's block AND meets the tile's or it lies causally wholly before the
 * group's first key, clear when the group's block OR misses the tile's and,
 * causally, the tile starts at or after the group's last key, mixed
 * otherwise.  Summed over tasks times B x H. */
cqsa_status cqsa_plan_bwd_tile_decisions(const cqsa_plan_t* plan, int64_t* dq, int64_t* kv);
/* Host only: the query rows T of one dK/dV tile at head dim d (64 at d = 96,
 * else 32; the unit of the kv counts above), or 0 for a d the kernels do not
 * take (not a multiple of 32 in [32, 256]). */
int32_t cqsa_bwd_kv_query_tile(int32_t d);
void cqsa_plan_destroy(cqsa_plan_t* plan);                 /* NULL is a no-op */

/* Decomposed forward (Alg. 1 computed with the max-shifted merge of App. A.1).
 * Q, K, V: inputs matching the plan (B, L, H, d, dtype, and residency
 * inputs_on_device).  O: fp32 [B, L, H, d] (the plan's 16-bit dtype when the plan
 * has out16 = 1), where = acc_on_device ? device : host.
 * LSE: fp32 [B, H, L] in `lse_where` memory (must equal O's residency).
 * scale <= 0 selects 1/sqrt(d) (Section 3.1).  Device-resident outputs are
 * written in stream order on hip_stream; host-resident outputs are complete
 * on return.
 * OOM guardrail (Section 3.4): with an automatic depth, a workspace allocation
 * failure (CQSA_ERR_DEVICE_OOM) is retried with fewer task working sets
 * resident at once (halved tasks per launch group, then fewer staging
 * slots), then one level deeper, up to max_depth; the configuration that
 * succeeded is kept with the plan for later calls, and
 * cqsa_run_stats.guard_steps counts the fallbacks.  A forced depth reports
 * the failure.  Nothing is enqueued by an attempt that fails to allocate. */
cqsa_status cqsa_forward(const cqsa_plan_t* plan, const cqsa_tensor* Q, const cqsa_tensor* K,
                         const cqsa_tensor* V, cqsa_tensor* O, float* LSE, cqsa_mem lse_where,
                         float scale, void* hip_stream);

/* Decomposed backward in the global-LSE form (App. A.1, Eq. "globallse"),
 * equal to Alg. 2.  Q, K, V, dO: inputs matching the plan, resident where the
 * plan's inputs are (inputs_on_device); O, LSE: the forward's outputs, and
 * dQ, dK, dV: fp32 [B, L, H, d], overwritten, all resident where the plan's
 * accumulator is (acc_on_device; Sec. 4.1 keeps Q, K, V in host memory, and
 * Table "recovery" runs forward+backward with the accumulator on the host).
 * Host-resident inputs are staged task by task through the device slots (a
 * token the previously staged task also holds is copied on the device);
 * D = rowsum(dO * O) is computed from chunks of host-resident O or dO;
 * host-resident gradients are computed per task on the device, copied back
 * and added into dQ, dK, dV on host threads, and the call then blocks until
 * they are complete.  Needs a 16-bit dtype and a plan made with
 * with_backward = 1 or an uncapped budget; the OOM guardrail of cqsa_forward
 * applies (fewer staging slots, then deeper plans). */
cqsa_status cqsa_backward(const cqsa_plan_t* plan, const cqsa_tensor* Q, const cqsa_tensor* K,
                          const cqsa_tensor* V, const cqsa_tensor* O, const float* LSE,
                          cqsa_mem lse_where, const cqsa_tensor* dO, cqsa_tensor* dQ,
                          cqsa_tensor* dK, cqsa_tensor* dV, float scale, void* hip_stream);

/* Bytes of the fixed device scratch array that cqsa_forward_noalloc works in
 * (64 MiB; one array per GPU the library runs on, held until the process
 * ends). */
#define CQSA_NOALLOC_SCRATCH_BYTES (64u << 20)

/* cqsa_forward for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, results and ordering as cqsa_forward (bit-identical outputs), but
 * the call allocates nothing: no hipMalloc, no hipFree, no pinned host memory,
 * no caller-allocator call, no new streams or events (those it records into
 * exist from the device's set-up).  Its workspace is a fixed device
 * array of CQSA_NOALLOC_SCRATCH_BYTES per GPU, looked up once per device when
 * the library first runs there.  The plan image is copied from the plan
 * itself (pageable host memory), so the copy may block the host until the
 * stream reaches it.
 * Limits, each reported as CQSA_ERR_INVALID_ARG before any device work:
 *   - the plan must keep O and LSE on the device (acc_on_device = 1);
 *   - the call's workspace (the plan image plus the task statistics and, for
 *     staged plans, the staged inputs) must fit CQSA_NOALLOC_SCRATCH_BYTES;
 *   - at most 3 staging slots;
 *   - per-stage timing (cqsa_set_timing) is not recorded.
 * No OOM guardrail runs (nothing is allocated).  Nothing in the scratch has
 * to start at zero: each call writes every byte it reads before reading it.
 * Every call on a GPU shares that GPU's scratch and finds the previous
 * call's contents there.  Two calls whose device work overlapped on one GPU
 * would race in it, so each call's device work waits for the previous
 * no-allocation call's (an event the library records at the end of every
 * call): calls from different streams or host threads queue, they do not
 * overlap. */
cqsa_status cqsa_forward_noalloc(const cqsa_plan_t* plan, const cqsa_tensor* Q,
                                 const cqsa_tensor* K, const cqsa_tensor* V, cqsa_tensor* O,
                                 float* LSE, cqsa_mem lse_where, float scale, void* hip_stream);

/* Route the library's device workspace through a caller allocator (e.g. a
 * framework's caching allocator).  alloc(bytes, ctx) returns device memory or
 * NULL (reported as CQSA_ERR_DEVICE_OOM); release(ptr, ctx) frees it.  Passing
 * NULL functions restores the built-in cached hipMalloc workspace. */
cqsa_status cqsa_set_allocator(void* (*alloc)(size_t bytes, void* ctx),
                               void (*release)(void* ptr, void* ctx), void* ctx);

/* Enable (1) or disable (0) per-stage HIP-event timing for later calls on
 * this thread. */
cqsa_status cqsa_set_timing(int32_t enable);

/* Enable (1) or disable (0) counting the kernels' tile decisions
 * (cqsa_run_stats.kernel_tiles_*, kernel_kv_tiles_*) for later cqsa_forward
 * and cqsa_backward calls on this thread (a diagnostic: the launches run
 * counting instances of the kernels, which add one atomic per wave; the
 * counters live in a small device buffer per GPU and a pinned host copy per
 * thread, both allocated on first use, so counted calls that overlap on one
 * GPU mix their counts; cqsa_forward_noalloc does not count). */
cqsa_status cqsa_set_tile_counting(int32_t enable);

/* Statistics of the last cqsa_forward/cqsa_backward on this thread; waits for
 * that call's timing events to complete. */
cqsa_status cqsa_last_stats(cqsa_run_stats* out);

/* Free the built-in workspace cache of the current device. */
cqsa_status cqsa_release_workspace(void);

/* Thread-local description of the last error; valid until the next call on
 * this thread.  Never NULL. */
const char* cqsa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CQSA_H */
