// C-ABI entry points for planning (host only; no HIP calls).
#include <algorithm>
#include <cstring>
#include <exception>
#include <new>
#include <string>

#include "errors.hpp"
#include "plan.hpp"

using namespace cqsa;

namespace cqsa {
std::string& error_slot() {
  thread_local std::string s;
  return s;
}
}  // namespace cqsa

extern "C" {

void cqsa_plan_opts_default(cqsa_plan_opts* o) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->B = 1;
  o->dtype = CQSA_BF16;
  o->c = 7;
  o->l = 3;
  o->interest[0] = 0;
  o->interest[1] = 1;
  o->interest[2] = 3;
  o->depth = -1;
  o->min_depth = 1;
  o->max_depth = 4;
  o->n_slots = 2;
  o->inputs_on_device = 1;
  o->acc_on_device = 1;
  o->with_backward = 0;
  o->tasks_per_slot = 0;
  o->read_in_place = -1;
  o->out16 = 0;
}

cqsa_status cqsa_plan(int64_t L, int32_t H, int32_t d, int32_t causal,
                      uint64_t device_budget_bytes, const cqsa_plan_opts* opts,
                      cqsa_plan_t** out) {
  clear_error();
  if (!out) return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan: out is NULL");
  *out = nullptr;
  try {
    cqsa_plan_opts o;
    if (opts)
      o = *opts;
    else
      cqsa_plan_opts_default(&o);
    std::string err;
    cqsa_status s = validate_plan_args(L, H, d, o, &err);
    if (s != CQSA_OK) return fail(s, "cqsa_plan: " + err);
    // inputs read in place when every batch element's slice is addressable
    // by a 32-bit byte offset (the kernels' buffer loads)
    if (o.read_in_place < 0) o.read_in_place = (o.inputs_on_device && in_place_fits(L, H, d, o)) ? 1 : 0;
    Geometry g{L, H, d, causal ? 1 : 0};
    auto* p = new cqsa_plan_s();
    p->g = g;
    p->budget = device_budget_bytes;
    p->opts = o;
    auto fits = [&](const Footprint& f) {
      return device_budget_bytes == 0 || f.peak <= device_budget_bytes;
    };
    // Plans `tasks` at `dep` with the largest group size that fits the budget
    // (or the forced one); returns whether the result fits.
    auto plan_depth = [&](int32_t dep, std::vector<Task>&& tasks) {
      const int64_t ntask = int64_t(tasks.size());
      int32_t g_hi = 1;
      if (o.tasks_per_slot > 0) {
        g_hi = int32_t(std::min<int64_t>(o.tasks_per_slot, std::max<int64_t>(1, ntask)));
      } else if (o.acc_on_device && o.read_in_place == 1) {
        // nothing is staged, so a group costs only its statistics: one
        // launch over as many tasks as a merge accepts keeps every work
        // group in one grid (no tails between launches, one merge)
        g_hi = int32_t(std::min<int64_t>(kMaxContrib, std::max<int64_t>(1, ntask)));
      } else if (o.acc_on_device) {
        // enough tasks per launch for kLaunchWgs 128-query strips (two waves
        // of the GPU's resident 4-wave work groups; an 8-wave work group
        // counts as two); large tasks launch one by one
        int64_t Lmax = 1;
        for (const Task& t : tasks) Lmax = std::max(Lmax, t.L_local);
        const int64_t rows = o.dtype == CQSA_F32 ? 32 : 128;
        const int64_t wgs = std::max<int64_t>(1, (Lmax + rows - 1) / rows * o.B * H);
        g_hi = int32_t(std::min<int64_t>({(kLaunchWgs + wgs - 1) / wgs, int64_t(kMaxContrib),
                                          std::max<int64_t>(1, ntask)}));
      }
      const SegmentCover sc = segment_cover(L, tasks);
      bool ok = false;
      for (int32_t gs = std::max(1, g_hi); gs >= 1; --gs) {
        std::vector<Group> groups = make_groups(ntask, gs);
        std::vector<uint8_t> image;
        std::vector<TableOffsets> offs;
        pack_image(tasks, sc, H, causal != 0, fwd_rows_per_wg(o.dtype, d), dq_rows_per_wg(d),
                   dkdv_rows_per_wg(d), &groups, &image, &offs);
        Footprint f = footprint(g, o, dep, tasks, gs, image.size());
        ok = fits(f);
        if (ok || gs == 1 || o.tasks_per_slot > 0) {
          p->depth = dep;
          p->fp = f;
          p->groups = std::move(groups);
          p->packed = std::move(image);
          p->table_off = std::move(offs);
          break;
        }
      }
      // backward launch groups: with inputs read in place and device-resident
      // gradients, every task (up to 32) in one dQ and one dK/dV launch whose
      // task-local gradients a gather-merge sums, reduced until the budget
      // fits.  The automatic size takes only balanced splits (49 tasks: 25 +
      // 24, not 32 + 17): the same launches, and task-local buffers for the
      // larger half only.
      p->bwd_groups.clear();
      const int32_t bf = o.bwd_tasks_per_launch;
      if (bwd_batchable(o, dep) && (bf > 1 || (bf == 0 && o.with_backward)) && ntask > 1) {
        const int32_t b_hi = int32_t(std::min<int64_t>(bf > 0 ? bf : kMaxContrib, ntask));
        for (int32_t gb = b_hi; gb >= 2; --gb) {
          const int64_t n_groups = (ntask + gb - 1) / gb;
          if (bf == 0 && (ntask + n_groups - 1) / n_groups != gb) continue;
          std::vector<Group> bg = make_groups(ntask, gb);
          // the merge of the last group covers only the tokens its tasks hold
          for (Group& x : bg) x.final = false;
          std::vector<uint8_t> im = p->packed;
          pack_groups(sc, H, &bg, &im);
          Footprint f = footprint(g, o, dep, tasks, p->fp.group_size, im.size(), gb);
          if (fits(f) || bf > 0) {
            ok = ok && fits(f);
            p->fp = f;
            p->packed = std::move(im);
            p->bwd_groups = std::move(bg);
            break;
          }
        }
      }
      p->tasks = std::move(tasks);
      return ok;
    };
    // residency (App. A.3): an automatic acc_on_device keeps the accumulator
    // on the device when some depth fits the budget there, else on the host
    const bool auto_acc = o.acc_on_device < 0;
    bool found = false;
    for (int32_t acc = auto_acc ? 1 : o.acc_on_device; acc >= (auto_acc ? 0 : o.acc_on_device) && !found;
         --acc) {
      o.acc_on_device = acc;
      p->opts.acc_on_device = acc;
      if (o.depth >= 0) {
        found = plan_depth(o.depth, build_tasks(L, o, o.depth)) || !auto_acc || acc == 0;
      } else {
        for (int32_t dep = o.min_depth; dep <= o.max_depth && !found; ++dep)
          found = plan_depth(dep, build_tasks(L, o, dep));
      }
    }
    if (!found) {
      delete p;
      return fail(CQSA_ERR_BUDGET,
                  "cqsa_plan: no depth in [min_depth, max_depth] fits the device budget");
    }
    p->max_L_local = 0;
    size_t max_runs = 0;
    for (const Task& t : p->tasks) {
      p->max_L_local = std::max(p->max_L_local, t.L_local);
      max_runs = std::max(max_runs, t.runs.size());
    }
    if (max_runs > size_t(kMaxRuns)) {
      delete p;
      return fail(CQSA_ERR_UNSUPPORTED, "cqsa_plan: a task has more than 128 runs (depth too large)");
    }
    *out = p;
    return CQSA_OK;
  } catch (const std::bad_alloc&) {
    return fail(CQSA_ERR_INTERNAL, "cqsa_plan: host allocation failed");
  } catch (const std::exception& e) {
    return fail(CQSA_ERR_INTERNAL, std::string("cqsa_plan: ") + e.what());
  }
}

int32_t cqsa_plan_depth(const cqsa_plan_t* p) { return p ? p->depth : -1; }

int32_t cqsa_plan_acc_on_device(const cqsa_plan_t* p) { return p ? p->opts.acc_on_device : -1; }

int32_t cqsa_plan_reads_in_place(const cqsa_plan_t* p) { return p ? p->opts.read_in_place : -1; }

int64_t cqsa_plan_num_tasks(const cqsa_plan_t* p) { return p ? int64_t(p->tasks.size()) : -1; }

cqsa_status cqsa_plan_get_task(const cqsa_plan_t* p, int64_t t, cqsa_task* out) {
  clear_error();
  if (!p || !out) return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan_get_task: NULL argument");
  if (t < 0 || t >= int64_t(p->tasks.size()))
    return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan_get_task: task index out of range");
  const Task& k = p->tasks[size_t(t)];
  out->index = t;
  out->depth = p->depth;
  out->quorum = k.quorum.data();
  out->L_local = k.L_local;
  out->n_runs = int32_t(k.abi_runs.size());
  out->runs = k.abi_runs.data();
  out->n_blocks = int64_t(k.blk_or.size());
  out->block_or = k.blk_or.data();
  out->block_and = k.blk_and.data();
  return CQSA_OK;
}

uint64_t cqsa_plan_modelled_device_bytes(const cqsa_plan_t* p) { return p ? p->fp.peak : 0; }

int32_t cqsa_plan_tasks_per_slot(const cqsa_plan_t* p) { return p ? p->fp.group_size : -1; }

int32_t cqsa_plan_bwd_tasks_per_launch(const cqsa_plan_t* p) {
  return p ? p->fp.bwd_group_size : -1;
}

cqsa_status cqsa_plan_tile_census(const cqsa_plan_t* p, int64_t* full, int64_t* clear,
                                  int64_t* mixed) {
  clear_error();
  if (!p || !full || !clear || !mixed)
    return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan_tile_census: NULL argument");
  std::call_once(p->census_once, [p] { tile_census(p->tasks, p->census); });
  *full = p->census[0];
  *clear = p->census[1];
  *mixed = p->census[2];
  return CQSA_OK;
}

cqsa_status cqsa_plan_fwd_tile_decisions(const cqsa_plan_t* p, int64_t* masked, int64_t* clear,
                                         int64_t* mixed) {
  clear_error();
  if (!p || !masked || !clear || !mixed)
    return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan_fwd_tile_decisions: NULL argument");
  if (p->opts.dtype == CQSA_F32)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_plan_fwd_tile_decisions: fp32 plans are not counted");
  int64_t acc[3] = {0, 0, 0};
  const int32_t rows = fwd_rows_per_wg(p->opts.dtype, p->g.d);
  for (const Task& t : p->tasks) fwd_tile_decisions(t, p->g.causal != 0, rows, acc);
  const int64_t bh = int64_t(p->opts.B) * p->g.H;
  *masked = acc[0] * bh;
  *clear = acc[1] * bh;
  *mixed = acc[2] * bh;
  return CQSA_OK;
}

int32_t cqsa_bwd_kv_query_tile(int32_t d) {
  if (d < 32 || d > 256 || d % 32 != 0) return 0;
  return dkdv_qtile_rows(d);
}

cqsa_status cqsa_plan_bwd_tile_decisions(const cqsa_plan_t* p, int64_t* dq, int64_t* kv) {
  clear_error();
  if (!p || !dq || !kv)
    return fail(CQSA_ERR_INVALID_ARG, "cqsa_plan_bwd_tile_decisions: NULL argument");
  if (p->opts.dtype == CQSA_F32)
    return fail(CQSA_ERR_UNSUPPORTED, "cqsa_plan_bwd_tile_decisions: the backward needs a 16-bit dtype");
  int64_t a[3] = {0, 0, 0}, b[3] = {0, 0, 0};
  const int32_t q_rows = dq_rows_per_wg(p->g.d), k_rows = dkdv_rows_per_wg(p->g.d);
  const int32_t k_tile = dkdv_qtile_rows(p->g.d);
  for (const Task& t : p->tasks) {
    fwd_tile_decisions(t, p->g.causal != 0, q_rows, a);
    kv_tile_decisions(t, p->g.causal != 0, k_rows, k_tile, b);
  }
  const int64_t bh = int64_t(p->opts.B) * p->g.H;
  for (int i = 0; i < 3; ++i) {
    dq[i] = a[i] * bh;
    kv[i] = b[i] * bh;
  }
  return CQSA_OK;
}

void cqsa_plan_destroy(cqsa_plan_t* p) { delete p; }

const char* cqsa_last_error(void) { return last_error_cstr(); }

}  // extern "C"
