// OOM guardrail (Section 3.4, "OOM guardrails").
//
// Plans are sized by a static footprint model, but a call can still fail to
// get its workspace: the device may hold less free memory than the budget,
// or a caller allocator may refuse.  Under an automatic depth the paper's
// rule applies: first lower n_cap, the number of task working sets resident
// on the device at once, without changing the decomposition; once n_cap is
// 1, increase the depth by one and re-establish n_cap.  Here n_cap is the
// number of forward sub-slots (tasks per launch group x staging slots, each
// holding one task's staged inputs and statistics) or, for the backward, the
// tasks per launch (each holding its task-local gradients) and the staging
// slots.  The reduction halves the tasks per launch group, then drops staging
// slots one at a time; a new depth restarts from the
// automatic group size and the requested slot count.  A forced depth is
// never changed: its failure is reported, as the paper does for explicit
// depths.  The configuration that succeeded is kept with the plan and tried
// first by later calls.
#include <functional>
#include <memory>
#include <string>

#include "errors.hpp"
#include "guard.hpp"
#include "plan.hpp"
#include "runtime.hpp"

namespace cqsa {

namespace {

struct Config {
  int32_t depth, group, slots, bgroup;
};

Config config_of(const cqsa_plan_t* p) {
  return Config{p->depth, p->fp.group_size, p->opts.n_slots, p->fp.bwd_group_size};
}

// The next configuration after an allocation failure, or false when none
// is left below max_depth.
bool next_config(Config& c, bool backward, const cqsa_plan_opts& o) {
  if (!backward && c.group > 1) {
    c.group /= 2;
    return true;
  }
  if (backward && c.bgroup > 1) {
    c.bgroup /= 2;
    return true;
  }
  if (c.slots > 1) {
    c.slots -= 1;
    return true;
  }
  if (c.depth < o.max_depth) {
    c.depth += 1;
    c.group = 0;  // automatic at the new depth
    c.bgroup = 0;
    c.slots = o.n_slots;
    return true;
  }
  return false;
}

std::shared_ptr<const cqsa_plan_s> build(const cqsa_plan_t* p, const Config& c, std::string* err) {
  cqsa_plan_opts o = p->opts;
  o.depth = c.depth;
  o.tasks_per_slot = c.group;
  o.bwd_tasks_per_launch = c.bgroup;
  o.n_slots = c.slots;
  cqsa_plan_t* out = nullptr;
  // the budget no longer applies: the allocation itself is the test
  const cqsa_status s = cqsa_plan(p->g.L, int32_t(p->g.H), int32_t(p->g.d), p->g.causal, 0, &o, &out);
  if (s != CQSA_OK) {
    *err = last_error_cstr();
    return nullptr;
  }
  return std::shared_ptr<const cqsa_plan_s>(out, [](const cqsa_plan_s* q) { delete q; });
}

}  // namespace

cqsa_status run_guarded(const cqsa_plan_t* p, bool backward,
                        const std::function<cqsa_status(const cqsa_plan_t*)>& run) {
  if (!p) return run(p);
  std::shared_ptr<const cqsa_plan_s> cached;  // keeps the fallback alive for this call
  {
    std::lock_guard<std::mutex> g(p->guard_mu);
    cached = backward ? p->guard_bwd : p->guard_fwd;
  }
  const cqsa_plan_t* start = cached ? cached.get() : p;
  cqsa_status s = run(start);
  if (s != CQSA_ERR_DEVICE_OOM || p->opts.depth >= 0) {
    if (s == CQSA_OK) call_record().stats.guard_steps = 0;
    return s;
  }
  std::string first = last_error_cstr();
  Config c = config_of(start);
  int64_t steps = 0;
  while (next_config(c, backward, p->opts)) {
    ++steps;
    std::string err;
    std::shared_ptr<const cqsa_plan_s> fb = build(p, c, &err);
    if (!fb) return fail(CQSA_ERR_INTERNAL, "OOM guardrail: re-planning failed: " + err);
    c = config_of(fb.get());
    clear_error();
    s = run(fb.get());
    if (s == CQSA_OK) {
      call_record().stats.guard_steps = steps;
      std::lock_guard<std::mutex> g(p->guard_mu);
      (backward ? p->guard_bwd : p->guard_fwd) = std::move(fb);
      return CQSA_OK;
    }
    if (s != CQSA_ERR_DEVICE_OOM) return s;
  }
  return fail(CQSA_ERR_DEVICE_OOM, "OOM guardrail: no configuration up to max_depth = " +
                                       std::to_string(p->opts.max_depth) +
                                       " got its workspace (first failure: " + first + ")");
}

}  // namespace cqsa
