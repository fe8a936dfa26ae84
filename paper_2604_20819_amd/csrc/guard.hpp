// OOM guardrail around the forward and backward calls (Section 3.4).
#pragma once

#include <functional>

#include "cqsa.h"

namespace cqsa {

// Runs `run` on the plan (or on the fallback that last succeeded); after an
// allocation failure under an automatic depth, retries with fewer resident
// task working sets and then deeper plans, up to the plan's max_depth.
cqsa_status run_guarded(const cqsa_plan_t* plan, bool backward,
                        const std::function<cqsa_status(const cqsa_plan_t*)>& run);

}  // namespace cqsa
