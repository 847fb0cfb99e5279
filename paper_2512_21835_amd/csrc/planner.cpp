// Online memory-aware planner (Section III-E, Eqs. (6)-(7)): the step function from the number
// of cached tokens to the (alpha, beta) block offloading plan.  Implements include/stage_planner.h.
//
// Rather than solving Eq. (7) for every token count, the plans are sorted by the memory they
// free.  For n tokens the deficit is d(n) = n * kv_bytes_per_token - mem_left and the feasible
// plans are those freeing more than d(n); between two consecutive distinct freed amounts
// v_k <= d(n) < v_{k+1} the feasible set is fixed (every plan freeing at least v_{k+1}), so its
// cheapest member, a suffix minimum over the sorted plans, is the step's plan, and the step
// starts at the least n with n * kv_bytes_per_token >= mem_left + v_k.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "stage.h"
#include "stage_planner.h"

namespace {

constexpr int32_t kMaxFree = 1024;  // bounds the (alpha, beta) enumeration

struct Plan {
    int64_t freed, cost;
    int32_t alpha, beta;
};

// Least cost, then most memory freed, then fewest MHA blocks.
bool better(const Plan &x, const Plan &y) {
    if (x.cost != y.cost) return x.cost < y.cost;
    if (x.freed != y.freed) return x.freed > y.freed;
    return x.alpha < y.alpha;
}

// Least n >= 0 with n * per >= bound (per > 0).
int64_t least_tokens(int64_t bound, int64_t per) {
    if (bound <= 0) return 0;
    return bound / per + (bound % per != 0);
}

}  // namespace

extern "C" int stage_plan_offload(const stage_plan_input *in, stage_plan_step *steps, int32_t cap, int32_t *n,
                                  int64_t *capacity) {
    if (!in || !n || !capacity || cap < 0 || (cap > 0 && !steps)) return STAGE_EINVAL;
    const stage_plan_input &p = *in;
    if (p.kv_bytes_per_token <= 0 || p.mha_bytes <= 0 || p.mlp_bytes <= 0 || p.mha_cost <= 0 || p.mlp_cost <= 0 ||
        p.mha_free < 0 || p.mlp_free < 0 || p.mha_free > kMaxFree || p.mlp_free > kMaxFree || p.n_stage < 1)
        return STAGE_EINVAL;

    std::vector<Plan> plans;
    plans.reserve((size_t)(p.mha_free + 1) * (p.mlp_free + 1));
    const int64_t copies = p.n_stage - 1;
    for (int32_t a = 0; a <= p.mha_free; ++a)
        for (int32_t b = 0; b <= p.mlp_free; ++b) {
            int64_t ma, mb, bytes, freed, ca, cb, cost;
            if (__builtin_mul_overflow((int64_t)a, p.mha_bytes, &ma) ||
                __builtin_mul_overflow((int64_t)b, p.mlp_bytes, &mb) || __builtin_add_overflow(ma, mb, &bytes) ||
                __builtin_mul_overflow(bytes, copies, &freed) ||
                __builtin_mul_overflow((int64_t)a, p.mha_cost, &ca) ||
                __builtin_mul_overflow((int64_t)b, p.mlp_cost, &cb) || __builtin_add_overflow(ca, cb, &cost))
                return STAGE_EINVAL;
            plans.push_back({freed, cost, a, b});
        }
    std::sort(plans.begin(), plans.end(), [](const Plan &x, const Plan &y) { return x.freed < y.freed; });

    // best[i]: the cheapest plan among plans[i..]
    std::vector<Plan> best(plans.size());
    best.back() = plans.back();
    for (size_t i = plans.size() - 1; i-- > 0;) best[i] = better(plans[i], best[i + 1]) ? plans[i] : best[i + 1];

    // distinct freed amounts v_0 < v_1 < ... and where each group starts
    std::vector<size_t> group;
    for (size_t i = 0; i < plans.size(); ++i)
        if (i == 0 || plans[i].freed != plans[i - 1].freed) group.push_back(i);

    auto start_of = [&](int64_t v, int64_t *t) {  // least n with n * kv >= mem_left + v
        int64_t bound;
        if (__builtin_add_overflow(p.mem_left, v, &bound)) return false;
        *t = least_tokens(bound, p.kv_bytes_per_token);
        return true;
    };

    std::vector<stage_plan_step> out;
    auto emit = [&](int64_t from, int64_t to, const Plan &pl) {
        if (from >= to) return;
        if (!out.empty() && out.back().alpha == pl.alpha && out.back().beta == pl.beta) return;
        out.push_back({from, pl.alpha, pl.beta});
    };
    int64_t from = 0, to = 0;
    if (!start_of(plans[group[0]].freed, &to)) return STAGE_EINVAL;
    emit(from, to, best[0]);  // deficit below the smallest freed amount: every plan is feasible
    for (size_t k = 0; k + 1 < group.size(); ++k) {
        from = to;
        if (!start_of(plans[group[k + 1]].freed, &to)) return STAGE_EINVAL;
        emit(from, to, best[group[k + 1]]);
    }
    *capacity = to;
    *n = (int32_t)out.size();
    for (int32_t i = 0; i < std::min<int32_t>(cap, *n); ++i) steps[i] = out[i];
    return STAGE_OK;
}
