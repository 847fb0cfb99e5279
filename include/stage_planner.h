/*
 * stage_planner.h -- the online memory-aware planner of arXiv 2512.21835 (Section III-E,
 * Eqs. (6)-(7)) as a host function of the stage library.
 *
 * As a device's KV cache grows past what its memory holds next to the layers it keeps, the
 * planner offloads more weight blocks: alpha MHA blocks and beta MLP blocks beyond the layer
 * allocation, chosen to cost the least extra loading time while the memory they free (in every
 * stage of the device but the one being computed, hence the factor #Stage - 1) holds the cache
 * (Eq. (7)).  The first threshold is the token count the memory left after allocation holds
 * (Eq. (6)); every later threshold is where the cheapest feasible (alpha, beta) changes.  Plans
 * are not nested: a later step may reload a block an earlier one offloaded (the paper's example:
 * MHA block offloaded at TS^1, then the MLP block offloaded and the MHA block reloaded at TS^2).
 *
 * The stage applies such a plan itself (stage_config.plan_mode = 1, include/stage.h).
 *
 * Conventions as in stage.h: 0 (STAGE_OK) or a negative stage_status; nothing throws.
 * This function only computes: no GPU, no allocation, no state.
 */
#ifndef PAPER_2512_21835_STAGE_PLANNER_H
#define PAPER_2512_21835_STAGE_PLANNER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int64_t mem_left;           /* Mem_i: bytes left for the KV cache after the layer allocation
                                   (may be <= 0: then even an empty cache needs a plan) */
    int64_t kv_bytes_per_token; /* bytes one token's K and V take over the device's layers, > 0 */
    int64_t mha_bytes;          /* p_A * l_size: bytes of one MHA block, > 0 */
    int64_t mlp_bytes;          /* p_M * l_size: bytes of one MLP block, > 0 */
    int64_t mha_cost;           /* extra loading time of one offloaded MHA block (any unit, e.g. ns,
                                   or its bytes when the host link is the bound), > 0 */
    int64_t mlp_cost;           /* the same for one MLP block, > 0 */
    int32_t mha_free;           /* |L_i^A| - |L~_i^A|: MHA blocks still resident that may go, >= 0 */
    int32_t mlp_free;           /* |L_i^M| - |L~_i^M|: MLP blocks likewise, >= 0 */
    int32_t n_stage;            /* #Stage >= 1: an offloaded block frees its bytes n_stage - 1 times */
} stage_plan_input;

typedef struct {
    int64_t tokens;  /* the step holds from this many tokens on, up to the next step's `tokens` */
    int32_t alpha;   /* MHA blocks offloaded beyond the allocation */
    int32_t beta;    /* MLP blocks offloaded beyond the allocation */
} stage_plan_step;

/* Computes the planner's steps for every token count the device can hold.
   For n tokens the plan is the (alpha, beta), 0 <= alpha <= mha_free, 0 <= beta <= mlp_free, of
   least alpha*mha_cost + beta*mlp_cost with
       n * kv_bytes_per_token < mem_left + (alpha*mha_bytes + beta*mlp_bytes) * (n_stage - 1)
   (Eq. (7), memory in bytes); ties go to the plan freeing more memory, then to the smaller alpha.
   Steps are written in ascending `tokens`, the first at 0, consecutive steps with different
   plans; writes min(cap, count) steps, *n = count (at most (mha_free+1)*(mlp_free+1)).
   *capacity = the least token count no plan holds (the cache no longer fits); *n = 0 when not
   even 0 tokens fit.  Integer arithmetic throughout; EINVAL on a bad input or if a product
   overflows int64. */
int stage_plan_offload(const stage_plan_input *in, stage_plan_step *steps, int32_t cap, int32_t *n,
                       int64_t *capacity);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2512_21835_STAGE_PLANNER_H */
