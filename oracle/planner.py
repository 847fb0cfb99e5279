"""Online memory-aware planner, brute force -- TEST INFRASTRUCTURE.

Section III-E: as the KV cache grows, a device offloads alpha more MHA blocks and beta more MLP
blocks, the pair of least extra loading time whose freed memory -- counted in every stage of
the device but one, hence the factor (#Stage - 1) -- lets the cache fit (Eq. (7)); the first
threshold is the token count the memory left after allocation holds (Eq. (6)).

This module answers Eq. (7) for one token count at a time by trying every (alpha, beta), and
derives the steps by scanning token counts one by one.  Readings (the paper leaves them open):
memory and loading time are the integers given (bytes, any time unit); ties in loading time go
to the plan freeing more memory, then to the smaller alpha.
"""
from __future__ import annotations

from typing import List, NamedTuple, Optional, Tuple


class PlanInput(NamedTuple):
    mem_left: int            # Mem_i: bytes left for the KV cache after the layer allocation
    kv_bytes_per_token: int  # mem(token): one token's K and V over the device's layers
    mha_bytes: int           # p_A * l_size
    mlp_bytes: int           # p_M * l_size
    mha_cost: int            # loading time of one MHA block
    mlp_cost: int            # loading time of one MLP block
    mha_free: int            # |L^A| - |L~^A|: the range of alpha
    mlp_free: int            # |L^M| - |L~^M|: the range of beta
    n_stage: int             # #Stage


def plan_for(p: PlanInput, n_tokens: int) -> Optional[Tuple[int, int]]:
    """Eq. (7) for n cached tokens: the (alpha, beta) of least loading time whose freed memory
    holds them, or None when no plan does."""
    best = None
    for alpha in range(p.mha_free + 1):
        for beta in range(p.mlp_free + 1):
            freed = (alpha * p.mha_bytes + beta * p.mlp_bytes) * (p.n_stage - 1)
            if not n_tokens * p.kv_bytes_per_token < p.mem_left + freed:
                continue
            key = (alpha * p.mha_cost + beta * p.mlp_cost, -freed, alpha)
            if best is None or key < best[0]:
                best = (key, (alpha, beta))
    return None if best is None else best[1]


def first_threshold(p: PlanInput) -> float:
    """Eq. (6): TS^1 = Mem_i / mem(token), as a real number of tokens."""
    return p.mem_left / p.kv_bytes_per_token


def plan_steps(p: PlanInput, limit: int = 1 << 20) -> Tuple[List[Tuple[int, int, int]], int]:
    """[(first token count, alpha, beta)] where the plan changes, and the capacity (the least
    token count no plan holds), by scanning n = 0, 1, ... (at most `limit` counts)."""
    steps: List[Tuple[int, int, int]] = []
    for n in range(limit + 1):
        plan = plan_for(p, n)
        if plan is None:
            return steps, n
        if not steps or steps[-1][1:] != plan:
            steps.append((n, plan[0], plan[1]))
    raise ValueError("capacity beyond the scan limit")
