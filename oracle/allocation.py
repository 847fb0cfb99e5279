"""Fine-grained allocation scheduler, step by step -- TEST INFRASTRUCTURE.

Alg. 1 of Section III-D in the paper's order and notation: memory-based allocation of L_i
layers per device, then for every #Stage s the overlap windows T_i^idle (Eq. (2)), the dynamic
program F_allo(l, i) with its predecessor table P_pre (Eqs. (3)-(4)), backtracking, the
feasibility test, and the refinement of the bottleneck device's offloaded layers into
block-level offloading; finally T_total of Eq. (1).  Integers throughout.

Readings (shared with the library's documentation of stage_allocate, decided from the paper,
not from the library): windows before offloading (L~_i empty), F_allo clamped at zero from the
first device on, "<=" updates over increasing k, a device infeasible when C_i + |L~_i| > s*C_i,
the refinement saving the load of the block that stays resident (MHA-only offloading keeps the
MLP block, and frees its load), the max-heap breaking ties by the lower device index, ties in
T_total to the smaller s.  Without left layers, devices take layers in order up to capacity,
#Stage = 1.
"""
from __future__ import annotations

import heapq
from typing import Dict, List, NamedTuple, Optional, Sequence, Tuple


class Device(NamedTuple):
    mem: int        # Mem_i, bytes
    comp: int       # comp of one layer
    load_mha: int   # load of one MHA block (p_A of a layer)
    load_mlp: int   # load of one MLP block (p_M of a layer)


class DevicePlan(NamedTuple):
    first_layer: int
    assigned: int   # |L_i|
    offloaded: int  # |L~_i|
    mha_only: int   # |L~_i^A| among them: MLP block resident
    mlp_only: int   # |L~_i^M| among them: MHA block resident


def chain_delay(loads: Sequence[int], idle: Sequence[int], shares: Sequence[int]) -> int:
    """The uncovered delay F_allo accumulates along the devices for one distribution of the
    left layers (the quantity the dynamic program minimises)."""
    f = 0
    for load, window, k in zip(loads, idle, shares):
        f = max(0, f + k * load - window)
    return f


def stage_alloc(s: int, n_left: int, devices: Sequence[Device], cap: Sequence[int], mem_left: Sequence[int],
                idle: Sequence[int], mha_bytes: int, mlp_bytes: int):
    """StageAlloc of Alg. 1: offloaded layers per device and their block-level refinement, or
    None when the stage count is infeasible."""
    D = len(devices)
    load = [d.load_mha + d.load_mlp for d in devices]
    INF = float("inf")
    F: Dict[Tuple[int, int], float] = {}
    P: Dict[Tuple[int, int], int] = {}
    for i in range(1, D + 1):
        F[(0, i)] = 0
    for l in range(1, n_left + 1):            # Eq. (3): the first device takes l offloaded layers
        F[(l, 1)] = max(0, l * load[0] - idle[0])
        P[(l, 1)] = l
    for i in range(2, D + 1):                 # Eq. (4)
        for l in range(1, n_left + 1):
            F[(l, i)] = INF
            for k in range(0, l + 1):
                t_cur = max(0, F[(l - k, i - 1)] + k * load[i - 1] - idle[i - 1])
                if t_cur <= F[(l, i)]:
                    F[(l, i)] = t_cur
                    P[(l, i)] = k
    offl = [0] * D                            # backtrack P_pre
    l = n_left
    for i in range(D, 1, -1):
        offl[i - 1] = P[(l, i)] if l > 0 else 0
        l -= offl[i - 1]
    offl[0] = l
    for i in range(D):                        # feasibility: one stage's layers within capacity
        if cap[i] + offl[i] > s * cap[i]:
            return None
    whole, mha_only, mlp_only = list(offl), [0] * D, [0] * D
    mem = list(mem_left)
    T = [whole[i] * load[i] for i in range(D)]
    heap = [(-T[i], i) for i in range(D)]
    heapq.heapify(heap)
    while heap:
        _, i = heapq.heappop(heap)
        if mem[i] >= mlp_bytes and whole[i] >= 1:        # MHA-only offloading: MLP block stays
            whole[i] -= 1
            mha_only[i] += 1
            mem[i] -= mlp_bytes
            T[i] -= devices[i].load_mlp
            heapq.heappush(heap, (-T[i], i))
        elif mem[i] >= mha_bytes and whole[i] >= 1:      # MLP-only offloading: MHA block stays
            whole[i] -= 1
            mlp_only[i] += 1
            mem[i] -= mha_bytes
            T[i] -= devices[i].load_mha
            heapq.heappush(heap, (-T[i], i))
        else:
            break
    return offl, whole, mha_only, mlp_only


def t_total(s: int, devices: Sequence[Device], assigned: Sequence[int], retained: Sequence[int],
            whole: Sequence[int], mha_only: Sequence[int], mlp_only: Sequence[int], comm: int) -> int:
    """Eq. (1): computing time, s * |D| hops, and the largest uncovered loading time."""
    D = len(devices)
    comp = [assigned[i] * devices[i].comp for i in range(D)]
    T_comp = sum(comp)
    T_comm = s * D * comm
    T_uncover = 0
    for i, d in enumerate(devices):
        load = whole[i] * (d.load_mha + d.load_mlp) + mha_only[i] * d.load_mha + mlp_only[i] * d.load_mlp
        window = retained[i] * d.comp + (T_comp - comp[i]) + D * comm
        T_uncover = max(T_uncover, max(0, load - window))
    return T_comp + T_comm + T_uncover


def allocate(n_layers: int, mha_bytes: int, mlp_bytes: int, comm: int,
             devices: Sequence[Device]) -> Optional[Tuple[int, int, List[DevicePlan]]]:
    """Alg. 1: (#Stage, T_total, per-device plans), or None when no stage count is feasible."""
    D = len(devices)
    l_size = mha_bytes + mlp_bytes
    cap = [d.mem // l_size for d in devices]             # memory-based allocation
    mem_left = [d.mem - c * l_size for d, c in zip(devices, cap)]
    n_left = n_layers - sum(cap)

    def plans(assigned, offl, mha_only, mlp_only):
        out, first = [], 0
        for i in range(D):
            out.append(DevicePlan(first, assigned[i], offl[i], mha_only[i], mlp_only[i]))
            first += assigned[i]
        return out

    if n_left <= 0:
        assigned, need = [], n_layers
        for c in cap:
            assigned.append(min(c, need))
            need -= assigned[-1]
        zero = [0] * D
        return 1, t_total(1, devices, assigned, assigned, zero, zero, zero, comm), plans(assigned, zero, zero, zero)

    best = None
    s_max = min(max(2, n_left), -(-n_layers // D))
    for s in range(2, s_max + 1):
        # Eq. (2) with nothing offloaded yet: own retained layers, the others' layers, the hops
        idle = [cap[i] * devices[i].comp + sum(cap[j] * devices[j].comp for j in range(D) if j != i) + D * comm
                for i in range(D)]
        res = stage_alloc(s, n_left, devices, cap, mem_left, idle, mha_bytes, mlp_bytes)
        if res is None:
            continue
        offl, whole, mha_only, mlp_only = res
        assigned = [cap[i] + offl[i] for i in range(D)]
        t = t_total(s, devices, assigned, cap, whole, mha_only, mlp_only, comm)
        if best is None or t < best[1]:
            best = (s, t, plans(assigned, offl, mha_only, mlp_only))
    return best
