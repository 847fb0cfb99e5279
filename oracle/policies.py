"""Integer policies of the stage runtime, written independently -- TEST INFRASTRUCTURE.

The HIP runtime must reproduce these bit-exactly (block tables, slot log,
residency changes).  Each is a reading of the paper where it leaves the detail
open; the readings are:

* Paged KV allocation.  One pool of blocks of ``block`` tokens shared by all
  sequences of the stage (one block id addresses the same block in every
  layer's pool).  Free blocks are handed out lowest id first.  A sequence takes
  a new block when it writes a position that is a multiple of ``block``.  Within
  a call, sequences allocate in call order (micro-batch ids in the order given,
  then batch rows ascending), each taking all blocks its new tokens need before
  the next.  A call that would exhaust the pool changes nothing.
* Residency is per block (Section III-D: a layer splits into its MHA block and
  its MLP block, each offloadable alone), given per layer as a code: 1 both
  resident, 0 both offloaded, 2 MHA block offloaded ("MHA-only offloading"),
  3 MLP block offloaded.
* Slot assignment (Section III-C: a reusable loading buffer is refilled once the
  GPU signals it is done with the previous layer).  A layer with any offloaded
  block is streamed.  The k-th layer load of the stage's life (k = 0, 1, ...)
  goes to slot k mod S.  Each call loads each streamed layer once, in ascending
  layer order, and runs it for every micro-batch of the call before its slot is
  reused.
* Residency schedule (Section III-E, online memory-aware planner: progressive
  offloading at token-length thresholds TS^j).  Before a call, let c be the
  longest sequence length in the stage once the call's tokens are appended.
  Every threshold TS^j <= c not yet applied offloads both blocks of one layer
  that still has a resident block, the highest id first, so with whole-layer
  residency a prefix of layers stays resident.
* Planner steps (Section III-E, Eq. (7): alpha more MHA blocks and beta more MLP
  blocks offloaded once the cache reaches a threshold; plans are not nested).
  Before a call, let h be the tokens the stage holds over all sequences once the
  call's tokens are appended; the last step with threshold <= h gives (alpha,
  beta), none below the first.  Starting from the allocation (the codes the
  layers were loaded with), the alpha highest-id layers whose MHA block it keeps
  resident offload that block, likewise beta MLP blocks; layers whose code
  differs from this target change, ascending, each change logged.
"""
from __future__ import annotations

import heapq
from typing import Dict, Hashable, Iterable, List, Optional, Sequence, Tuple

OFFLOADED, RESIDENT, MHA_OFFLOADED, MLP_OFFLOADED = 0, 1, 2, 3


class BlockAllocator:
    def __init__(self, n_blocks: int, block: int = 16):
        self.block = block
        self.free: List[int] = list(range(n_blocks))
        heapq.heapify(self.free)
        self.tables: Dict[Hashable, List[int]] = {}
        self.lengths: Dict[Hashable, int] = {}

    def _blocks_for(self, length: int) -> int:
        return -(-length // self.block)

    def need(self, key: Hashable, n_new: int) -> int:
        length = self.lengths.get(key, 0)
        return self._blocks_for(length + n_new) - len(self.tables.get(key, []))

    def call(self, keys_and_counts: Sequence[Tuple[Hashable, int]]) -> Dict[Hashable, List[int]]:
        """Append n tokens to each listed sequence, in the order given.  Returns new block ids."""
        total = sum(self.need(k, n) for k, n in keys_and_counts)
        if total > len(self.free):
            raise MemoryError("KV pool exhausted")
        new = {}
        for key, n in keys_and_counts:
            got = [heapq.heappop(self.free) for _ in range(self.need(key, n))]
            self.tables.setdefault(key, []).extend(got)
            self.lengths[key] = self.lengths.get(key, 0) + n
            new[key] = got
        return new

    def truncate(self, key: Hashable, n_drop: int) -> None:
        """Drop the last n_drop tokens; blocks left empty return to the pool."""
        length = self.lengths[key] - n_drop
        assert length >= 0
        keep = self._blocks_for(length)
        for b in self.tables[key][keep:]:
            heapq.heappush(self.free, b)
        self.tables[key] = self.tables[key][:keep]
        self.lengths[key] = length

    def release(self, key: Hashable) -> None:
        for b in self.tables.pop(key, []):
            heapq.heappush(self.free, b)
        self.lengths.pop(key, None)

    def table(self, key: Hashable) -> List[int]:
        return list(self.tables.get(key, []))


class SlotSchedule:
    """Which HBM slot each streamed-layer load goes to."""

    def __init__(self, n_slots: int):
        self.n_slots = n_slots
        self.loads = 0
        self.log: List[Tuple[int, int, int]] = []   # (call number, layer, slot)

    def call(self, call_no: int, streamed_layers: Iterable[int]) -> None:
        for layer in sorted(streamed_layers):
            self.log.append((call_no, layer, self.loads % self.n_slots))
            self.loads += 1


class ResidencySchedule:
    """Residency code of every layer and its threshold-driven shrinking.

    ``resident`` lists the wholly resident layers (the others offloaded), unless ``codes``
    gives every layer's code."""

    def __init__(self, n_layers: int, resident: Iterable[int] = (), thresholds: Sequence[int] = (),
                 codes: Optional[Sequence[int]] = None, plan: Optional[Sequence[Tuple[int, int, int]]] = None):
        self.n_layers = n_layers
        keep = set(resident)
        self.codes = list(codes) if codes is not None else [RESIDENT if l in keep else OFFLOADED
                                                            for l in range(n_layers)]
        assert len(self.codes) == n_layers
        self.allocation = list(self.codes)
        self.thresholds = list(thresholds)
        self.plan = None if plan is None else [tuple(p) for p in plan]
        self.applied = 0
        self.log: List[Tuple[int, int]] = []        # (call number, demoted layer), threshold schedule
        self.changes: List[Tuple[int, int, int]] = []   # (call number, layer, new code), either schedule

    def _plan_target(self, alpha: int, beta: int) -> List[int]:
        mha = [c in (RESIDENT, MLP_OFFLOADED) for c in self.allocation]   # MHA block resident
        mlp = [c in (RESIDENT, MHA_OFFLOADED) for c in self.allocation]
        for keep, count in ((mha, alpha), (mlp, beta)):
            for layer in reversed(range(self.n_layers)):
                if count == 0:
                    break
                if keep[layer]:
                    keep[layer] = False
                    count -= 1
        table = {(True, True): RESIDENT, (False, False): OFFLOADED, (False, True): MHA_OFFLOADED,
                 (True, False): MLP_OFFLOADED}
        return [table[(a, m)] for a, m in zip(mha, mlp)]

    def before_call_planned(self, call_no: int, held_after_call: int) -> None:
        alpha = beta = 0
        for tokens, a, b in self.plan:
            if tokens <= held_after_call:
                alpha, beta = a, b
        for layer, code in enumerate(self._plan_target(alpha, beta)):
            if code != self.codes[layer]:
                self.codes[layer] = code
                self.changes.append((call_no, layer, code))

    @property
    def resident(self) -> set:
        return {l for l, c in enumerate(self.codes) if c == RESIDENT}

    def before_call(self, call_no: int, longest_after_call: int) -> List[int]:
        demoted = []
        while self.applied < len(self.thresholds) and self.thresholds[self.applied] <= longest_after_call:
            self.applied += 1
            holders = [l for l, c in enumerate(self.codes) if c != OFFLOADED]
            if holders:
                layer = max(holders)
                self.codes[layer] = OFFLOADED
                demoted.append(layer)
                self.log.append((call_no, layer))
                self.changes.append((call_no, layer, OFFLOADED))
        return demoted

    def streamed(self) -> List[int]:
        return [l for l, c in enumerate(self.codes) if c != RESIDENT]
