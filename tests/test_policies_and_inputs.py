"""CPU checks of the oracle's integer policies (hand-enumerated tables) and of
the seeded input generator (published reference outputs, distribution)."""
import math
import os

import numpy as np
import pytest

import synth
from oracle.policies import BlockAllocator, ResidencySchedule, SlotSchedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- paged KV allocation
def test_block_allocation_hand_table():
    a = BlockAllocator(n_blocks=8, block=16)
    # one call: prefill 20 tokens for mb 1 then 5 for mb 0 (call order, not id order)
    new = a.call([((1, 0), 20), ((0, 0), 5)])
    assert new == {(1, 0): [0, 1], (0, 0): [2]}
    # decode: mb 1 goes to 21 (block 1 has room), mb 0 to 6
    assert a.call([((1, 0), 1), ((0, 0), 1)]) == {(1, 0): [], (0, 0): []}
    # mb 1 grows 21 -> 33: positions 32 needs block index 2 -> lowest free id 3
    assert a.call([((1, 0), 12)]) == {(1, 0): [3]}
    assert a.table((1, 0)) == [0, 1, 3] and a.lengths[(1, 0)] == 33
    # drop mb 1's last 17 tokens (33 -> 16): blocks 1 and 3 return
    a.truncate((1, 0), 17)
    assert a.table((1, 0)) == [0] and sorted(a.free) == [1, 3, 4, 5, 6, 7]
    # mb 0 grows 6 -> 40: needs blocks 1 and 2 of its table -> ids 1, 3
    assert a.call([((0, 0), 34)]) == {(0, 0): [1, 3]}
    assert a.table((0, 0)) == [2, 1, 3]


def test_block_allocation_exhaustion_changes_nothing():
    a = BlockAllocator(n_blocks=3, block=16)
    a.call([(("x", 0), 16)])
    before = (list(a.free), dict(a.lengths), {k: list(v) for k, v in a.tables.items()})
    with pytest.raises(MemoryError):
        a.call([(("y", 0), 16), (("x", 0), 32)])   # needs 1 + 2 > 2 free
    assert (list(a.free), dict(a.lengths), {k: list(v) for k, v in a.tables.items()}) == before


def test_block_release_returns_lowest_first():
    a = BlockAllocator(n_blocks=6, block=4)
    a.call([("a", 9), ("b", 4)])          # a: 0,1,2  b: 3
    a.release("a")
    assert a.call([("c", 5)]) == {"c": [0, 1]}


# ----------------------------------------------------------------- slot assignment
def test_slot_log_hand_table():
    s = SlotSchedule(n_slots=2)
    s.call(0, [6, 4, 5])
    s.call(1, [4, 5, 6])
    assert s.log == [(0, 4, 0), (0, 5, 1), (0, 6, 0), (1, 4, 1), (1, 5, 0), (1, 6, 1)]
    s3 = SlotSchedule(n_slots=3)
    s3.call(7, range(4, 16))
    assert [slot for _, _, slot in s3.log] == [0, 1, 2] * 4


# ----------------------------------------------------------------- residency schedule
def test_residency_thresholds_hand_table():
    r = ResidencySchedule(16, range(16), thresholds=[512 + 960 * j for j in range(1, 9)])
    assert r.before_call(0, 512) == []
    assert r.before_call(1, 1471) == []
    assert r.before_call(2, 1472) == [15]
    assert r.before_call(3, 2431) == []
    assert r.before_call(4, 8192) == [14, 13, 12, 11, 10, 9, 8]
    assert sorted(r.resident) == list(range(8))
    assert r.streamed() == list(range(8, 16))
    assert r.before_call(5, 100000) == []


def test_residency_one_demotion_per_round():
    r = ResidencySchedule(4, range(4), thresholds=[33, 34, 35])
    assert [r.before_call(c, 32 + c) for c in range(5)] == [[], [3], [2], [1], []]


def test_residency_codes_block_granular():
    """Layers with one offloaded block stream; a threshold offloads both blocks of the highest
    layer holding any resident block."""
    r = ResidencySchedule(5, thresholds=[10, 20, 30], codes=[1, 1, 2, 3, 0])
    assert r.streamed() == [2, 3, 4] and r.resident == {0, 1}
    assert r.before_call(0, 10) == [3]
    assert r.codes == [1, 1, 2, 0, 0]
    assert r.before_call(1, 30) == [2, 1]
    assert r.codes == [1, 0, 0, 0, 0] and r.streamed() == [1, 2, 3, 4]
    s = SlotSchedule(n_slots=2)
    s.call(0, r.streamed())
    assert s.log == [(0, 1, 0), (0, 2, 1), (0, 3, 0), (0, 4, 1)]


def test_planned_residency_hand_table():
    """Planner steps (Section III-E, Eq. (7)) over an allocation that mixes whole-layer, MHA-only and
    MLP-only offloading: the alpha MHA blocks and beta MLP blocks come from the highest-id layers
    whose block the allocation keeps resident (a layer whose MHA block is already offloaded is not
    counted again), plans are not nested (a later step brings MHA blocks back), and the plan
    follows the token count down to the allocation.  Expected codes written out by hand."""
    alloc = [1, 3, 1, 2, 1, 1]          # layer 1: MLP offloaded; layer 3: MHA offloaded
    plan = [(100, 1, 0), (200, 3, 0), (300, 0, 1), (400, 2, 2), (900, 9, 0)]
    r = ResidencySchedule(6, codes=alloc, plan=plan)
    expect = [
        # (held tokens, codes after the call's step, changes logged by that call)
        (50, [1, 3, 1, 2, 1, 1], []),                                # below the first threshold
        (100, [1, 3, 1, 2, 1, 2], [(5, 2)]),                         # MHA of layer 5
        (150, [1, 3, 1, 2, 1, 2], []),                               # same step: nothing moves
        (250, [1, 3, 2, 2, 2, 2], [(2, 2), (4, 2)]),                 # MHA of 5, 4, 2 (3 has none)
        (350, [1, 3, 1, 2, 1, 3], [(2, 1), (4, 1), (5, 3)]),         # MHA back; MLP of layer 5
        (450, [1, 3, 1, 2, 0, 0], [(4, 0), (5, 0)]),                 # MHA of 5, 4 and MLP of 5, 4
        (120, [1, 3, 1, 2, 1, 2], [(4, 1), (5, 2)]),                 # cache shrank: step (1, 0)
        (10, [1, 3, 1, 2, 1, 1], [(5, 1)]),                          # back to the allocation
        (1000, [2, 0, 2, 2, 2, 2], [(0, 2), (1, 0), (2, 2), (4, 2), (5, 2)]),   # alpha > 5 blocks
    ]
    for call, (held, codes, changes) in enumerate(expect):
        before = len(r.changes)
        r.before_call_planned(call, held)
        assert r.codes == codes, (call, r.codes)
        assert r.changes[before:] == [(call, l, c) for l, c in changes], (call, r.changes[before:])
    assert r.allocation == alloc
    assert r.streamed() == [0, 1, 2, 3, 4, 5]


# ----------------------------------------------------------------- generator
def test_splitmix64_matches_published_reference():
    ref = [int(l) for l in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) if l.strip() and l[0] != "#"]
    assert synth.draws(1234567, 5).tolist() == ref


def test_box_muller_definition_on_first_elements():
    seed = synth.seed_of(1, 2, 3)
    d = synth.draws(seed, 8)
    z = synth.normal_f32(seed, (8,))
    for i in range(8):
        p = i // 2
        u1 = ((int(d[2 * p]) >> 11) + 0.5) * 2.0 ** -53
        u2 = (int(d[2 * p + 1]) >> 11) * 2.0 ** -53
        r = math.sqrt(-2 * math.log(u1))
        ang = 2 * math.pi * u2
        want = r * (math.sin(ang) if i % 2 else math.cos(ang))
        assert z[i] == np.float32(want)


def test_generator_distribution_and_offsets():
    x = synth.normal_f32(99, (2_000_000,))
    assert abs(float(x.mean())) < 5 / math.sqrt(2e6)
    assert abs(float(x.std()) - 1) < 5e-3
    assert np.array_equal(synth.normal_f32(99, (999,), offset=1001), x[1001:2000])
    w = synth.bf16_to_f32(synth.normal_bf16(7, (1_000_000,), std=0.02))
    assert abs(float(w.std()) - 0.02) < 2e-4
    assert np.all((w.view(np.uint32) & 0xFFFF) == 0)


def test_layer_weights_shapes_and_seeding():
    w0 = synth.layer_weights(synth.TINY, 0)
    w1 = synth.layer_weights(synth.TINY, 1)
    shapes = synth.layer_weight_shapes(synth.TINY)
    assert {k: v.shape for k, v in w0.items()} == shapes
    assert not np.array_equal(w0["wq"], w1["wq"])
    assert np.array_equal(w0["wq"], synth.layer_weights(synth.TINY, 0)["wq"])
    g = synth.bf16_to_f32(w0["g1"])
    assert abs(float(g.mean()) - 1) < 0.01
