"""Slot tag check mode (stage_config.slot_check): the runtime evidence that a reusable slot is read
only after its copy has completed and refilled only after the kernels reading it have finished
(Section III-C: ready signal and buffer reuse).  Correct runs only: with the check on, every tag
matches, the outputs are those of the unchecked stage bit for bit, and the number of checks run is
the number enqueued.  The detection path is exercised by the self-test mode, which asks the checks
before MHA blocks for the next load number: they fail, are reported by stage_sync, and change no
weight and no output."""
import dataclasses

import numpy as np
import pytest

import synth
from tests.harness import Scenario, run_gpu

pytestmark = pytest.mark.gpu

# 8B-shaped layers, 3 micro-batches of batch 3; every residency kind: resident, both blocks
# offloaded, MHA only, MLP only; two slots for six layers that stream
WL = synth.Workload("llama8b_slotcheck", 104, synth.LLAMA8B_STAGE, n_mb=3, batch=3, prefill=24, decode_steps=3)
CODES = (1, 0, 2, 3, 0, 2, 3, 0)


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _checks_per_call(codes):
    # one check before and one after each offloaded block of each streamed layer
    return sum(2 * ((c in (0, 2)) + (c in (0, 3))) for c in codes)


@pytest.mark.parametrize("calls,slots", [("one", 2), ("all", 3)])
def test_slot_check_passes_and_changes_nothing(calls, slots):
    _gpu()
    base = Scenario(WL, prefill=WL.prefill, decode_steps=WL.decode_steps, calls=calls, residency=CODES,
                    slots=slots)
    ref = run_gpu(base)
    got = run_gpu(dataclasses.replace(base, slot_check=1))   # stage_sync inside raises on a mismatch
    assert len(got.outputs) == len(ref.outputs)
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    assert got.slot_log == ref.slot_log
    st = got.stats
    n_calls = len(base.call_plan())
    assert st["slot_check"] == 1
    assert st["slot_checks"] == n_calls * _checks_per_call(CODES)
    assert st["slot_checks_run"] == st["slot_checks"]
    assert st["slot_check_failures"] == 0
    assert ref.stats["slot_checks"] == 0


def test_slot_check_self_test_reports_mismatches():
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    from tests.harness import compute_stream, weights_of
    shape = WL.shape
    w = weights_of(shape)
    x = torch.from_numpy(np.stack([synth.prefill_inputs(WL, 0, b, WL.prefill) for b in range(WL.batch)])[None]).cuda()
    outs = {}
    for mode in (0, 2):
        with compute_stream() as cs:
            cfg = P.config_for(shape, max_microbatches=WL.n_mb, max_batch=WL.batch, max_context=64,
                               n_resident_max=sum(c != 0 for c in CODES), compute_stream=cs.handle,
                               slot_check=mode)
            h = P.stage_init(cfg)
            try:
                for l, c in enumerate(CODES):
                    P.stage_load_layer(h, l, w(l), c)
                y = torch.empty_like(x)
                P.stage_prefill(h, [0], WL.batch, WL.prefill, x, y)
                if mode == 2:
                    with pytest.raises(P.StageError) as ei:
                        P.stage_sync(h)
                    assert ei.value.code == P.STAGE_ESLOT
                    msg = str(ei.value)
                    n_mha = sum(c in (0, 2) for c in CODES)
                    assert f"{n_mha} slot tag check(s) failed" in msg
                    # the first streamed layer with an offloaded MHA block is layer 1, load 0
                    assert "before the MHA block's kernels expected layer 1 load 1, found layer 1 load 0" in msg
                    st = P.stage_get_stats(h)
                    assert st["slot_check_failures"] == n_mha
                    assert st["slot_checks_run"] == _checks_per_call(CODES)
                    P.stage_sync(h)   # reported once: the record was cleared
                else:
                    P.stage_sync(h)
                outs[mode] = y.cpu().numpy()
            finally:
                P.stage_destroy(h)
    assert np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("kind", ["thresholds", "planner", "zero_copy"])
def test_slot_check_under_changing_residency(kind):
    """The tags follow the stage's own slot use when residency changes between calls (threshold
    demotions; planner steps that offload and reload blocks) and when only prefills stage (zero
    copy decode): every check passes, and the outputs equal the unchecked stage's."""
    _gpu()
    tiny = synth.Workload("tiny_slotcheck", 105, synth.TINY, n_mb=3, batch=2, prefill=37, decode_steps=6)
    if kind == "thresholds":
        base = Scenario(tiny, prefill=37, decode_steps=6, calls="one", thresholds=(39, 40, 41))
    elif kind == "planner":
        # held tokens grow 37 per prefill and 2 per decode call: the steps offload one MHA block,
        # then one MLP block and reload the MHA block
        base = Scenario(tiny, prefill=37, decode_steps=6, calls="one", residency=(1, 1),
                        plan=((100, 1, 0), (230, 0, 1)))
    else:
        base = Scenario(tiny, prefill=37, decode_steps=6, calls="one", n_resident=0, zero_copy=True)
    ref = run_gpu(base)
    got = run_gpu(dataclasses.replace(base, slot_check=1))
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    assert got.slot_log == ref.slot_log and got.residency_log == ref.residency_log
    st = got.stats
    assert st["slot_checks"] > 0
    assert st["slot_checks_run"] == st["slot_checks"]
    assert st["slot_check_failures"] == 0


def test_slot_check_on_the_70b_streamed_stage():
    """The 70B-shaped stage with 4 resident and 12 streamed layers through 2 slots, its copies
    overlapping compute on the library's own copy stream: 4 micro-batches, a 64-token prefill each
    in one call, then 16 decode calls of all four.  Every tag check passes (each call refills the
    two slots six times each while the previous layer's kernels still read the other), and the
    outputs equal the unchecked stage's."""
    _gpu()
    wl = synth.WORKLOADS["llama70b_offload"]
    base = Scenario(wl, prefill=64, decode_steps=16, calls="all", n_resident=4)
    ref = run_gpu(base)
    got = run_gpu(dataclasses.replace(base, slot_check=1))
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    st = got.stats
    assert st["layer_loads"] == 12 * 17
    assert st["slot_checks"] == 17 * 12 * 4      # 12 streamed layers x 2 blocks x (before + after)
    assert st["slot_checks_run"] == st["slot_checks"]
    assert st["slot_check_failures"] == 0
