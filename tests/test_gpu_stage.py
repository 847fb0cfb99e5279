"""GPU parity of the HIP stage (through the C ABI) against the float64 CPU oracle.

Tolerance (stated for the stage output): max |GPU - oracle| <= 2e-2 and cosine >=
0.9995, on the output and on the stage contribution (output - input).  Integer
state -- block tables, slot log, demotions -- must match the oracle's independent
policies exactly.  Offloading must not change a single bit (lossless).
"""
import dataclasses

import numpy as np
import pytest

import synth
from tests.harness import (Scenario, bf16_kv_tolerance, compare, compute_stream, run_gpu, run_oracle, teacher_forced,
                           weights_of)

pytestmark = pytest.mark.gpu

TOL_ABS = 2e-2
TOL_COS = 0.9995

TINY_RAGGED = synth.Workload("tiny_ragged", 100, synth.TINY, n_mb=3, batch=2, prefill=37, decode_steps=20)
# 8B-shaped layers, 3 micro-batches of batch 3: 9 rows per call when all share it, 3 otherwise
LLAMA8B_MULTI = synth.Workload("llama8b_multi", 101, synth.LLAMA8B_STAGE, n_mb=3, batch=3, prefill=24,
                               decode_steps=3)
# row counts that stay on one decode engine under both groupings: 1 vs 2 rows (vector), 8 vs 16
# (matrix cores); and 2 vs 6 rows, one call of each engine
TINY_2x1 = synth.Workload("tiny_2x1", 102, synth.TINY, n_mb=2, batch=1, prefill=37, decode_steps=4)
LLAMA8B_2x8 = synth.Workload("llama8b_2x8", 103, synth.LLAMA8B_STAGE, n_mb=2, batch=8, prefill=24,
                             decode_steps=3)
LLAMA8B_3x2 = synth.Workload("llama8b_3x2", 104, synth.LLAMA8B_STAGE, n_mb=3, batch=2, prefill=24,
                             decode_steps=3)


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def check(name, sc, got, ref, tol_abs=TOL_ABS):
    m = compare(got.flat_out(), ref.flat_out(), got.flat_in(), ref.flat_in())
    print(f"\n[{name}] {m}", flush=True)
    assert m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m
    assert m["max_abs"] <= tol_abs, m
    assert got.block_tables == ref.block_tables
    assert got.slot_log == ref.slot_log
    assert got.demotion_log == ref.demotion_log
    assert got.residency_log == ref.residency_log
    assert got.residency == ref.residency
    return m


@pytest.mark.parametrize("kv_fp32", [False, True])
def test_tiny_feedback_matches_oracle(kv_fp32):
    _gpu()
    sc = Scenario(synth.WORKLOADS["tiny"], prefill=16, decode_steps=16, kv_fp32=kv_fp32)
    check(f"tiny kv_fp32={kv_fp32}", sc, run_gpu(sc), run_oracle(sc))


@pytest.mark.parametrize("calls", ["one", "all"])
def test_tiny_ragged_multi_sequence(calls):
    _gpu()
    sc = Scenario(TINY_RAGGED, prefill=37, decode_steps=20, calls=calls)
    check(f"tiny ragged calls={calls}", sc, run_gpu(sc), run_oracle(sc))


@pytest.mark.parametrize("slots", [1, 2, 3])
def test_streamed_layers_are_lossless(slots):
    """Offloaded layers streamed through S slots give the all-resident outputs bit for bit."""
    _gpu()
    base = Scenario(TINY_RAGGED, prefill=37, decode_steps=6, calls="all")
    ref = run_gpu(base)
    sc = dataclasses.replace(base, n_resident=0, slots=slots)
    got = run_gpu(sc)
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    orc = run_oracle(sc)
    assert got.slot_log == orc.slot_log
    assert got.residency == [0, 0]
    assert got.stats["layer_loads"] == 2 * len(sc.call_plan())


@pytest.mark.parametrize("wl,prefill,steps", [(TINY_RAGGED, 37, 6), (LLAMA8B_MULTI, 24, 3)])
def test_zero_copy_decode_equals_slot_staging(wl, prefill, steps):
    """Decode kernels reading the offloaded layers from pinned host memory give the slot-staged
    outputs bit for bit; only prefill calls load slots, and every decode call reads each offloaded
    layer once over the host link."""
    _gpu()
    staged = Scenario(wl, prefill=prefill, decode_steps=steps, calls="all", n_resident=1)
    direct = dataclasses.replace(staged, zero_copy=True)
    ref = run_gpu(staged)
    got = run_gpu(direct)
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    orc = run_oracle(direct, floats=False)
    assert got.slot_log == orc.slot_log
    assert all(call == 0 for call, _, _ in got.slot_log)
    n_off = wl.shape.n_layers - 1
    assert got.stats["layer_loads"] == n_off
    assert got.stats["bytes_direct"] == steps * n_off * got.stats["layer_bytes"]
    assert ref.stats["bytes_direct"] == 0


@pytest.mark.parametrize("wl,prefill,steps,codes,zero_copy", [
    (TINY_RAGGED, 37, 6, (2, 3), False),
    (TINY_RAGGED, 37, 6, (3, 0), True),
    (LLAMA8B_MULTI, 24, 3, (1, 2, 3, 0, 2, 3, 1, 0), False),
])
def test_block_offload_is_lossless(wl, prefill, steps, codes, zero_copy):
    """MHA-only and MLP-only offloading (Section III-D) give the all-resident outputs bit for bit;
    every layer with an offloaded block takes one slot load per staged call, and exactly the
    offloaded blocks cross the host link."""
    _gpu()
    base = Scenario(wl, prefill=prefill, decode_steps=steps, calls="all")
    ref = run_gpu(base)
    sc = dataclasses.replace(base, residency=codes, zero_copy=zero_copy)
    got = run_gpu(sc)
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    orc = run_oracle(sc, floats=False)
    assert got.slot_log == orc.slot_log
    assert got.residency == list(codes)
    st = got.stats
    per_call = sum((c in (0, 2)) * st["mha_block_bytes"] + (c in (0, 3)) * st["mlp_block_bytes"] for c in codes)
    staged_calls = 1 if zero_copy else 1 + steps
    assert st["bytes_streamed"] == staged_calls * per_call
    assert st["bytes_direct"] == (steps * per_call if zero_copy else 0)
    assert st["offloaded_mha_blocks"] == sum(c in (0, 2) for c in codes)
    assert st["offloaded_mlp_blocks"] == sum(c in (0, 3) for c in codes)


def test_block_residency_changes_between_calls_and_budget():
    """Blocks move between HBM and host memory between calls without changing a bit; the weight
    budget is counted in bytes, so one layer's worth holds the MHA block of one layer and the MLP
    block of another."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape = synth.TINY
    w = weights_of(shape)
    wl = TINY_RAGGED
    cs = compute_stream().__enter__()
    x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 37)).cuda()
    steps = [torch.from_numpy(synth.decode_input(wl, 0, 0, t)[None]).cuda() for t in range(4)]

    def run(budget, codes_per_call):
        cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=budget,
                           compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            for l in range(2):
                P.stage_load_layer(h, l, w(l), codes_per_call[0][l])
            P.stage_prefill(h, [0], 1, 37, x, torch.empty_like(x))
            outs = []
            for t, xt in enumerate(steps):
                for l, c in enumerate(codes_per_call[t + 1]):
                    P.stage_load_layer(h, l, None, c)
                y = torch.empty_like(xt)
                P.stage_decode(h, [0], 1, xt, y)
                outs.append(y)
            P.stage_sync(h)
            return [o.cpu() for o in outs], P.stage_get_residency(h, 2), P.stage_get_stats(h)
        finally:
            P.stage_destroy(h)

    ref, _, st = run(2, [(1, 1)] * 5)
    assert st["host_weight_bytes"] == 0
    plan = [(1, 1), (2, 3), (3, 2), (0, 1), (1, 0)]
    got, res, st = run(2, plan)
    assert res == [1, 0]
    assert st["host_weight_bytes"] == 2 * st["layer_bytes"]     # host copies kept once made
    for a, b in zip(got, ref):
        assert torch.equal(a, b)
    # budget of one layer: MHA of layer 0 plus MLP of layer 1 fit, a whole extra layer does not
    got, res, st = run(1, [(3, 2)] * 5)
    assert res == [3, 2] and st["hbm_weight_bytes"] == st["layer_bytes"] * (1 + st["stream_slots"])
    for a, b in zip(got, ref):
        assert torch.equal(a, b)
    cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=1,
                       compute_stream=cs.handle)
    h = P.stage_init(cfg)
    try:
        P.stage_load_layer(h, 0, w(0), P.STAGE_RES_MLP_OFFLOADED)
        P.stage_load_layer(h, 1, w(1), P.STAGE_RES_MHA_OFFLOADED)
        with pytest.raises(P.StageError) as e:
            P.stage_load_layer(h, 0, None, P.STAGE_RES_RESIDENT)
        assert e.value.code == P.STAGE_ENOMEM
        assert P.stage_get_residency(h, 2) == [3, 2]
        with pytest.raises(P.StageError) as e:
            P.stage_load_layer(h, 0, None, 4)
        assert e.value.code == P.STAGE_EINVAL
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def test_attention_starts_before_the_mlp_block_arrives():
    """Per-block readiness: a streamed layer's kernels start once its MHA block is in the slot,
    while its MLP block is still being copied, and finish after that copy (8B-shaped layers, all
    streamed, events on both streams)."""
    _gpu()
    import paper_2512_21835_amd as P
    wl = LLAMA8B_MULTI
    sc = Scenario(wl, prefill=24, decode_steps=2, calls="all", n_resident=0,
                  timing=P.STAGE_TIME_CALLS | P.STAGE_TIME_LAYERS)
    got = run_gpu(sc)
    ref = run_gpu(dataclasses.replace(sc, n_resident=None, timing=0))
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    tl = got.timeline
    ends = [i for i, r in enumerate(tl) if r[0] == 0]
    seg = tl[ends[-2] + 1: ends[-1] + 1]          # the last decode call
    mha_copy = {int(l): (a, b) for k, l, a, b in seg if k == 1}
    mlp_copy = {int(l): (a, b) for k, l, a, b in seg if k == 4}
    mha_comp = {int(l): (a, b) for k, l, a, b in seg if k == 3}
    mlp_comp = {int(l): (a, b) for k, l, a, b in seg if k == 5}
    layers = list(range(wl.shape.n_layers))
    assert sorted(mha_copy) == sorted(mlp_copy) == sorted(mha_comp) == sorted(mlp_comp) == layers
    for l in layers:
        assert mha_copy[l][1] <= mha_comp[l][0] + 1e-3    # MHA block in place before attention starts
        assert mha_comp[l][1] < mlp_copy[l][1]            # attention done while the MLP block streams
        assert mlp_comp[l][0] >= mlp_copy[l][1] - 1e-3    # the MLP kernels waited for it
        assert mlp_comp[l][0] >= mha_comp[l][1] - 1e-3


def test_streaming_overlaps_compute_whatever_streams_the_process_made():
    """Loading under computation (Section III-A; the reusable buffer refilled on the GPU's signal,
    Section III-C) must not depend on the caller's other streams.  HIP shares a few hardware queues
    among a process's streams in creation order, so the process first creates 8 more streams and
    then, for four consecutive positions of the compute stream in that order, builds an 8B-shaped
    stage whose 8 layers all stream through 2 slots on the library's own copy stream, and times a
    decode call (3 micro-batches of batch 3): the layer kernels must run under the slot copies
    (hidden-shorter >= 0.8), and the call must take about the copy time alone."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    from tests.harness import overlap_of_last_call

    wl = LLAMA8B_MULTI
    shape = wl.shape
    weights = weights_of(shape)
    others = [torch.cuda.Stream() for _ in range(8)]
    x = torch.from_numpy(np.stack([np.stack([synth.prefill_inputs(wl, m, b, 8) for b in range(wl.batch)])
                                   for m in range(wl.n_mb)])).cuda()
    xd = x[:, :, 0].contiguous()
    for shift in range(4):
        others += [torch.cuda.Stream() for _ in range(shift)]
        cs = torch.cuda.Stream()
        with torch.cuda.stream(cs):
            cfg = P.config_for(shape, max_microbatches=wl.n_mb, max_batch=wl.batch, max_context=16, n_resident_max=0,
                               compute_stream=cs.cuda_stream)
            h = P.stage_init(cfg)
            try:
                for l in range(shape.n_layers):
                    P.stage_load_layer(h, l, weights(l), 0)
                y = torch.empty_like(x)
                P.stage_prefill(h, list(range(wl.n_mb)), wl.batch, 8, x, y)
                yd = torch.empty_like(xd)
                P.stage_decode(h, list(range(wl.n_mb)), wl.batch, xd, yd)
                P.stage_sync(h)
                P.stage_get_timeline(h)
                P.stage_set_timing(h, P.STAGE_TIME_CALLS | P.STAGE_TIME_LAYERS)
                for _ in range(2):
                    P.stage_decode(h, list(range(wl.n_mb)), wl.batch, xd, yd)
                tl = P.stage_get_timeline(h)
            finally:
                P.stage_destroy(h)
        ov = overlap_of_last_call(tl)
        call = [b - a for k, _, a, b in tl if k == 0][-1]
        print(f"\n[overlap, compute stream shifted by {shift}] {ov}, call {call:.3f} ms", flush=True)
        assert ov["hidden_shorter"] >= 0.8, (shift, ov)
        assert call <= 1.1 * ov["copy_ms"] + 0.5, (shift, call, ov)


@pytest.mark.parametrize("zero_copy", [False, True])
def test_planner_steps_drive_block_residency(zero_copy):
    """Steps of the online planner (Eq. (7), computed by stage_plan_offload for a device whose
    cache takes 8 KiB per token) applied while six ragged sequences grow: blocks leave and come
    back (an MHA block is reloaded when the plan swaps it for an MLP block) exactly as the
    oracle's policy says, and no output bit changes."""
    _gpu()
    import paper_2512_21835_amd as P
    base = Scenario(TINY_RAGGED, prefill=37, decode_steps=20, calls="one")
    ref = run_gpu(base)
    st = ref.stats
    steps, _ = P.stage_plan_offload(120 * 8192, 8192, st["mha_block_bytes"], st["mlp_block_bytes"],
                                    st["mha_block_bytes"], st["mlp_block_bytes"], 2, 2, 2)
    assert any(b[1] < a[1] for a, b in zip(steps, steps[1:]))     # a later step reloads MHA blocks
    sc = dataclasses.replace(base, plan=tuple(steps), zero_copy=zero_copy)
    got = run_gpu(sc)
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)
    orc = run_oracle(sc, floats=False)
    assert got.residency_log == orc.residency_log and len(got.residency_log) >= 4
    assert got.slot_log == orc.slot_log
    assert got.residency == orc.residency
    assert got.demotion_log == []


def test_planner_reloads_blocks_when_the_cache_shrinks():
    """The plan follows the token count down: dropping a sequence brings offloaded blocks back
    at the next call."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape = synth.TINY
    w = weights_of(shape)
    wl = TINY_RAGGED
    cs = compute_stream().__enter__()
    cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=64, n_resident_max=2,
                       compute_stream=cs.handle, plan=[(0, 0, 0), (60, 1, 0), (70, 2, 1)])
    h = P.stage_init(cfg)
    try:
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 1)
        x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 37)).cuda()
        P.stage_prefill(h, [0], 1, 37, x, torch.empty_like(x))           # 37 tokens: allocation
        assert P.stage_get_residency(h, 2) == [1, 1]
        P.stage_prefill(h, [1], 1, 37, x, torch.empty_like(x))           # 74: two MHA + one MLP out
        assert P.stage_get_residency(h, 2) == [2, 0]
        P.stage_reset_sequence(h, 1, 0)
        xt = torch.from_numpy(synth.decode_input(wl, 0, 0, 0)[None]).cuda()
        P.stage_decode(h, [0], 1, xt, torch.empty_like(xt))               # 38: back to the allocation
        P.stage_sync(h)
        assert P.stage_get_residency(h, 2) == [1, 1]
        assert P.stage_get_residency_log(h) == [(1, 0, 2), (1, 1, 0), (2, 0, 1), (2, 1, 1)]
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def _one_vs_all(wl, prefill, steps):
    """(rows of the round robin, rows of the one-call run, their common inputs) per call group."""
    a = run_gpu(Scenario(wl, prefill=prefill, decode_steps=steps, calls="one"))
    b = run_gpu(Scenario(wl, prefill=prefill, decode_steps=steps, calls="all"))
    H, n = wl.shape.hidden, wl.n_mb
    rows = lambda outs: np.concatenate([o.reshape(-1, H) for o in outs])
    out = [(rows(a.outputs[:n]), b.outputs[0].reshape(-1, H), rows(a.inputs[:n]))]
    for s in range(steps):
        grp = slice(n + n * s, 2 * n + n * s)
        out.append((rows(a.outputs[grp]), b.outputs[1 + s].reshape(-1, H), rows(a.inputs[grp])))
    for one, all_, x in out:
        assert x.shape == one.shape == all_.shape
    return out


@pytest.mark.parametrize("wl,prefill,steps", [(TINY_2x1, 37, 4), (LLAMA8B_2x8, 24, 3)])
def test_round_robin_equals_all_in_one_call_bitwise(wl, prefill, steps):
    """Per-row arithmetic does not depend on how many micro-batches share a call, as long as the
    decode projections run on the same engine: 1 vs 2 rows per call on the vector kernels (tiny
    shape), 8 vs 16 rows per call on the matrix cores (8B shape)."""
    _gpu()
    for one, all_, _ in _one_vs_all(wl, prefill, steps):
        assert np.array_equal(one, all_)


@pytest.mark.parametrize("wl,prefill,steps", [(TINY_RAGGED, 37, 4), (LLAMA8B_3x2, 24, 3)])
def test_vector_and_matrix_engines_agree(wl, prefill, steps):
    """Calls of 2 rows (vector kernels) and of 6 rows (matrix cores) give the same rows up to
    rounding: prefill bit for bit (the prefill GEMM is row-count independent), decode within the
    parity bound (the engines round differently, and a decode row's K/V can round to a neighbouring
    bf16 value, which the later steps carry)."""
    _gpu()
    for i, (one, all_, x) in enumerate(_one_vs_all(wl, prefill, steps)):
        if i == 0:
            assert np.array_equal(one, all_)
            continue
        m = compare(one, all_, x, x)
        print(f"\n[engines {wl.name} decode step {i - 1}] max|d| {m['max_abs']:.3g} cos {m['cos']:.10f} "
              f"cos(out - in) {m['cos_delta']:.10f}")
        assert m["max_abs"] <= TOL_ABS and m["cos"] >= 0.99999 and m["cos_delta"] >= TOL_COS, m


LLAMA8B_4x1 = synth.Workload("llama8b_4x1", 106, synth.LLAMA8B_STAGE, n_mb=4, batch=1, prefill=70,
                             decode_steps=3)


@pytest.mark.parametrize("alternate", [False, True])
def test_lanes_equal_one_lane_bitwise(alternate):
    """Prefills and round-robin decode of four micro-batches on two lanes (micro-batch m's prefill
    on lane m mod 2; each call on its lane's stream, inputs ordered on that stream) give the rows
    of the one-lane run bit for bit.  alternate: a micro-batch's decode steps switch lanes every
    step, so each step must wait for the previous one on the other lane."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    from tests.harness import _inputs, compute_stream

    wl = LLAMA8B_4x1
    sc = Scenario(wl, prefill=70, decode_steps=3)
    ref = run_gpu(sc)
    shape, H = wl.shape, wl.shape.hidden
    weights = weights_of(shape)
    with compute_stream() as cs:
        lane1 = torch.cuda.Stream()
        streams = [cs.stream, lane1]
        cfg = P.config_for(shape, max_microbatches=wl.n_mb, max_batch=1, max_context=sc.ctx(),
                           n_resident_max=shape.n_layers, compute_stream=cs.handle, n_lanes=2,
                           lane_streams=[None, lane1.cuda_stream])
        h = P.stage_init(cfg)
        outs, keep = [], []
        try:
            for l in range(shape.n_layers):
                P.stage_load_layer(h, l, weights(l), 1)
            for kind, mbs, step in sc.call_plan():
                x = _inputs(sc, kind, mbs, step, {})
                m = mbs[0]
                lane = m % 2 if kind == "prefill" else ((m + step) % 2 if alternate else m % 2)
                with torch.cuda.stream(streams[lane]):
                    x_in = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
                    x_out = torch.empty_like(x_in)
                if kind == "prefill":
                    P.stage_prefill_lane(h, lane, mbs, 1, x.shape[2], x_in, x_out)
                else:
                    P.stage_decode_lane(h, lane, mbs, 1, x_in, x_out)
                outs.append(x_out)
                keep.append(x_in)
            P.stage_sync(h)
            got = [o.cpu().numpy() for o in outs]
            with pytest.raises(P.StageError):
                P.stage_decode_lane(h, 2, [0], 1, keep[-1], outs[-1])   # only lanes 0 and 1
        finally:
            P.stage_destroy(h)
    assert len(got) == len(ref.outputs)
    for c, (a, b) in enumerate(zip(got, ref.outputs)):
        assert np.array_equal(a, b), f"call {c} differs"


def test_decode_lanes_refuse_streamed_layers():
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    from tests.harness import compute_stream

    shape = synth.TINY
    weights = weights_of(shape)
    with compute_stream() as cs:
        cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=32, n_resident_max=1,
                           compute_stream=cs.handle, n_lanes=2)
        h = P.stage_init(cfg)
        try:
            P.stage_load_layer(h, 0, weights(0), 1)
            P.stage_load_layer(h, 1, weights(1), 0)                     # streamed through the slots
            x = torch.zeros(1, 1, 4, shape.hidden, device="cuda")
            y = torch.empty_like(x)
            P.stage_prefill(h, [0], 1, 4, x, y)
            xd, yd = x[:, :, 0].contiguous(), torch.empty_like(x[:, :, 0]).contiguous()
            with pytest.raises(P.StageError) as e:
                P.stage_decode_lane(h, 1, [0], 1, xd, yd)
            assert e.value.code == P.STAGE_ESTATE
            P.stage_decode_lane(h, 0, [0], 1, xd, yd)                   # lane 0 streams as before
            P.stage_sync(h)
        finally:
            P.stage_destroy(h)


def test_threshold_demotions_follow_schedule_and_stay_lossless():
    _gpu()
    ths = (39, 40, 41)   # prefill 37: decode rounds 2, 3, 4 each demote one layer (2 layers: 2 demotions)
    sc = Scenario(TINY_RAGGED, prefill=37, decode_steps=6, calls="one", thresholds=ths)
    got = run_gpu(sc)
    orc = run_oracle(sc)
    assert got.demotion_log == orc.demotion_log and len(got.demotion_log) == 2
    assert got.slot_log == orc.slot_log
    assert got.residency == [0, 0]
    ref = run_gpu(dataclasses.replace(sc, thresholds=()))
    for a, b in zip(got.outputs, ref.outputs):
        assert np.array_equal(a, b)


def test_kv_tail_export_and_append_round_trip():
    """Alg. 2's tail move: export, drop, re-append -> the next outputs are bit-identical."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape = synth.TINY
    w = weights_of(shape)
    wl = TINY_RAGGED

    cs = compute_stream().__enter__()

    def make():
        cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=2,
                           compute_stream=cs.handle)
        h = P.stage_init(cfg)
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 1)
        x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 37)).cuda()
        P.stage_prefill(h, [0], 1, 37, x, torch.empty_like(x))
        return h

    nxt = torch.from_numpy(synth.decode_input(wl, 0, 0, 0)[None]).cuda()
    h1 = make()
    want = torch.empty_like(nxt)
    P.stage_decode(h1, [0], 1, nxt, want)
    P.stage_sync(h1)
    table_before = P.stage_get_block_table(h1, 0, 0)
    P.stage_destroy(h1)

    h2 = make()
    try:
        k = np.zeros((2, 21, 2, 64), np.uint16)
        v = np.zeros_like(k)
        P.stage_kv_export_tail(h2, 0, 0, 21, k, v, True)    # 37 -> 16: blocks 1 and 2 freed
        assert P.stage_get_length(h2, 0, 0) == 16
        assert P.stage_get_block_table(h2, 0, 0) == table_before[:1]
        kd = torch.from_numpy(k.view(np.int16)).cuda()
        vd = torch.from_numpy(v.view(np.int16)).cuda()
        P.stage_kv_append(h2, 0, 0, 21, kd, vd)              # device source
        assert P.stage_get_length(h2, 0, 0) == 37
        got = torch.empty_like(nxt)
        P.stage_decode(h2, [0], 1, nxt, got)
        P.stage_sync(h2)
        assert torch.equal(got, want)
        # the exported K/V are the values the oracle stores, up to one bf16 rounding flip
        from oracle.stage_oracle import OracleStage, widen_bf16
        orc = OracleStage(shape, w, kv_dtype="bf16")
        orc.forward([("s", synth.prefill_inputs(wl, 0, 0, 37))])
        ok, ov = orc.export_tail("s", 21, drop=False)
        gk = widen_bf16(k).numpy()
        assert np.abs(gk - ok).max() <= 2 ** -7 * np.abs(ok).max()
        assert np.mean(gk == ok) > 0.99
    finally:
        P.stage_destroy(h2)
        cs.__exit__(None, None, None)


def test_zero_copy_decode_only_stage_needs_no_slots():
    """A decode-only zero-copy stage (context received as a KV tail, Alg. 2) holds no HBM slot and
    no weights in HBM, and decodes bit-identically to an all-resident stage; a multi-token prefill
    then needs a slot and is refused without changing the stage."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape = synth.TINY
    w = weights_of(shape)
    wl = TINY_RAGGED
    cs = compute_stream().__enter__()
    nxt = torch.from_numpy(synth.decode_input(wl, 0, 0, 0)[None]).cuda()
    k = np.zeros((2, 37, 2, 64), np.uint16)
    v = np.zeros_like(k)
    cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=2,
                       compute_stream=cs.handle)
    h = P.stage_init(cfg)
    try:
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 1)
        x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 37)).cuda()
        P.stage_prefill(h, [0], 1, 37, x, torch.empty_like(x))
        P.stage_kv_export_tail(h, 0, 0, 37, k, v, False)
        want = torch.empty_like(nxt)
        P.stage_decode(h, [0], 1, nxt, want)
        P.stage_sync(h)
    finally:
        P.stage_destroy(h)

    cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=0,
                       n_stream_slots=0, compute_stream=cs.handle, zero_copy=True)
    h = P.stage_init(cfg)
    try:
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 0)
        P.stage_kv_append(h, 0, 0, 37, k, v)
        got = torch.empty_like(nxt)
        P.stage_decode(h, [0], 1, nxt, got)
        P.stage_sync(h)
        assert torch.equal(got, want)
        st = P.stage_get_stats(h)
        assert st["hbm_weight_bytes"] == 0 and st["stream_slots"] == 0 and st["layer_loads"] == 0
        assert st["bytes_direct"] == 2 * st["layer_bytes"]
        x4 = torch.zeros(1, 1, 4, 256, device="cuda")
        with pytest.raises(P.StageError) as e:
            P.stage_prefill(h, [0], 1, 4, x4, torch.empty_like(x4))    # would stage: no slots
        assert e.value.code == P.STAGE_EINVAL
        assert P.stage_get_length(h, 0, 0) == 38 and P.stage_get_slot_log(h) == []
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def _parking_run(park: bool, pool_blocks: int, rounds: int = 6, n_park: int = 32):
    """Three micro-batches of two sequences (tiny shape): prefill 37 each, then decode rounds
    one micro-batch per call.  With `park`, each call is followed by parking the micro-batch's
    tails (Alg. 2) and by the prefetch of the next micro-batch's tails; the same steps drive the
    oracle's block allocator."""
    import torch
    import paper_2512_21835_amd as P
    from oracle.policies import BlockAllocator
    shape, wl = synth.TINY, TINY_RAGGED
    w = weights_of(shape)
    cs = compute_stream().__enter__()
    cfg = P.config_for(shape, max_microbatches=3, max_batch=2, max_context=64, n_resident_max=2,
                       kv_pool_blocks=pool_blocks, compute_stream=cs.handle, kv_park_tokens=n_park if park else 0)
    h = P.stage_init(cfg)
    alloc = BlockAllocator(pool_blocks, 16)
    parked = {}

    def model_call(m, n):
        keys = [(m, b) for b in range(2)]
        for k in keys:                       # a parked tail comes back first
            if parked.get(k):
                alloc.call([(k, parked.pop(k))])
        alloc.call([(k, n) for k in keys])

    def model_park(m):
        for b in range(2):
            k = (m, b)
            n = min(n_park, alloc.lengths[k])
            alloc.truncate(k, n)
            parked[k] = n

    def model_unpark(m):
        for b in range(2):
            if parked.get((m, b)):
                alloc.call([((m, b), parked.pop((m, b)))])

    outs = []
    try:
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 1)
        plan = [("prefill", m, -1) for m in range(3)] + [("decode", m, t) for t in range(rounds) for m in range(3)]
        for kind, m, t in plan:
            if kind == "prefill":
                x = np.stack([synth.prefill_inputs(wl, m, b, 37) for b in range(2)])[None]
                xi = torch.from_numpy(x).cuda()
                y = torch.empty_like(xi)
                P.stage_prefill(h, [m], 2, 37, xi, y)
                model_call(m, 37)
            else:
                x = np.stack([synth.decode_input(wl, m, b, t) for b in range(2)])[None]
                xi = torch.from_numpy(x).cuda()
                y = torch.empty_like(xi)
                P.stage_decode(h, [m], 2, xi, y)
                model_call(m, 1)
            outs.append(y)
            if park:
                P.stage_kv_park(h, [m], n_park)
                model_park(m)
                if kind == "decode":
                    P.stage_kv_unpark(h, [(m + 1) % 3])     # prefetch the next micro-batch's tails
                    model_unpark((m + 1) % 3)
        P.stage_sync(h)
        tables = {(m, b): P.stage_get_block_table(h, m, b) for m in range(3) for b in range(2)}
        lengths = {(m, b): P.stage_get_length(h, m, b) for m in range(3) for b in range(2)}
        st = P.stage_get_stats(h)
        return [o.cpu().numpy() for o in outs], tables, lengths, st, alloc, parked
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def test_kv_parking_is_lossless_and_fits_a_smaller_pool():
    """Alg. 2 on one GPU: tails parked in host memory between a micro-batch's calls and fetched
    back ahead of its next call leave every output bit unchanged, let 12 KV blocks serve six
    sequences that need 18 without parking, and take blocks exactly as the oracle's allocator
    does."""
    _gpu()
    import paper_2512_21835_amd as P
    ref, _, ref_len, _, _, _ = _parking_run(False, 18)
    got, tables, lengths, st, alloc, parked = _parking_run(True, 12)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)
    assert lengths == ref_len
    for k, t in tables.items():
        assert t == alloc.table(k), k
    assert st["parked_tokens"] == sum(parked.values()) > 0
    assert st["bytes_parked"] > 0 and st["bytes_unparked"] > 0
    with pytest.raises(P.StageError) as e:
        _parking_run(False, 12)
    assert e.value.code == P.STAGE_ENOMEM


def test_kv_parking_errors_and_automatic_return():
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape, wl = synth.TINY, TINY_RAGGED
    w = weights_of(shape)
    cs = compute_stream().__enter__()
    cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=64, n_resident_max=2,
                       compute_stream=cs.handle, kv_park_tokens=16)
    h = P.stage_init(cfg)
    try:
        for l in range(2):
            P.stage_load_layer(h, l, w(l), 1)
        x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 37)[None, None]).cuda()
        P.stage_prefill(h, [0], 1, 37, x, torch.empty_like(x))
        with pytest.raises(P.StageError) as e:
            P.stage_kv_park(h, [0], 17)                     # beyond kv_park_tokens
        assert e.value.code == P.STAGE_EINVAL
        k_ref = np.zeros((2, 37, 2, 64), np.uint16)
        v_ref = np.zeros_like(k_ref)
        P.stage_kv_export_tail(h, 0, 0, 37, k_ref, v_ref, False)
        P.stage_kv_park(h, [0, 1], 16)                      # micro-batch 1 is empty: skipped
        with pytest.raises(P.StageError) as e:
            P.stage_kv_park(h, [0], 4)                      # already parked
        assert e.value.code == P.STAGE_ESTATE
        assert P.stage_get_length(h, 0, 0) == 37 and len(P.stage_get_block_table(h, 0, 0)) == 2
        k = np.zeros_like(k_ref)
        v = np.zeros_like(v_ref)
        P.stage_kv_export_tail(h, 0, 0, 37, k, v, False)    # brings the tail back first
        assert np.array_equal(k, k_ref) and np.array_equal(v, v_ref)
        assert P.stage_get_stats(h)["parked_tokens"] == 0
    finally:
        P.stage_destroy(h)
    cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=64, n_resident_max=2,
                       compute_stream=cs.handle)
    h = P.stage_init(cfg)
    try:
        with pytest.raises(P.StageError) as e:
            P.stage_kv_park(h, [0], 4)                      # parking off
        assert e.value.code == P.STAGE_ESTATE
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def test_error_paths_leave_stage_usable():
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    shape = synth.TINY
    w = weights_of(shape)
    cs = compute_stream().__enter__()
    cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=20, n_resident_max=1,
                       kv_pool_blocks=2, compute_stream=cs.handle)
    h = P.stage_init(cfg)
    try:
        x = torch.zeros(1, 1, 16, 256, device="cuda")
        y = torch.empty_like(x)
        with pytest.raises(P.StageError) as e:
            P.stage_prefill(h, [0], 1, 16, x, y)          # layers not loaded
        assert e.value.code == P.STAGE_EINVAL
        P.stage_load_layer(h, 0, w(0), 1)
        with pytest.raises(P.StageError) as e:
            P.stage_load_layer(h, 1, w(1), 1)             # budget: 1 resident layer
        assert e.value.code == P.STAGE_ENOMEM
        P.stage_load_layer(h, 1, w(1), 0)
        with pytest.raises(P.StageError) as e:
            P.stage_decode(h, [0], 1, x[:, :, 0], y[:, :, 0])   # empty sequence
        assert e.value.code == P.STAGE_ESTATE
        with pytest.raises(P.StageError) as e:
            P.stage_prefill(h, [0, 0], 1, 16, x, y)       # repeated micro-batch
        assert e.value.code == P.STAGE_EINVAL
        xx = torch.zeros(1, 1, 21, 256, device="cuda")
        with pytest.raises(P.StageError) as e:
            P.stage_prefill(h, [0], 1, 21, xx, torch.empty_like(xx))   # > max_context
        assert e.value.code == P.STAGE_ERANGE
        P.stage_prefill(h, [0], 1, 16, x, y)              # takes 1 of 2 blocks
        x2 = torch.zeros(1, 1, 17, 256, device="cuda")
        with pytest.raises(P.StageError) as e:
            P.stage_prefill(h, [1], 1, 17, x2, torch.empty_like(x2))   # needs 2 blocks, 1 free
        assert e.value.code == P.STAGE_ENOMEM
        assert P.stage_get_length(h, 1, 0) == 0 and P.stage_get_stats(h)["kv_blocks_free"] == 1
        P.stage_decode(h, [0], 1, x[:, :, 0], y[:, :, 0])  # still usable
        P.stage_sync(h)
        assert P.stage_get_length(h, 0, 0) == 17
        assert torch.isfinite(y[:, :, 0]).all()
    finally:
        P.stage_destroy(h)
        cs.__exit__(None, None, None)


def test_llama8b_stage_full_length_bf16_kv():
    """The 8B-shaped stage at its full size, as benchmarked: prefill 1024, then 128 decode steps
    (batch 1), bf16 KV; tolerance 2e-2 plus twice the oracle's own spread under KV rounding."""
    _gpu()
    sc = Scenario(synth.WORKLOADS["llama8b_stage"], prefill=1024, decode_steps=128)
    got = run_gpu(sc)
    ref = run_oracle(sc)
    tol, spread = bf16_kv_tolerance(sc, ref)
    print(f"\n[llama8b bf16-kv] oracle spread under KV rounding {spread:.4g} -> tolerance {tol:.4g}")
    check("llama8b full bf16-kv", sc, got, ref, tol_abs=tol)


def test_llama8b_layers_teacher_forced_bf16_kv():
    """The literal gate with the production bf16 KV cache, layer by layer: each of the 8 layers,
    run alone on the oracle's own inputs for every position (prefill 1024 + 128 decode steps),
    matches the oracle's output of that layer within max|d| <= 2e-2 and cosine >= 0.9995."""
    _gpu()
    sc = Scenario(synth.WORKLOADS["llama8b_stage"], prefill=1024, decode_steps=128)
    ref = run_oracle(sc, trace=True)
    worst = 0.0
    for layer, m in enumerate(teacher_forced(sc, ref)):
        print(f"\n[llama8b teacher-forced layer {layer}] {m}", flush=True)
        assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, (layer, m)
        worst = max(worst, m["max_abs"])
    print(f"[llama8b teacher-forced] worst layer max|d| {worst:.3g}")


def test_llama8b_stage_full_length_fp32_kv():
    """fp32 KV removes the rounding point: the literal gate max|d| <= 2e-2, cosine >= 0.9995."""
    _gpu()
    sc = Scenario(synth.WORKLOADS["llama8b_stage"], prefill=1024, decode_steps=128, kv_fp32=True)
    check("llama8b full fp32-kv", sc, run_gpu(sc), run_oracle(sc))
