"""GPU parity of the 70B-shaped 16-layer stage (hidden 8192, 64 query / 8 KV heads, head_dim 128,
SwiGLU 28672) at full width, for the three 70B-shaped workloads: all layers resident with four
interleaved micro-batches; 4 resident layers with 12 streamed through 2 HBM slots; and eight
micro-batches of batch 2 under KV pressure with the residency shrinking 16 -> 8.

Token counts are reduced where the float64 oracle has to follow every token (prefill 32-64,
a few decode rounds; thresholds compressed to one demotion per round); full contexts (2048 and
8192) are reached by appending seeded K/V through stage_kv_append, after which one decode round
is checked against the oracle holding the same cache.  Offloading must change no bit.
"""
import dataclasses

import numpy as np
import pytest

import synth
from tests.harness import (Scenario, teacher_forced, _progress, bf16_kv_tolerance, compare, compute_stream, row_origin,
                           run_gpu, run_oracle, weights_of)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL_ABS = 2e-2
TOL_COS = 0.9995
SHAPE = synth.LLAMA70B_STAGE
C3 = synth.WORKLOADS["llama70b_resident"]
C5 = synth.WORKLOADS["llama70b_kvpressure"]


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _report(name, m):
    print(f"\n[{name}] {m}", flush=True)


# Oracle runs shared between tests of this module (the float64 oracle at 70B width dominates their time).
_ORACLE = {}


def _oracle(key, sc, **kw):
    if key not in _ORACLE:
        _ORACLE[key] = run_oracle(sc, **kw)
    return _ORACLE[key]


# The bf16-KV end-to-end errors last measured (four micro-batches in one call, prefill 64 + 8 rounds):
# a regression ceiling of 1.5x beside the derived bound, which sits near 2.0 at this size.
RECORDED_BF16_MAX_ABS = {"c3_all": 0.579}

C3_FP32 = Scenario(C3, prefill=64, decode_steps=8, calls="one", kv_fp32=True)


def _where(sc, m):
    call, kind, mb, b, pos = row_origin(sc, m["worst_row"])
    return f"call {call} ({kind}) mb {mb} b {b} position {pos} column {m['worst_col']} (oracle {m['worst_ref']:.4g})"


def test_70b_c3_fp32_kv_literal_and_c4_streamed_bit_identical():
    """The literal gate (fp32 KV cache; max|d| <= 2e-2, cosine >= 0.9995 on the output and on the
    stage contribution) at the protocol length: four interleaved micro-batches, prefill 64 each,
    then 8 decode rounds round robin (one micro-batch per call).  Then the offloaded configuration
    (4 resident + 12 layers streamed through 2 slots) on the same calls gives the same bits, and
    its slot log follows the oracle's policy."""
    _gpu()
    ref = _oracle("c3_fp32", C3_FP32, trace=True)
    got3 = run_gpu(C3_FP32)
    m = compare(got3.flat_out(), ref.flat_out(), got3.flat_in(), ref.flat_in())
    _report(f"70b C3 fp32-kv literal, worst at {_where(C3_FP32, m)}", m)
    assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m
    assert got3.block_tables == ref.block_tables

    sc4 = dataclasses.replace(C3_FP32, n_resident=4, slots=2)
    got4 = run_gpu(sc4)
    pol = run_oracle(sc4, floats=False)
    assert got4.slot_log == pol.slot_log and len(got4.slot_log) == 12 * (4 + 4 * 8)
    assert got4.residency == [1] * 4 + [0] * 12
    assert len(got4.outputs) == len(got3.outputs)
    for c, (o4, o3) in enumerate(zip(got4.outputs, got3.outputs)):
        assert np.array_equal(o4, o3), f"call {c} differs"


def test_70b_resident_bf16_kv_and_offloaded_is_bit_identical():
    """bf16 KV, the four micro-batches in one call (4 rows: the matrix-core decode engine, the O
    projection on the vector kernel): oracle parity (cosine gates; max|d| within the bound derived
    from the oracle's own spread under K/V rounding, and within 1.5x the last measured error), then
    the same workload with 12 of 16 layers streamed through two slots gives the same bits."""
    _gpu()
    sc3 = Scenario(C3, prefill=64, decode_steps=8, calls="all")
    got3 = run_gpu(sc3)
    ref = _oracle("c3_bf16_all", sc3)
    m = compare(got3.flat_out(), ref.flat_out(), got3.flat_in(), ref.flat_in())
    tol, spread = bf16_kv_tolerance(sc3, ref)
    ceiling = 1.5 * RECORDED_BF16_MAX_ABS["c3_all"]
    _report(f"70b bf16-kv resident (oracle spread {spread:.4g}, tolerance {tol:.4g}, ceiling {ceiling:.4g})", m)
    assert m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m
    assert m["max_abs"] <= tol and m["max_abs"] <= ceiling, m
    assert got3.block_tables == ref.block_tables

    sc4 = dataclasses.replace(sc3, calls="all", n_resident=4, slots=2)
    got4 = run_gpu(sc4)
    pol = run_oracle(sc4, floats=False)
    assert got4.slot_log == pol.slot_log and len(got4.slot_log) == 12 * (1 + 8)
    assert got4.residency == [1] * 4 + [0] * 12
    assert len(got4.outputs) == len(got3.outputs)
    for c, (o4, o3) in enumerate(zip(got4.outputs, got3.outputs)):
        assert np.array_equal(o4, o3), f"call {c} differs"


def test_70b_layers_teacher_forced_fp32_and_bf16_kv():
    """The literal gate layer by layer (four interleaved micro-batches, prefill 64, 8 decode rounds
    round robin): each of the 16 layers, run alone on the GPU on the oracle's own inputs for every
    position, is within max|d| <= 2e-2, cosine >= 0.9995 of the oracle's output of that layer --
    with the fp32 KV cache (the arithmetic alone: both sides build the layer's K/V from the same
    inputs and store them exactly) and with the production bf16 cache (where a K/V element whose
    fp32 and float64 values straddle a rounding boundary stores neighbouring bf16 values).  Each
    layer's worst element is reported with its call, sequence, position and column."""
    _gpu()
    ref32 = _oracle("c3_fp32", C3_FP32, trace=True)
    fp32 = teacher_forced(C3_FP32, ref32)
    sc = dataclasses.replace(C3_FP32, kv_fp32=False)
    ref16 = _oracle("c3_bf16_one", sc, trace=True)
    bf16 = teacher_forced(sc, ref16)
    for layer, (m32, m16) in enumerate(zip(fp32, bf16)):
        _report(f"70b teacher-forced layer {layer} fp32-kv, worst at {_where(C3_FP32, m32)}", m32)
        _report(f"70b teacher-forced layer {layer} bf16-kv, worst at {_where(sc, m16)}", m16)
    for layer, m in enumerate(fp32 + bf16):
        assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, (layer % 16, m)


def test_70b_kv_pressure_fp32_kv_literal_demotions_and_bf16_bit_identical():
    """Eight micro-batches of batch 2 (all in one call: 16 rows, matrix-core engine), prefill 32
    each, thresholds compressed to one per decode round so that layers 15, 14, ..., 8 are demoted in
    turn: with the fp32 KV cache the output meets the literal gate against the oracle, and the
    demotion log, slot log and block tables follow the oracle's policies; with the bf16 cache the
    demoting run gives the all-resident run's bits."""
    _gpu()
    ths = tuple(32 + j for j in range(1, 9))
    sc = Scenario(C5, prefill=32, decode_steps=8, calls="all", thresholds=ths, kv_fp32=True)
    got = run_gpu(sc)
    ref = run_oracle(sc)
    assert got.demotion_log == ref.demotion_log
    assert [l for _, l in got.demotion_log] == list(range(15, 7, -1))
    assert got.residency == [1] * 8 + [0] * 8
    assert got.slot_log == ref.slot_log
    assert got.block_tables == ref.block_tables
    m = compare(got.flat_out(), ref.flat_out(), got.flat_in(), ref.flat_in())
    _report(f"70b kv-pressure fp32-kv literal, worst at {_where(sc, m)}", m)
    assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m
    sc16 = dataclasses.replace(sc, kv_fp32=False)
    demoting = run_gpu(sc16)
    resident = run_gpu(dataclasses.replace(sc16, thresholds=()))
    assert demoting.demotion_log == got.demotion_log
    for a, b in zip(demoting.outputs, resident.outputs):
        assert np.array_equal(a, b)


def _full_context_round(n_mb, B, ctx, n_resident, kv_fp32, seed_tag, sampled):
    """Append ctx-1 K/V positions to every sequence, then one decode round on the GPU.

    Sequences in `sampled` get K/V and inputs from the seeded generator (the oracle recomputes
    them); the others get device-generated random K/V that only the GPU sees.
    """
    import torch
    import paper_2512_21835_amd as P
    w = weights_of(SHAPE)
    L, hkv, d, H = SHAPE.n_layers, SHAPE.n_kv_heads, SHAPE.head_dim, SHAPE.hidden
    kvs, xs = {}, {}
    with compute_stream() as cs:
        cfg = P.config_for(SHAPE, max_microbatches=n_mb, max_batch=B, max_context=ctx, n_resident_max=n_resident,
                           kv_fp32=kv_fp32, compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                P.stage_load_layer(h, l, w(l), 1 if l < n_resident else 0)
            gen = torch.Generator(device="cuda").manual_seed(seed_tag)
            for m in range(n_mb):
                for b in range(B):
                    if (m, b) in sampled:
                        seed = synth.seed_of(0xC0, seed_tag, m, b)
                        k = synth.normal_bf16(seed, (L, ctx - 1, hkv, d))
                        v = synth.normal_bf16(seed + 1, (L, ctx - 1, hkv, d))
                        kvs[(m, b)] = (k, v)
                        if kv_fp32:
                            kd = torch.from_numpy(synth.bf16_to_f32(k)).cuda()
                            vd = torch.from_numpy(synth.bf16_to_f32(v)).cuda()
                        else:
                            kd = torch.from_numpy(k.view(np.int16)).cuda()
                            vd = torch.from_numpy(v.view(np.int16)).cuda()
                    else:
                        dt = torch.float32 if kv_fp32 else torch.bfloat16
                        kd = torch.randn(L, ctx - 1, hkv, d, generator=gen, device="cuda").to(dt)
                        vd = torch.randn(L, ctx - 1, hkv, d, generator=gen, device="cuda").to(dt)
                        if not kv_fp32:
                            kd, vd = kd.view(torch.int16), vd.view(torch.int16)
                    P.stage_kv_append(h, m, b, ctx - 1, kd, vd)
                    xs[(m, b)] = synth.normal_f32(synth.seed_of(0xC1, seed_tag, m, b), (H,))
            x = np.stack([np.stack([xs[(m, b)] for b in range(B)]) for m in range(n_mb)])
            x_in = torch.from_numpy(x).cuda()
            x_out = torch.empty_like(x_in)
            P.stage_decode(h, list(range(n_mb)), B, x_in, x_out)
            P.stage_sync(h)
            out = x_out.cpu().numpy()
            tables = {(m, b): P.stage_get_block_table(h, m, b) for m in range(n_mb) for b in range(B)}
        finally:
            P.stage_destroy(h)
    return out, x, kvs, xs, tables


def _oracle_full_context(kvs, xs, kv_fp32):
    """Oracle outputs of the sampled sequences: {key: [H]}."""
    from oracle.stage_oracle import OracleStage
    orc = OracleStage(SHAPE, _progress(weights_of(SHAPE), "oracle"), kv_dtype="f32" if kv_fp32 else "bf16")
    keys = sorted(kvs)
    for key in keys:
        k, v = kvs[key]
        orc.append_kv(key, synth.bf16_to_f32(k).astype(np.float64), synth.bf16_to_f32(v).astype(np.float64))
    outs = orc.forward([(key, xs[key][None]) for key in keys])
    return {key: o[0] for key, o in zip(keys, outs)}


def _check_sampled(name, out, xs, ref):
    keys = sorted(ref)
    got = np.stack([out[m, b] for m, b in keys])
    want = np.stack([ref[k] for k in keys])
    x = np.stack([xs[k] for k in keys])
    m = compare(got, want, x, x)
    _report(name, m)
    assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m


@pytest.mark.parametrize("kv_fp32", [True, False])
def test_70b_decode_at_context_8192_batch2(kv_fp32):
    """Eight micro-batches of batch 2 at context 8192 (paged, 512 blocks each): one decode round."""
    _gpu()
    sampled = {(0, 0), (5, 1)}
    out, x, kvs, xs, tables = _full_context_round(8, 2, 8192, 16, kv_fp32, 5, sampled)
    _check_sampled(f"70b ctx8192 B=2 kv_fp32={kv_fp32}", out, xs, _oracle_full_context(kvs, xs, kv_fp32))
    # block ids: each sequence took 512 blocks in call order (mb, then b), lowest first
    for i, key in enumerate(sorted(tables)):
        assert tables[key] == list(range(512 * i, 512 * (i + 1)))


def test_70b_offloaded_decode_at_context_2048_equals_resident():
    """Four micro-batches at context 2048: 4 resident + 12 streamed layers give the resident bits."""
    _gpu()
    sampled = {(0, 0), (3, 0)}
    res = _full_context_round(4, 1, 2048, 16, False, 7, sampled)
    off = _full_context_round(4, 1, 2048, 4, False, 7, sampled)
    assert np.array_equal(res[0], off[0])
    _check_sampled("70b ctx2048 offloaded", off[0], off[3], _oracle_full_context(off[2], off[3], False))


def _prefill_one_layer(bits, x, kv_fp32):
    """One 70B-shaped layer's prefill of x [T, H] (one sequence) on the GPU: (outputs [T, H], stored
    K, V [T, Hkv, d] as fp32 values)."""
    import torch
    import paper_2512_21835_amd as P
    one = dataclasses.replace(SHAPE, n_layers=1)
    T, H, hkv, d = x.shape[0], SHAPE.hidden, SHAPE.n_kv_heads, SHAPE.head_dim
    with compute_stream() as cs:
        cfg = P.config_for(one, max_microbatches=1, max_batch=1, max_context=T, n_resident_max=1,
                           kv_fp32=kv_fp32, compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            P.stage_load_layer(h, 0, bits, 1)
            x_in = torch.from_numpy(x).cuda().reshape(1, 1, T, H)
            x_out = torch.empty_like(x_in)
            P.stage_prefill(h, [0], 1, T, x_in, x_out)
            dt = torch.float32 if kv_fp32 else torch.int16
            k_dev = torch.empty(1, T, hkv, d, dtype=dt, device="cuda")
            v_dev = torch.empty_like(k_dev)
            P.stage_kv_export_tail(h, 0, 0, T, k_dev, v_dev, False)
            P.stage_sync(h)
            got = x_out.cpu().numpy().reshape(T, H)
            if kv_fp32:
                k, v = k_dev.cpu().numpy()[0], v_dev.cpu().numpy()[0]
            else:
                k = synth.bf16_to_f32(k_dev.cpu().numpy().view(np.uint16)[0])
                v = synth.bf16_to_f32(v_dev.cpu().numpy().view(np.uint16)[0])
        finally:
            P.stage_destroy(h)
    return got, k.astype(np.float64), v.astype(np.float64)


def test_70b_prefill_2048_one_layer():
    """Full-size prefill of one 70B-shaped layer (T = 2048 tokens of one sequence, 256 x 256 GEMM
    tiles, matrix-core prefill attention with 8 query heads per KV head).  With the fp32 cache,
    sampled output rows -- at the 16-token block, 16-row query block and 32-key tile edges and at
    the ends -- meet the literal gate against the oracle's own computation of the layer (its own
    K/V, nothing from the GPU).  With the production bf16 cache, at least 99% of the stored K/V
    elements equal the oracle's bf16 K/V bit for bit, and every one is within a bf16 step of it or
    within 2^-8 of the tensor's rms (a value that comes out of cancellation carries the fp32
    rounding of its larger terms); the same sampled rows, against the oracle over its own bf16
    K/V, are reported (cosine gates)."""
    _gpu()
    import torch
    from oracle import stage_oracle as O

    one = dataclasses.replace(SHAPE, n_layers=1)
    T = 2048
    bits = weights_of(SHAPE)(0)
    x = synth.normal_f32(synth.seed_of(0xC7, 2048), (T, SHAPE.hidden))
    rows = [0, 1, 15, 16, 17, 31, 32, 127, 128, 1000, 1023, 1024, 1535, 2032, 2046, 2047]
    w = O.LayerWeights(bits)
    x64 = torch.as_tensor(x, dtype=torch.float64)

    got32, _, _ = _prefill_one_layer(bits, x, True)
    k32, v32 = O.layer_kv(x64, w, one, O.round_to_f32)
    want32 = O.decoder_layer_rows(x64, w, one, rows, k32, v32).numpy()
    m = compare(got32[rows], want32, x[rows], x[rows])
    _report("70b prefill 2048 one layer fp32-kv, sampled rows against the oracle's own K/V", m)
    assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m

    got16, k_gpu, v_gpu = _prefill_one_layer(bits, x, False)
    k16, v16 = O.layer_kv(x64, w, one, O.round_to_bf16)
    for name, g, o in (("K", k_gpu, k16), ("V", v_gpu, v16)):
        o = o.numpy()
        rms = float(np.sqrt(np.mean(o * o)))
        bound = np.abs(o) * 2.0 ** -7 + rms * 2.0 ** -8      # one bf16 step at |o|, plus cancellation
        diff = np.abs(g - o)
        equal = float(np.mean(diff == 0))
        worst = int(np.argmax(diff / bound))
        print(f"\n[70b prefill 2048 stored {name}] bit-equal {equal:.6f}, rms {rms:.4g}, max |d| {float(diff.max()):.3g}, "
              f"worst |d| / bound {float(diff.flat[worst] / bound.flat[worst]):.3g} at |o| {abs(float(o.flat[worst])):.3g}",
              flush=True)
        assert np.all(diff <= bound), name
        assert equal >= 0.99, (name, equal)
    want16 = O.decoder_layer_rows(x64, w, one, rows, k16, v16).numpy()
    m = compare(got16[rows], want16, x[rows], x[rows])
    _report("70b prefill 2048 one layer bf16-kv, sampled rows against the oracle's own bf16 K/V", m)
    assert m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, m


def test_70b_prefill_is_deterministic_and_independent_of_the_weight_source():
    """The same one-layer 70B-shaped prefill, on fresh stages, gives the same output and K/V bits
    whether the layer's weights are loaded from host memory or from device memory, at T = 256
    (128 x 128 GEMM tiles) and T = 2048 (256 x 256 tiles), three times each.  Regression test of a
    race: stage_load_layer copied device sources with hipMemcpy on the null stream, which returns
    before a device-to-device copy completes and which a non-blocking compute stream does not wait
    for, so the first GEMMs could read a half-copied layer."""
    _gpu()
    import torch
    bits = weights_of(SHAPE)(0)
    dev_bits = {k: torch.from_numpy(v.view(np.int16)).cuda() for k, v in bits.items()}
    torch.cuda.synchronize()
    for T in (256, 2048):
        x = synth.normal_f32(synth.seed_of(0xC8, T), (T, SHAPE.hidden))
        runs = [_prefill_one_layer(bits, x, False)] + [_prefill_one_layer(dev_bits, x, False) for _ in range(3)]
        for r in runs[1:]:
            for a, b, name in zip(runs[0], r, ("output", "K", "V")):
                assert np.array_equal(a, b), (T, name)
        assert np.isfinite(runs[0][0]).all()
