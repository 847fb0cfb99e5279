"""GPU parity at the edges of the call sequence: a one-token prefill, prefills that continue a
sequence (chunked prefill, prefill after K/V appended through stage_kv_append), decode at the
largest context the library supports (16384 positions, 256 attention splits), and sequences of
very different lengths decoded in one call."""
import numpy as np
import pytest

import synth
from tests.harness import compare, compute_stream, weights_of

pytestmark = pytest.mark.gpu

TOL_ABS = 2e-2
TOL_COS = 0.9995


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(shape, plan, kv_fp32, seed_tag, max_context):
    """Runs `plan` ([("append", n) | ("prefill", T) | ("decode", 1)]) for one sequence on the GPU
    and on the oracle; returns [(name, compare dict)] for every prefill and decode call."""
    import torch
    import paper_2512_21835_amd as P
    from oracle.stage_oracle import OracleStage

    w = weights_of(shape)
    L, hkv, d, H = shape.n_layers, shape.n_kv_heads, shape.head_dim, shape.hidden
    orc = OracleStage(shape, w, kv_dtype="f32" if kv_fp32 else "bf16")
    results = []
    with compute_stream() as cs:
        cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=max_context,
                           n_resident_max=L, kv_fp32=kv_fp32, compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                P.stage_load_layer(h, l, w(l), 1)
            for i, (kind, n) in enumerate(plan):
                if kind == "append":
                    seed = synth.seed_of(0xE1, seed_tag, i)
                    k = synth.normal_bf16(seed, (L, n, hkv, d))
                    v = synth.normal_bf16(seed + 1, (L, n, hkv, d))
                    if kv_fp32:
                        kd = torch.from_numpy(synth.bf16_to_f32(k)).cuda()
                        vd = torch.from_numpy(synth.bf16_to_f32(v)).cuda()
                    else:
                        kd = torch.from_numpy(k.view(np.int16)).cuda()
                        vd = torch.from_numpy(v.view(np.int16)).cuda()
                    P.stage_kv_append(h, 0, 0, n, kd, vd)
                    orc.append_kv("s", synth.bf16_to_f32(k).astype(np.float64), synth.bf16_to_f32(v).astype(np.float64))
                    continue
                x = synth.normal_f32(synth.seed_of(0xE2, seed_tag, i), (n, H))
                xd = torch.from_numpy(x).cuda().reshape(1, 1, n, H)
                yd = torch.empty_like(xd)
                if kind == "prefill":
                    P.stage_prefill(h, [0], 1, n, xd, yd)
                else:
                    P.stage_decode(h, [0], 1, xd[:, :, 0], yd[:, :, 0])
                P.stage_sync(h)
                got = yd.cpu().numpy().reshape(n, H)
                want = orc.forward([("s", x)])[0]
                results.append((f"{kind} {n} (call {i})", compare(got, want, x, x)))
            assert P.stage_get_length(h, 0, 0) == orc.length("s")
        finally:
            P.stage_destroy(h)
    return results


def _check(tag, results):
    for name, m in results:
        print(f"\n[{tag} {name}] {m}", flush=True)
        assert m["max_abs"] <= TOL_ABS and m["cos"] >= TOL_COS and m["cos_delta"] >= TOL_COS, (name, m)


@pytest.mark.parametrize("kv_fp32", [False, True])
def test_one_token_prefill_then_chunked_prefill_then_decode(kv_fp32):
    """Tiny stage: prefill of 1 token, then 5, then 40 (crossing 16-token blocks, 32-key tiles and a
    128-row query block), then decode."""
    _gpu()
    plan = [("prefill", 1), ("prefill", 5), ("prefill", 40), ("decode", 1), ("decode", 1)]
    _check(f"tiny chunked kv_fp32={kv_fp32}", _run(synth.TINY, plan, kv_fp32, 1, 64))


def test_llama8b_prefill_continuing_a_long_appended_context():
    """8B-shaped stage: 3000 positions of K/V appended, then a 200-token prefill on top of them
    (matrix-core attention over a long history, ragged last query block), then decode."""
    _gpu()
    plan = [("append", 3000), ("prefill", 200), ("decode", 1)]
    _check("llama8b append+prefill", _run(synth.LLAMA8B_STAGE, plan, False, 2, 3300))


@pytest.mark.parametrize("kv_fp32", [False, True])
def test_decode_at_the_largest_context(kv_fp32):
    """Tiny stage: 16383 positions appended, one decode step brings the context to 16384, the
    largest supported (256 attention splits of 64 keys)."""
    _gpu()
    plan = [("append", 16383), ("decode", 1)]
    _check(f"tiny max-context kv_fp32={kv_fp32}", _run(synth.TINY, plan, kv_fp32, 3, 16384))


@pytest.mark.parametrize("kv_fp32,hist", [(False, (37, 200, 1100)), (True, (37, 200, 1100)),
                                          (False, (2047, 4095, 4161))])
def test_llama8b_ragged_contexts_in_one_decode_call(kv_fp32, hist):
    """8B-shaped stage: three sequences with `hist` positions appended, decoded together for two
    steps (3 rows per call: the matrix-core GEMVs; with the bf16 cache the matrix-core attention).
    (37, 200, 1100): the rows span 1, 4 and 18 attention splits, so workgroups of the shorter rows
    exit early and every row's last split is ragged.  (2047, 4095, 4161): with 32, 64 and 66
    splits (33, 65 and 66 on the second step) a row's last split falls well inside, exactly at the
    end of and just past the merge's first round of loads (8 splits on each of 8 lanes, 64 in all),
    and 33 splits leave lanes 1-7 one split short of lane 0.  Each row is checked against the
    oracle."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P
    from oracle.stage_oracle import OracleStage

    shape = synth.LLAMA8B_STAGE
    w = weights_of(shape)
    L, hkv, d, H = shape.n_layers, shape.n_kv_heads, shape.head_dim, shape.hidden
    orc = OracleStage(shape, w, kv_dtype="f32" if kv_fp32 else "bf16")
    with compute_stream() as cs:
        cfg = P.config_for(shape, max_microbatches=3, max_batch=1, max_context=max(hist) + 64, n_resident_max=L,
                           kv_fp32=kv_fp32, compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                P.stage_load_layer(h, l, w(l), 1)
            for m, n in enumerate(hist):
                seed = synth.seed_of(0xE3, m, n)
                k = synth.normal_bf16(seed, (L, n, hkv, d))
                v = synth.normal_bf16(seed + 1, (L, n, hkv, d))
                if kv_fp32:
                    kd = torch.from_numpy(synth.bf16_to_f32(k)).cuda()
                    vd = torch.from_numpy(synth.bf16_to_f32(v)).cuda()
                else:
                    kd = torch.from_numpy(k.view(np.int16)).cuda()
                    vd = torch.from_numpy(v.view(np.int16)).cuda()
                P.stage_kv_append(h, m, 0, n, kd, vd)
                orc.append_kv(f"s{m}", synth.bf16_to_f32(k).astype(np.float64), synth.bf16_to_f32(v).astype(np.float64))
            for step in range(2):
                x = synth.normal_f32(synth.seed_of(0xE4, step, 3), (3, H))
                xd = torch.from_numpy(x).cuda().reshape(3, 1, H)
                yd = torch.empty_like(xd)
                P.stage_decode(h, [0, 1, 2], 1, xd, yd)
                P.stage_sync(h)
                got = yd.cpu().numpy().reshape(3, H)
                want = orc.forward([(f"s{m}", x[m:m + 1]) for m in range(3)])
                for m in range(3):
                    cmp = compare(got[m:m + 1], want[m], x[m:m + 1], x[m:m + 1])
                    print(f"\n[ragged kv_fp32={kv_fp32} step {step} row {m} ctx {hist[m] + step + 1}] {cmp}", flush=True)
                    assert cmp["max_abs"] <= TOL_ABS and cmp["cos"] >= TOL_COS and cmp["cos_delta"] >= TOL_COS, (m, cmp)
            for m, n in enumerate(hist):
                assert P.stage_get_length(h, m, 0) == n + 2 == orc.length(f"s{m}")
        finally:
            P.stage_destroy(h)


@pytest.mark.parametrize("shape_name,kv_fp32", [("tiny", False), ("tiny", True), ("llama8b", False),
                                                ("llama8b", True)])
def test_single_split_rows_give_the_merged_bits(shape_name, kv_fp32):
    """Decode attention writes a row's output straight from its one split (o / l, no merge launch)
    when every row of the call fits one 64-key split, and merges the splits otherwise; for a row
    that fits one split the two give the same bits (the merge of a single split weighs it by
    exp(m - m) = 1).  Row 0 (contexts 31 and 32) is decoded alone, then together with row 1
    (contexts 301 and 302: 5 splits), both on the vector GEMV engine (1 and 2 rows).  tiny: 64-wide
    heads (vector attention kernel); llama8b: 128-wide heads (the matrix-core kernel with a bf16
    cache, the vector one with fp32)."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P

    shape = synth.TINY if shape_name == "tiny" else synth.LLAMA8B_STAGE
    w = weights_of(shape)
    L, hkv, d, H = shape.n_layers, shape.n_kv_heads, shape.head_dim, shape.hidden
    hist = (30, 300)
    kv = []
    for m, n in enumerate(hist):
        seed = synth.seed_of(0xE7, m, n)
        kv.append((synth.normal_bf16(seed, (L, n, hkv, d)), synth.normal_bf16(seed + 1, (L, n, hkv, d))))
    xs = [synth.normal_f32(synth.seed_of(0xE8, step, 2), (2, H)) for step in range(2)]

    def run(rows):
        outs = []
        with compute_stream() as cs:
            cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=400, n_resident_max=L,
                               kv_fp32=kv_fp32, compute_stream=cs.handle)
            h = P.stage_init(cfg)
            try:
                for l in range(L):
                    P.stage_load_layer(h, l, w(l), 1)
                for m, (k, v) in enumerate(kv):
                    if kv_fp32:
                        kd = torch.from_numpy(synth.bf16_to_f32(k)).cuda()
                        vd = torch.from_numpy(synth.bf16_to_f32(v)).cuda()
                    else:
                        kd = torch.from_numpy(k.view(np.int16)).cuda()
                        vd = torch.from_numpy(v.view(np.int16)).cuda()
                    P.stage_kv_append(h, m, 0, hist[m], kd, vd)
                for x in xs:
                    xd = torch.from_numpy(np.ascontiguousarray(x[:rows])).cuda().reshape(rows, 1, H)
                    yd = torch.empty_like(xd)
                    P.stage_decode(h, list(range(rows)), 1, xd, yd)
                    P.stage_sync(h)
                    outs.append(yd.cpu().numpy().reshape(rows, H))
            finally:
                P.stage_destroy(h)
        return outs

    alone, mixed = run(1), run(2)
    for step in range(2):
        assert np.isfinite(alone[step]).all()
        assert np.array_equal(alone[step][0], mixed[step][0]), f"step {step}"


# One narrow layer whose prefill gate/up GEMM (M = 2000 rows, 2F = 8000 gate/up rows: ragged in both
# dimensions) still fills the GPU with 256 x 256 tiles, over K = 64 or 96: the software-pipelined k
# loop with two tiles (only its peeled tail) and with three (one pass of the loop body).
NARROW_H64 = synth.StageShape("narrow-1L-h64", 3, 1, 64, 1, 1, 64, 4000)
NARROW_H96 = synth.StageShape("narrow-1L-h96", 4, 1, 96, 1, 1, 64, 4000)


@pytest.mark.parametrize("shape", [NARROW_H64, NARROW_H96], ids=["k64", "k96"])
def test_prefill_gemm_shortest_pipelined_k_loops(shape):
    _gpu()
    plan = [("prefill", 2000), ("decode", 1)]
    _check(f"{shape.name} prefill 2000", _run(shape, plan, False, 5, 2048))


# Every attention instance the library builds (query heads per KV head G in 1, 2, 4, 8; head
# width 64 or 128; bf16 or fp32 cache): one small layer, prefill 70 (three 32-key tiles, ragged;
# a 128-row query block of 128 / G positions) then two decode steps at contexts 71 and 72 (two
# 64-key splits and their merge), against the oracle.
_GD = [(g, d, f32) for f32 in (False, True) for d in (64, 128) for g in (1, 2, 4, 8)]


@pytest.mark.parametrize("g,d,kv_fp32", _GD, ids=[f"G{g}-d{d}-{'f32' if f else 'bf16'}" for g, d, f in _GD])
def test_every_attention_group_and_head_width(g, d, kv_fp32):
    _gpu()
    shape = synth.StageShape(f"gqa-g{g}-d{d}", 10 + 10 * g + d // 64, 1, 256, 2 * g, 2, d, 512)
    plan = [("prefill", 70), ("decode", 1), ("decode", 1)]
    _check(f"{shape.name} kv_fp32={kv_fp32}", _run(shape, plan, kv_fp32, 6, 80))


# Decode calls of 1 to 40 rows on one small layer whose projections can run on either engine
# (K a multiple of 128): the vector kernel's 1-, 2-, 4- and 8-row instances, the matrix-core
# engine from 3 rows (5 for the O projection), its unsplit launches and the down projection's K
# cut into two ranges, and calls of more
# than 16 rows cut into several launches (17: 16 + 1; 40: 16 + 16 + 8); every row against the
# oracle.
ROWS_SHAPE = synth.StageShape("rows-1L-h256", 5, 1, 256, 4, 2, 64, 1024)


@pytest.mark.parametrize("rows", [1, 2, 3, 4, 5, 7, 8, 9, 16, 17, 40])
def test_decode_rows_on_both_engines(rows):
    _gpu()
    _decode_rows(ROWS_SHAPE, rows)


# Matrix-core launch forms: an odd number of 128-wide k chunks (the engine takes them in pairs):
# hidden 384 and ffn 1152 leave the QKV, O and gate/up projections unsplit over 3 chunks and cut
# the down projection into ranges of 6 and 3 chunks; hidden 1152 cuts the QKV (RoPE epilogue) and
# gate/up projections, normalised over ranges, into 6 and 3 chunks.  Units per wavefront: small
# unsplit launches take 14, and ffn 16384 (256 workgroups of 64 gate/up units) keeps 16.
ODD_CHUNKS = [synth.StageShape("chunks-1L-h384", 9, 1, 384, 6, 6, 64, 1152),
              synth.StageShape("chunks-1L-h1152", 10, 1, 1152, 2, 2, 64, 256),
              synth.StageShape("wide-ffn-1L-h128", 11, 1, 128, 2, 2, 64, 16384)]


@pytest.mark.parametrize("rows", [3, 5, 16])
@pytest.mark.parametrize("shape", ODD_CHUNKS, ids=["h384", "h1152", "f16384"])
def test_matrix_core_odd_chunk_counts(shape, rows):
    _gpu()
    _decode_rows(shape, rows)


# A stage whose widths are off the 32 grid (hidden 200, ffn 440, four heads of 64): in prefill the
# QKV, gate/up and down GEMMs take the register-staged kernel (K % 32 != 0), gate/up stores both
# halves and a separate pass applies SwiGLU and writes the pair, and the O GEMM (K = 256) runs on
# the LDS-copy kernel with a ragged last column tile; in decode the vector GEMVs take K = 200 and
# 440 (not whole 512-wide steps), and at 6 rows the O projection runs on the matrix cores with a
# ragged last 64-unit block.
ODD_SHAPE = synth.StageShape("odd-2L-h200", 7, 2, 200, 4, 2, 64, 440)


@pytest.mark.parametrize("kv_fp32", [False, True])
def test_widths_off_the_32_grid(kv_fp32):
    _gpu()
    plan = [("prefill", 70), ("decode", 1), ("decode", 1)]
    _check(f"{ODD_SHAPE.name} kv_fp32={kv_fp32}", _run(ODD_SHAPE, plan, kv_fp32, 8, 80))


@pytest.mark.parametrize("rows", [2, 6])
def test_widths_off_the_32_grid_several_rows(rows):
    _gpu()
    _decode_rows(ODD_SHAPE, rows)


def _decode_rows(shape, rows):
    """Prefills `rows` sequences of ragged lengths one by one, then decodes all of them in one
    call; every row against the oracle."""
    import torch
    import paper_2512_21835_amd as P
    from oracle.stage_oracle import OracleStage

    w = weights_of(shape)
    L, H = shape.n_layers, shape.hidden
    orc = OracleStage(shape, w, kv_dtype="bf16")
    with compute_stream() as cs:
        cfg = P.config_for(shape, max_microbatches=40, max_batch=1, max_context=64, n_resident_max=L,
                           compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                P.stage_load_layer(h, l, w(l), 1)
            for m in range(rows):
                n = 20 + m % 23   # ragged histories
                x = synth.normal_f32(synth.seed_of(0xE9, m, n), (n, H))
                xd = torch.from_numpy(x).cuda().reshape(1, 1, n, H)
                P.stage_prefill(h, [m], 1, n, xd, torch.empty_like(xd))
                orc.forward([(f"s{m}", x)])
            x = synth.normal_f32(synth.seed_of(0xEA, rows, 1), (rows, H))
            xd = torch.from_numpy(x).cuda().reshape(rows, 1, H)
            yd = torch.empty_like(xd)
            P.stage_decode(h, list(range(rows)), 1, xd, yd)
            P.stage_sync(h)
            got = yd.cpu().numpy().reshape(rows, H)
        finally:
            P.stage_destroy(h)
    want = orc.forward([(f"s{m}", x[m:m + 1]) for m in range(rows)])
    for m in range(rows):
        cmp = compare(got[m:m + 1], want[m], x[m:m + 1], x[m:m + 1])
        assert cmp["max_abs"] <= TOL_ABS and cmp["cos"] >= TOL_COS and cmp["cos_delta"] >= TOL_COS, (rows, m, cmp)
