"""Pins of the float64 oracle against facts that do not come from the oracle itself.

Each test would fail on a plausible slip in the oracle: a dropped term, a wrong
sign or index, a transposed operand, a missing mask.  Nothing here touches the
HIP path.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import stage_oracle as O
from synth import StageShape

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F64 = torch.float64


def rand(*shape, seed=0):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=F64)


# ----------------------------------------------------------------- RMSNorm
def test_rmsnorm_closed_form_rms():
    x = rand(5, 64, seed=1) * 3.0
    eps = 1e-5
    y = O.rms_norm(x, torch.ones(64, dtype=F64), eps)
    ms = (x * x).mean(dim=1)
    # rms(x / sqrt(ms + eps)) = sqrt(ms / (ms + eps))
    assert torch.allclose(y.pow(2).mean(dim=1).sqrt(), torch.sqrt(ms / (ms + eps)), rtol=1e-14, atol=0)
    y0 = O.rms_norm(x, torch.ones(64, dtype=F64), 0.0)
    assert torch.allclose(y0.pow(2).mean(dim=1), torch.ones(5, dtype=F64), rtol=1e-14, atol=0)


def test_rmsnorm_gain_is_per_column_and_scale_free():
    x = rand(3, 16, seed=2)
    g = rand(16, seed=3)
    y = O.rms_norm(x, g, 0.0)
    assert torch.allclose(y / g, O.rms_norm(x, torch.ones(16, dtype=F64), 0.0), rtol=1e-13)
    assert torch.allclose(O.rms_norm(7.5 * x, g, 0.0), y, rtol=1e-13)


# ----------------------------------------------------------------- RoPE
def test_rope_unit_vectors_closed_form():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "rope_unit_vectors.txt")) if l.strip() and l[0] != "#"]
    for r in rows:
        i = int(r[0])
        expect = torch.tensor([float(v) for v in r[1:]], dtype=F64)
        e = torch.zeros(1, 1, 4, dtype=F64)
        e[0, 0, i] = 1.0
        got = O.rope(e, torch.tensor([3]), 10000.0)[0, 0]
        assert torch.allclose(got, expect, atol=1e-15, rtol=0), (i, got, expect)


def test_rope_position_zero_is_identity_and_norms_are_kept():
    x = rand(6, 3, 128, seed=4)
    assert torch.equal(O.rope(x[:1], torch.tensor([0]), 10000.0), x[:1])
    pos = torch.tensor([1, 17, 100, 1023, 4000, 8191])
    y = O.rope(x, pos, 10000.0)
    pn_x = x[..., :64] ** 2 + x[..., 64:] ** 2
    pn_y = y[..., :64] ** 2 + y[..., 64:] ** 2
    assert torch.allclose(pn_x, pn_y, rtol=1e-12, atol=1e-14)


def test_rope_scores_depend_on_relative_position_only():
    q = rand(1, 1, 128, seed=5)
    k = rand(1, 1, 128, seed=6)
    def score(pq, pk):
        return float((O.rope(q, torch.tensor([pq]), 1e4) * O.rope(k, torch.tensor([pk]), 1e4)).sum())
    assert math.isclose(score(10, 3), score(110, 103), rel_tol=1e-11)
    assert math.isclose(score(2000, 1990), score(10, 0), rel_tol=1e-11)
    assert not math.isclose(score(10, 3), score(10, 4), rel_tol=1e-6)


# ----------------------------------------------------------------- softmax / attention
def test_softmax_rows_sum_to_one_and_shift_invariant():
    s = rand(7, 33, seed=7) * 10
    p = O.softmax(s)
    assert torch.allclose(p.sum(dim=1), torch.ones(7, dtype=F64), rtol=0, atol=1e-14)
    assert torch.allclose(O.softmax(s + 123.0), p, rtol=1e-12)
    s[:, 5:] = -math.inf
    assert torch.all(O.softmax(s)[:, 5:] == 0)


def test_single_key_returns_v_exactly():
    q = rand(1, 4, 16, seed=8)
    k = rand(1, 2, 16, seed=9)
    v = rand(1, 2, 16, seed=10)
    o = O.gqa_attention(q, k, v, torch.tensor([0])).reshape(4, 16)
    for h in range(4):
        assert torch.equal(o[h], v[0, h // 2])


def test_zero_query_gives_causal_mean_of_v():
    t, n, hq, hkv, d = 4, 9, 4, 2, 8
    q = torch.zeros(t, hq, d, dtype=F64)
    k = rand(n, hkv, d, seed=11)
    v = rand(n, hkv, d, seed=12)
    pos = torch.tensor([0, 3, 5, 8])
    o = O.gqa_attention(q, k, v, pos).reshape(t, hq, d)
    for r in range(t):
        for h in range(hq):
            expect = v[: pos[r] + 1, h // 2].mean(dim=0)
            assert torch.allclose(o[r, h], expect, rtol=1e-13, atol=1e-15)


def brute_attention(q, k, v, pos):
    """Pure-Python loops: one query head against its KV head, keys j <= pos."""
    t, hq, d = q.shape
    hkv = k.shape[1]
    out = np.zeros((t, hq, d))
    for r in range(t):
        for h in range(hq):
            g = h // (hq // hkv)
            scores = []
            for j in range(int(pos[r]) + 1):
                scores.append(sum(float(q[r, h, c]) * float(k[j, g, c]) for c in range(d)) / math.sqrt(d))
            m = max(scores)
            w = [math.exp(s - m) for s in scores]
            z = sum(w)
            for c in range(d):
                out[r, h, c] = sum(w[j] * float(v[j, g, c]) for j in range(len(w))) / z
    return out.reshape(t, hq * d)


@pytest.mark.parametrize("hq,hkv", [(4, 4), (4, 2), (4, 1), (6, 3)])
def test_gqa_matches_loop_brute_force(hq, hkv):
    t, n, d = 3, 6, 4
    q = rand(t, hq, d, seed=13)
    k = rand(n, hkv, d, seed=14)
    v = rand(n, hkv, d, seed=15)
    pos = torch.tensor([2, 3, 5])
    np.testing.assert_allclose(O.gqa_attention(q, k, v, pos).numpy(), brute_attention(q, k, v, pos),
                               rtol=1e-12, atol=1e-14)


def test_attention_is_causal():
    t, n, hq, hkv, d = 3, 8, 2, 1, 8
    q = rand(t, hq, d, seed=16)
    k = rand(n, hkv, d, seed=17)
    v = rand(n, hkv, d, seed=18)
    pos = torch.tensor([2, 4, 7])
    base = O.gqa_attention(q, k, v, pos)
    k2, v2 = k.clone(), v.clone()
    k2[5:] += 100.0
    v2[5:] -= 50.0
    pert = O.gqa_attention(q, k2, v2, pos)
    assert torch.equal(base[:2], pert[:2])
    assert not torch.equal(base[2], pert[2])


# ----------------------------------------------------------------- SwiGLU
def test_silu_special_values():
    z = torch.tensor([0.0, 1.0, 40.0, -40.0], dtype=F64)
    s = O.silu(z)
    assert s[0] == 0.0
    assert math.isclose(float(s[1]), 0.73105857863000487925, rel_tol=1e-15)   # 1 / (1 + e^-1)
    assert math.isclose(float(s[2]), 40.0, rel_tol=1e-15)
    assert abs(float(s[3])) < 1e-15


# ----------------------------------------------------------------- element types
def test_bf16_rounding_matches_library_and_ties_to_even():
    x = rand(100000, seed=19) * torch.logspace(-20, 20, 100000, dtype=F64)
    ref = x.to(torch.float32).to(torch.bfloat16).to(F64)          # torch: nearest-even casts
    assert torch.equal(O.round_to_bf16(x), ref)
    one = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 1.0 + 2 ** -8 + 2 ** -20], dtype=F64)
    assert O.round_to_bf16(one).tolist() == [1.0, 1.015625, -1.0, 1.0078125]


def test_widen_bf16_is_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0001, 0x7F7F, 0x3FC0], dtype=np.uint16)
    assert O.widen_bf16(bits).tolist() == [1.0, -1.0, 2.0 ** -133, 3.3895313892515355e38, 1.5]


# ----------------------------------------------------------------- whole layer
TINY3 = StageShape("pin", 99, 2, 8, 2, 1, 4, 6)


def tiny_bits(seed):
    """bf16-exact small weights for the 8-wide layer (values k/64, |k| <= 8)."""
    g = torch.Generator().manual_seed(seed)
    out = {}
    for name, shp in {"wq": (8, 8), "wk": (4, 8), "wv": (4, 8), "wo": (8, 8), "wg": (6, 8),
                      "wu": (6, 8), "wd": (8, 6), "g1": (8,), "g2": (8,)}.items():
        vals = torch.randint(-8, 9, shp, generator=g).to(torch.float32) / 64
        if name in ("g1", "g2"):
            vals = 1.0 + vals / 2
        out[name] = O.bf16_bits(vals.to(F64))
    return out


def brute_layer(x, bits, p0, kcache, vcache, shape, round_kv):
    """Pure-Python loops for one decoder layer (no torch ops), rows at p0, p0+1, ..."""
    w = {n: O.widen_bf16(b).numpy() for n, b in bits.items()}
    hq, hkv, d, hdim, f = shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.hidden, shape.ffn
    def matvec(m, vec):
        return [sum(float(m[i, j]) * vec[j] for j in range(len(vec))) for i in range(m.shape[0])]
    def norm(vec, g):
        ms = sum(a * a for a in vec) / len(vec)
        return [a / math.sqrt(ms + shape.rms_eps) * float(g[i]) for i, a in enumerate(vec)]
    def rot(vec, p):
        out = list(vec)
        for i in range(d // 2):
            a = p * shape.rope_theta ** (-2.0 * i / d)
            x1, x2 = vec[i], vec[i + d // 2]
            out[i] = x1 * math.cos(a) - x2 * math.sin(a)
            out[i + d // 2] = x1 * math.sin(a) + x2 * math.cos(a)
        return out
    outs = []
    for r, row in enumerate(x):
        p = p0 + r
        row = [float(a) for a in row]
        y = norm(row, w["g1"])
        q, k, v = matvec(w["wq"], y), matvec(w["wk"], y), matvec(w["wv"], y)
        q = sum((rot(q[h * d:(h + 1) * d], p) for h in range(hq)), [])
        k = sum((rot(k[g * d:(g + 1) * d], p) for g in range(hkv)), [])
        kcache.append([round_kv(a) for a in k])
        vcache.append([round_kv(a) for a in v])
        o = []
        for h in range(hq):
            g = h // (hq // hkv)
            sc = [sum(q[h * d + c] * kcache[j][g * d + c] for c in range(d)) / math.sqrt(d) for j in range(p + 1)]
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            o += [sum(e[j] * vcache[j][g * d + c] for j in range(p + 1)) / sum(e) for c in range(d)]
        row = [a + b for a, b in zip(row, matvec(w["wo"], o))]
        y2 = norm(row, w["g2"])
        gate, up = matvec(w["wg"], y2), matvec(w["wu"], y2)
        hmid = [gv / (1 + math.exp(-gv)) * uv for gv, uv in zip(gate, up)]
        row = [a + b for a, b in zip(row, matvec(w["wd"], hmid))]
        outs.append(row)
    return np.array(outs)


def f32_round_scalar(a):
    return float(np.float32(a))


def test_layer_matches_loop_brute_force_f32_kv():
    bits = tiny_bits(20)
    x = rand(5, 8, seed=21).numpy()
    st = O.OracleStage(TINY3, lambda l: bits, kv_dtype="f32")
    # one layer only: run the stage's layer 0 through the public pieces
    cache = O.LayerCache(1, 4)
    got = O.decoder_layer(torch.as_tensor(x), O.LayerWeights(bits), cache, TINY3, O.round_to_f32).numpy()
    kc, vc = [], []
    ref = brute_layer(x, bits, 0, kc, vc, TINY3, f32_round_scalar)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)
    # stored cache equals the brute-force cache
    np.testing.assert_allclose(cache.k.reshape(5, 4).numpy(), np.array(kc), rtol=0, atol=0)
    np.testing.assert_allclose(cache.v.reshape(5, 4).numpy(), np.array(vc), rtol=0, atol=0)
    assert st.shape is TINY3


def test_layer_rows_match_loop_brute_force():
    """layer_kv (the K/V a layer stores) and decoder_layer_rows (the layer restricted to some rows,
    attending over given stored K/V) against the pure-Python loop brute force of the whole layer."""
    bits = tiny_bits(24)
    x = rand(9, 8, seed=25).numpy()
    kc, vc = [], []
    ref = brute_layer(x, bits, 0, kc, vc, TINY3, f32_round_scalar)
    w = O.LayerWeights(bits)
    xt = torch.as_tensor(x)
    k, v = O.layer_kv(xt, w, TINY3, O.round_to_f32)
    np.testing.assert_allclose(k.reshape(9, 4).numpy(), np.array(kc), rtol=0, atol=0)
    np.testing.assert_allclose(v.reshape(9, 4).numpy(), np.array(vc), rtol=0, atol=0)
    rows = [0, 3, 8]
    got = O.decoder_layer_rows(xt, w, TINY3, rows, k, v).numpy()
    np.testing.assert_allclose(got, ref[rows], rtol=1e-12, atol=1e-13)


def test_layer_with_zero_output_projections_is_identity():
    bits = tiny_bits(22)
    bits["wo"] = np.zeros_like(bits["wo"])
    bits["wd"] = np.zeros_like(bits["wd"])
    x = rand(3, 8, seed=23)
    out = O.decoder_layer(x, O.LayerWeights(bits), O.LayerCache(1, 4), TINY3, O.round_to_bf16)
    assert torch.equal(out, x)


def test_decode_rows_equal_prefill_rows():
    """Decode step t (one row on top of the cache) equals row t of one prefill."""
    bits = {l: tiny_bits(30 + l) for l in range(2)}
    x = rand(7, 8, seed=31).numpy()
    full = O.OracleStage(TINY3, lambda l: bits[l], kv_dtype="bf16")
    ref = full.forward([("s", x)])[0]
    inc = O.OracleStage(TINY3, lambda l: bits[l], kv_dtype="bf16")
    rows = [inc.forward([("s", x[:4])])[0]]
    for t in range(4, 7):
        rows.append(inc.forward([("s", x[t:t + 1])])[0])
    np.testing.assert_allclose(np.concatenate(rows), ref, rtol=1e-13, atol=1e-13)
    for l in range(2):
        assert torch.equal(inc.cache("s")[l].k, full.cache("s")[l].k) or torch.allclose(
            inc.cache("s")[l].k, full.cache("s")[l].k, rtol=0, atol=2 ** -8)


def test_sequences_are_independent_and_order_free():
    bits = {l: tiny_bits(40 + l) for l in range(2)}
    a = rand(3, 8, seed=41).numpy()
    b = rand(5, 8, seed=42).numpy()
    st1 = O.OracleStage(TINY3, lambda l: bits[l])
    ra, rb = st1.forward([("a", a), ("b", b)])
    st2 = O.OracleStage(TINY3, lambda l: bits[l])
    rb2, = st2.forward([("b", b)])
    ra2, = st2.forward([("a", a)])
    assert np.array_equal(ra, ra2) and np.array_equal(rb, rb2)


def test_kv_tail_export_and_reappend_round_trip():
    bits = {l: tiny_bits(50 + l) for l in range(2)}
    x = rand(9, 8, seed=51).numpy()
    nxt = rand(1, 8, seed=52).numpy()
    ref = O.OracleStage(TINY3, lambda l: bits[l])
    ref.forward([("s", x)])
    want = ref.forward([("s", nxt)])[0]
    st = O.OracleStage(TINY3, lambda l: bits[l])
    st.forward([("s", x)])
    k, v = st.export_tail("s", 4, drop=True)
    assert st.length("s") == 5 and k.shape == (2, 4, 1, 4)
    st.append_kv("s", k, v)
    assert np.array_equal(st.forward([("s", nxt)])[0], want)


def test_kv_jitter_zero_is_the_plain_definition_and_small_jitter_stays_close():
    bits = {l: tiny_bits(60 + l) for l in range(2)}
    x = rand(9, 8, seed=61).numpy()
    plain = O.OracleStage(TINY3, lambda l: bits[l]).forward([("s", x)])[0]
    zero = O.OracleStage(TINY3, lambda l: bits[l], kv_jitter=0.0).forward([("s", x)])[0]
    assert np.array_equal(plain, zero)
    jit = O.OracleStage(TINY3, lambda l: bits[l], kv_jitter=2.0 ** -16, jitter_seed=3).forward([("s", x)])[0]
    assert np.abs(jit - plain).max() < 0.05 * np.abs(plain).max()
