"""Decode throughput of one pipeline stage on one MI355X.

Headline workload: the LLaMA-3.3-70B-shaped stage (one of five pipeline stages: 16 decoder
layers, hidden 8192, 64 query / 8 KV heads, head_dim 128, SwiGLU 28672, bf16 weights all
resident in HBM, bf16 paged KV cache) serving 4 interleaved micro-batches of batch 1: a prefill
of 2048 tokens each (one call, timed), then decode steps round robin across the micro-batches,
one micro-batch per call (Section III-A: micro-batches take turns through a stage).  One timed
step is one decode call: every layer (RMSNorm, QKV, RoPE + KV store, GQA attention over the
cache, O + residual, RMSNorm, gate/up + SwiGLU, down + residual) for one new token of one
micro-batch, its input already in HBM.  Weights are random bf16(N(0, 0.02)) (gains
bf16(1 + N(0, 0.02))) generated on the device, hidden states N(0, 1): timing only; the parity of
every configuration here is covered by the tests.

Prints one JSON line: value = decode tokens/s of the stage; the roofline of the dominant kernel
(the one-row 70B gate/up projection, HIP events on the compute stream over the timed region);
whole-step HBM bandwidth; the prefill's MFMA utilisation; the float64 CPU oracle timed per unit on
the machine's host (single thread, extrapolated); and sub-legs: the 8B-shaped stage (1024-token
prefill + 128 decode steps), the tiny stage (latency: us and kernels per step), other groupings
of the 70B micro-batches, the offloaded stage (4 resident + 12 streamed layers: prefill and decode
overlap), zero copy, KV pressure, KV parking, the online planner and the allocation scheduler.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, published
MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak, published
OVERLAP_TARGET = 0.8    # hidden-shorter fraction the offloaded stage should reach

# HBM bytes of one one-row gate/up launch, from two rocprofv3 --pmc runs of this script (FETCH_SIZE,
# then WRITE_SIZE, per dispatch, each scaled by what the counter reads for a plain 1 GiB device copy
# in the same run).  Valid for the GEMV source it was taken on: with any other source the field is
# reported as null.
GATEUP_TRAFFIC = {
    "llama3.3-70b-shaped-16L": {"bytes": 940172778,
                                "source_sha256": "b86a279723f17c625b0331b91585831d31090808d9141c423fd3f7f5a4f43d1b"},
    "llama3-8b-shaped-8L": {"bytes": 235246452,
                            "source_sha256": "b86a279723f17c625b0331b91585831d31090808d9141c423fd3f7f5a4f43d1b"},
}
KERNEL_SOURCES = ("paper_2512_21835_amd/csrc/gemv.hip", "paper_2512_21835_amd/csrc/stage_kernels.h")


def gateup_bytes(shape, rows: int) -> int:
    """Algorithmic HBM bytes of one gate/up launch: both weight matrices once, gains, x in, h out."""
    h, f = shape.hidden, shape.ffn
    return 2 * f * h * 2 + h * 2 + rows * h * 4 + rows * f * 4


def decode_step_bytes(shape, ctx_before: int) -> int:
    """Algorithmic HBM bytes of one batch-1 decode step at a context of ctx_before tokens.

    Every layer's weights once, the KV cache read (ctx_before + 1 positions, K and V, bf16),
    the new K/V written, and the hidden state in and out of each projection (fp32).
    """
    h, f, qd, kvd = shape.hidden, shape.ffn, shape.q_dim, shape.kv_dim
    weights = shape.layer_bytes()
    kv = (ctx_before + 1) * 2 * kvd * 2 + 2 * kvd * 2
    acts = 4 * (h + (qd + 2 * kvd) + qd + qd + h + h + 2 * h + f + f + 2 * h)
    return shape.n_layers * (weights + kv + acts)


def kernel_source_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def gateup_traffic(shape):
    t = GATEUP_TRAFFIC.get(shape.name)
    if not t or t["bytes"] is None or t["source_sha256"] != kernel_source_sha256():
        return None
    return t["bytes"]


def prefill_flops(shape, T: int):
    """Algorithmic flops of a T-token prefill of one sequence: (projection GEMMs, causal attention)."""
    h, f, qd, kvd = shape.hidden, shape.ffn, shape.q_dim, shape.kv_dim
    params = h * (qd + 2 * kvd) + qd * h + 2 * f * h + f * h
    gemm = 2 * params * T * shape.n_layers
    attn = 4 * (T * (T + 1) // 2) * shape.n_q_heads * shape.head_dim * shape.n_layers
    return gemm, attn


def prefill_report(shape, T: int, n_seqs: int, seconds: float):
    gemm, attn = prefill_flops(shape, T)
    gemm, attn = gemm * n_seqs, attn * n_seqs
    peak = MFMA_BF16_PEAK_TFLOPS * 1e12 * seconds
    return {"tokens": T * n_seqs, "sequences": n_seqs, "tokens_per_s": T * n_seqs / seconds, "ms": seconds * 1e3,
            "tflop_algorithmic": (gemm + attn) / 1e12,
            # algorithmic flops against the bf16 matrix peak; the projections issue two MFMAs per
            # product (the fp32 activation as a bf16 hi/lo pair)
            "mfma_frac_algorithmic": (gemm + attn) / peak, "mfma_frac_issued": (2 * gemm + attn) / peak}


def _union(iv):
    out = []
    for s, e in sorted(iv):
        if out and s <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e)
        else:
            out.append([s, e])
    return out


def _length(iv):
    return sum(e - s for s, e in iv)


def _intersect(a, b):
    i = j = 0
    tot = 0.0
    while i < len(a) and j < len(b):
        lo, hi = max(a[i][0], b[j][0]), min(a[i][1], b[j][1])
        tot += max(0.0, hi - lo)
        if a[i][1] < b[j][1]:
            i += 1
        else:
            j += 1
    return tot


def overlap(seg):
    """Copy/compute overlap of one call's timeline records (kind, layer, start, end)."""
    copies = _union([(s, e) for k, _, s, e in seg if k in (1, 4)])
    comp = _union([(s, e) for k, _, s, e in seg if k in (3, 5)])
    call = [(s, e) for k, _, s, e in seg if k == 0][0]
    t_copy, t_comp = _length(copies), _length(comp)
    t_call = max(call[1], copies[-1][1]) - min(call[0], copies[0][0])
    both = _intersect(copies, comp)
    hs = both / min(t_copy, t_comp)
    return {"ms_per_call": t_call, "copy_ms": t_copy, "compute_ms": t_comp,
            "hidden_copy_frac": both / t_copy, "hidden_copy_ceiling": min(1.0, t_comp / t_copy),
            "hidden_shorter_frac": hs, "exposed_copy_ms": t_call - t_comp,
            "overlap_below_target": hs < OVERLAP_TARGET}


def last_call(tl):
    """The records of the last call of a timeline (a call's copy and layer records precede its
    call record)."""
    ends = [i for i, r in enumerate(tl) if r[0] == 0]
    return tl[ends[-2] + 1: ends[-1] + 1] if len(ends) > 1 else tl[: ends[-1] + 1]


def device_weights(shape, layer, gen, dev):
    """Random bf16 weights of one layer generated on the device: N(0, 0.02), gains 1 + N(0, 0.02)."""
    import synth
    import torch
    w = {}
    for name, shp in synth.layer_weight_shapes(shape).items():
        t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
        w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
    return w


def load_random(P, h, shape, gen, dev, code_of):
    for l in range(shape.n_layers):
        w = device_weights(shape, l, gen, dev)
        P.stage_load_layer(h, l, w, code_of(l))
        del w


def random_kv(shape, n, gen, dev):
    import torch
    return [torch.randn(shape.n_layers, n, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
            .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


# ---------------------------------------------------------------------------------------------- legs
def cpu_baseline(layers_timed: int = 8, ctx: int = 2048):
    """The float64 oracle as it stands, single-threaded, timed per unit on the headline workload
    and extrapolated: one decode step of one sequence at context `ctx` (its cache filled with seeded
    K/V) through `layers_timed` of the 16 70B-shaped layers (each layer's bf16 weights widened as the
    oracle does on every pass), scaled to 16 layers."""
    import numpy as np
    import torch

    import synth
    from oracle.stage_oracle import OracleStage
    shape = synth.LLAMA70B_STAGE
    wl = synth.WORKLOADS["llama70b_resident"]
    part = synth.StageShape(shape.name + "-part", shape.shape_id, layers_timed, shape.hidden, shape.n_q_heads,
                            shape.n_kv_heads, shape.head_dim, shape.ffn, shape.rope_theta, shape.rms_eps)
    weights = [synth.layer_weights(shape, l) for l in range(layers_timed)]
    threads = torch.get_num_threads()
    torch.set_num_threads(1)
    try:
        orc = OracleStage(part, lambda l: weights[l], kv_dtype="bf16")
        seed = synth.seed_of(0xB0, 2, 0)
        k = synth.bf16_to_f32(synth.normal_bf16(seed, (layers_timed, ctx, shape.n_kv_heads, shape.head_dim)))
        v = synth.bf16_to_f32(synth.normal_bf16(seed + 1, (layers_timed, ctx, shape.n_kv_heads, shape.head_dim)))
        orc.append_kv("s", k.astype(np.float64), v.astype(np.float64))
        x = synth.decode_input(wl, 0, 0, 0)[None]
        t0 = time.perf_counter()
        orc.forward([("s", x)])
        dt = time.perf_counter() - t0
    finally:
        torch.set_num_threads(threads)
    per_token = dt * shape.n_layers / layers_timed
    return {"value": 1.0 / per_token, "unit": "decode tokens/s", "cores": 1, "kind": "oracle",
            "extrapolated": True, "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "sample": f"one decode step of one sequence at context {ctx} through {layers_timed} of the 16 "
                      f"70B-shaped layers (float64 torch, 1 thread, weights widened per pass), "
                      f"{dt:.2f} s, extrapolated linearly to 16 layers"}


def c3_leg(K: int, W: int, T: int, other_rounds: int):
    """The headline: 70B-shaped stage, all layers resident, 4 micro-batches of batch 1.

    One prefill call of 4 x T tokens is timed (after the same prefill of four other sequences as a
    warm-up); then W warm-up and K timed decode steps round robin, one micro-batch per call, with
    HIP events around one gate/up launch per call.  Then, on the same stage and weights, the other
    groupings (`other_rounds` rounds each): the round robin on two and four decode lanes, the 4
    micro-batches in one call, and 8 micro-batches of batch 2 in one call."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    L, H, n_mb = shape.n_layers, shape.hidden, 4
    dev = torch.device("cuda", 0)
    cs = torch.cuda.current_stream(dev)
    max_ctx = T + (W + K) // n_mb + 2 + 5 * (other_rounds + 1) + 8
    cfg = P.config_for(shape, max_microbatches=8, max_batch=2, max_context=max_ctx, n_resident_max=L,
                       compute_stream=cs.cuda_stream, n_lanes=4)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2513)
    out = {}
    try:
        t_gen = time.perf_counter()
        load_random(P, h, shape, gen, dev, lambda l: 1)
        torch.cuda.synchronize()
        out["weight_setup_s"] = time.perf_counter() - t_gen
        xp = torch.randn(n_mb, 1, T, H, generator=gen, device=dev)
        yp = torch.empty_like(xp)
        P.stage_prefill(h, [4, 5, 6, 7], 1, T, xp, yp)             # warm-up: four other sequences
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.stage_prefill(h, [0, 1, 2, 3], 1, T, xp, yp)
        torch.cuda.synchronize()
        out["prefill"] = prefill_report(shape, T, n_mb, time.perf_counter() - t0)
        out["prefill"]["kernels_per_call"] = P.stage_get_stats(h)["last_call_kernels"]
        assert bool(torch.isfinite(yp).all()), "non-finite prefill output"

        xw = torch.randn(max(W, 1), 1, H, generator=gen, device=dev)
        xd = torch.randn(K, 1, H, generator=gen, device=dev)
        yw, yd = torch.empty_like(xw), torch.empty_like(xd)
        host = []   # host side of one call with nothing queued: argument checks, metadata, 97 launches
        for s in range(W):
            torch.cuda.synchronize()
            th = time.perf_counter()
            P.stage_decode(h, [s % n_mb], 1, xw[s:s + 1], yw[s:s + 1])
            host.append(time.perf_counter() - th)
        torch.cuda.synchronize()
        out["host_ms_per_call"] = sorted(host)[len(host) // 2] * 1e3 if host else None
        P.stage_get_timeline(h)                       # clear
        P.stage_set_timing(h, P.STAGE_TIME_GATEUP)   # HIP events around one gate/up launch per call
        ctx0 = [P.stage_get_length(h, m, 0) for m in range(n_mb)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(K):
            P.stage_decode(h, [s % n_mb], 1, xd[s:s + 1], yd[s:s + 1])
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        P.stage_set_timing(h, 0)
        tl = P.stage_get_timeline(h)
        out["kernels_per_step"] = P.stage_get_stats(h)["last_call_kernels"]
        assert bool(torch.isfinite(yd).all()), "non-finite decode output"
        gu = [e - s for kind, _, s, e in tl if kind == 2]
        step_bytes = sum(decode_step_bytes(shape, ctx0[s % n_mb] + s // n_mb) for s in range(K)) / K
        out.update({"K": K, "dt": dt, "gu_ms": sum(gu) / len(gu), "gu_launches": len(gu),
                    "step_bytes": step_bytes, "ctx": (min(ctx0), max(ctx0) + (K - 1) // n_mb + 1)})

        if other_rounds <= 0:
            return out
        # other groupings on the same stage: fill the batch-2 rows and sequences 4..7 to the same context
        for m in range(8):
            for b in range(2):
                need = P.stage_get_length(h, 0, 0) - P.stage_get_length(h, m, b)
                if need > 0:
                    kv = random_kv(shape, need, gen, dev)
                    P.stage_kv_append(h, m, b, need, kv[0], kv[1])
                    del kv
        out["other_groupings"] = other_groupings(P, h, shape, gen, dev, other_rounds)
    finally:
        P.stage_destroy(h)
    return out


def other_groupings(P, h, shape, gen, dev, rounds):
    import torch
    L, layer = shape.n_layers, shape.layer_bytes()
    x = torch.randn(8, 2, shape.hidden, generator=gen, device=dev)
    res = {}
    modes = {"round_robin_2_lanes": ([[m] for m in range(4)], 1, 2),
             "round_robin_4_lanes": ([[m] for m in range(4)], 1, 4),
             "4_in_one_call": ([list(range(4))], 1, 1), "16_rows_in_one_call": ([list(range(8))], 2, 1)}
    ctx = P.stage_get_length(h, 0, 0)
    for mode, (groups, B, lanes) in modes.items():
        xs = [x[g[0]: g[0] + len(g), :B].contiguous() for g in groups]
        ys = [torch.empty_like(xi) for xi in xs]
        torch.cuda.synchronize()

        def one_round():
            for i, (g, xi, yi) in enumerate(zip(groups, xs, ys)):
                P.stage_decode_lane(h, i % lanes, g, B, xi, yi)
        one_round()                              # warm-up round
        P.stage_sync(h)
        t0 = time.perf_counter()
        for _ in range(rounds):
            one_round()
        P.stage_sync(h)
        dt = time.perf_counter() - t0
        calls = rounds * len(groups)
        tokens = rounds * sum(len(g) for g in groups) * B
        alg = calls * L * layer + tokens * L * (ctx + 2 * rounds) * 2 * shape.kv_dim * 2
        # algorithmic bytes (weights once per call, KV per token); the lanes' overlapping calls read
        # the same layer's weights at nearly the same time, so part of the second read may hit cache
        res[mode] = {"tokens_per_s": tokens / dt, "ms_per_call": dt * 1e3 / calls,
                     "algorithmic_GBs": alg / dt / 1e9, "algorithmic_frac": alg / dt / 1e9 / HBM_PEAK_GBS}
    res["workload"] = (f"llama70b_resident decode at context {ctx}: 4 micro-batches of batch 1 round robin on two or "
                       f"four decode lanes (micro-batch m on lane m mod n), or all 4 in one call; 8 micro-batches "
                       f"of batch 2 in one call (16 rows, matrix cores)")
    return res


def c2_leg(K: int, W: int, T: int):
    """The 8B-shaped stage (8 layers, all resident), batch 1: a T-token prefill (timed), then W
    warm-up and K timed decode steps with events around one gate/up launch per call.  Seeded
    weights and inputs (the same as the parity tests')."""
    import numpy as np
    import torch

    import synth
    import paper_2512_21835_amd as P

    wl = synth.WORKLOADS["llama8b_stage"]
    shape = wl.shape
    dev = torch.device("cuda", 0)
    cs = torch.cuda.current_stream(dev)
    ctx = T + max(K, W)
    weights = [synth.layer_weights(shape, l) for l in range(shape.n_layers)]
    cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=ctx, n_resident_max=shape.n_layers,
                       compute_stream=cs.cuda_stream)
    h = P.stage_init(cfg)
    try:
        for l, w in enumerate(weights):
            P.stage_load_layer(h, l, w, 1)
        xp = [torch.from_numpy(synth.prefill_inputs(wl, m, 0, T)).to(dev) for m in (0, 1)]
        yp = [torch.empty_like(x) for x in xp]
        P.stage_prefill(h, [0], 1, T, xp[0], yp[0])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.stage_prefill(h, [1], 1, T, xp[1], yp[1])
        torch.cuda.synchronize()
        prefill_s = time.perf_counter() - t0
        xw = torch.from_numpy(np.stack([synth.decode_input(wl, 0, 0, s) for s in range(W)])).to(dev)
        xd = torch.from_numpy(np.stack([synth.decode_input(wl, 1, 0, s) for s in range(K)])).to(dev)
        yw, yd = torch.empty_like(xw), torch.empty_like(xd)
        for s in range(W):
            P.stage_decode(h, [0], 1, xw[s:s + 1], yw[s:s + 1])
        torch.cuda.synchronize()
        P.stage_get_timeline(h)
        P.stage_set_timing(h, P.STAGE_TIME_GATEUP)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(K):
            P.stage_decode(h, [1], 1, xd[s:s + 1], yd[s:s + 1])
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        P.stage_set_timing(h, 0)
        tl = P.stage_get_timeline(h)
        kernels = P.stage_get_stats(h)["last_call_kernels"]
        assert bool(torch.isfinite(yd).all()), "non-finite decode output"
    finally:
        P.stage_destroy(h)
    step_bytes = sum(decode_step_bytes(shape, T + s) for s in range(K)) / K
    gu = [e - s for kind, _, s, e in tl if kind == 2]
    gu_ms = sum(gu) / len(gu)
    ms = dt * 1e3 / K
    return {
        "workload": f"llama8b_stage decode: 8 layers, hidden 4096, 32/8 heads x 128, ffn 14336, bf16 weights "
                    f"resident, bf16 paged KV, batch 1, context {T}->{T + K}",
        "tokens_per_s": K / dt, "ms_per_step": ms, "kernels_per_step": kernels,
        "roofline": {"bound": "hbm", "kernel": "gate/up projection + SwiGLU (gemv, 1 row)",
                     "achieved": gateup_bytes(shape, 1) / (gu_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gateup_bytes(shape, 1) / (gu_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": gateup_traffic(shape), "bytes_per_launch": gateup_bytes(shape, 1),
                     "avg_launch_ms": gu_ms, "launches": len(gu)},
        "step_hbm": {"bytes_per_step": step_bytes, "achieved_GBs": step_bytes / (ms * 1e-3) / 1e9,
                     "frac": step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "prefill": prefill_report(shape, T, 1, prefill_s),
    }


def c1_leg(K: int = 256, W: int = 16):
    """The tiny stage (2 layers, hidden 256) on its own call sequence: prefill 16 tokens, then 16
    decode steps each feeding its output back as the next input (on the device), contexts 17..32.
    The sequence is reset and run again until K decode steps have been timed (after W warm-up
    steps).  Latency-bound: reports microseconds per step (host clock over each run of 16
    back-to-back steps), the GPU span of one call from its events, and the kernels a step enqueues."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    wl = synth.WORKLOADS["tiny"]
    shape = wl.shape
    steps = 16
    dev = torch.device("cuda", 0)
    cs = torch.cuda.current_stream(dev)
    cfg = P.config_for(shape, max_microbatches=1, max_batch=1, max_context=16 + steps + 2,
                       n_resident_max=shape.n_layers, compute_stream=cs.cuda_stream)
    h = P.stage_init(cfg)
    try:
        for l in range(shape.n_layers):
            P.stage_load_layer(h, l, synth.layer_weights(shape, l), 1)
        x = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 16)).to(dev)
        y = torch.empty_like(x)
        buf = torch.empty(steps + 1, 1, shape.hidden, device=dev)
        warm, runs = max(1, W // steps), max(1, K // steps)

        def run(timed_last: bool) -> float:
            P.stage_reset_sequence(h, 0, 0)
            P.stage_prefill(h, [0], 1, 16, x, y)
            buf[0].copy_(y[-1])
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for s in range(steps):
                if timed_last and s == steps - 1:
                    torch.cuda.synchronize()
                    P.stage_get_timeline(h)
                    P.stage_set_timing(h, P.STAGE_TIME_CALLS)
                P.stage_decode(h, [0], 1, buf[s:s + 1], buf[s + 1:s + 2])
            torch.cuda.synchronize()
            return time.perf_counter() - t0

        dt = 0.0
        for r in range(warm + runs):
            t = run(False)
            if r >= warm:
                dt += t
        kernels = P.stage_get_stats(h)["last_call_kernels"]
        run(True)   # the last step (context 32) timed by its events
        tl = P.stage_get_timeline(h)
        P.stage_set_timing(h, 0)
        assert bool(torch.isfinite(buf).all()), "non-finite decode output"
    finally:
        P.stage_destroy(h)
    call = [e - s for k, _, s, e in tl if k == 0][-1]
    return {"workload": "tiny decode: 2 layers, hidden 256, 4/2 heads x 64, ffn 688, batch 1, prefill 16 then 16 "
                        "decode steps, outputs fed back as the next inputs (contexts 17..32), the sequence reset "
                        "and run again",
            "us_per_step": dt * 1e6 / (runs * steps), "gpu_us_per_call": call * 1e3, "kernels_per_step": kernels,
            "steps": runs * steps, "weight_bytes": 2 * shape.layer_bytes(), "bound": "latency (weights fit in L2)"}


def offload_leg(calls: int, ctx: int = 2048, zero_copy: bool = False, prefill: bool = True, slots: int = 2,
                decode: bool = True):
    """The 70B-shaped stage with 4 resident layers and 12 streamed through 2 HBM slots from pinned
    host memory (the library's own copy stream), 4 micro-batches.  Without zero copy: a prefill of
    4 x `ctx` tokens in one call (the regime where compute and copies are of the same order), then
    decode calls carrying all four micro-batches (streamed layers loaded once per call); both timed
    with events on the copy and compute streams.  With `zero_copy` the contexts are filled through
    stage_kv_append and the decode kernels of the 12 offloaded layers read their pinned host blobs
    directly (no slot copies); the report gives the call time and the host-link rate of those reads.
    `slots`: streaming slots; `decode=False` returns after the prefill."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    n_mb, L = 4, shape.n_layers
    cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=1, max_context=ctx + calls + 2, n_resident_max=4,
                       n_stream_slots=slots, compute_stream=cstream.cuda_stream, zero_copy=zero_copy)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2512)
    res = {}
    try:
        load_random(P, h, shape, gen, dev, lambda l: 1 if l < 4 else 0)
        blob = P.stage_get_stats(h)["layer_bytes"]
        # pinned host -> HBM copy rate of one layer blob, on a side stream
        src = torch.empty(blob, dtype=torch.uint8, pin_memory=True)
        dst = torch.empty(blob, dtype=torch.uint8, device=dev)
        side = torch.cuda.Stream(dev)
        with torch.cuda.stream(side):
            dst.copy_(src, non_blocking=True)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(side)
            for _ in range(3):
                dst.copy_(src, non_blocking=True)
            e1.record(side)
        e1.synchronize()
        h2d_gbs = 3 * blob / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del src, dst
        streamed = 12 * blob
        if prefill and not zero_copy:
            xp = torch.randn(n_mb, 1, ctx, shape.hidden, generator=gen, device=dev)
            yp = torch.empty_like(xp)
            P.stage_sync(h)
            P.stage_get_timeline(h)
            P.stage_set_timing(h, P.STAGE_TIME_CALLS | P.STAGE_TIME_LAYERS)
            t0 = time.perf_counter()
            P.stage_prefill(h, list(range(n_mb)), 1, ctx, xp, yp)
            P.stage_sync(h)
            wall = time.perf_counter() - t0
            P.stage_set_timing(h, 0)
            ov = overlap(last_call(P.stage_get_timeline(h)))
            res["prefill"] = dict(ov, tokens=n_mb * ctx, tokens_per_s=n_mb * ctx / wall,
                                  link_GBs=streamed / (ov["ms_per_call"] * 1e-3) / 1e9)
            del xp, yp
            if not decode:
                return {"slots": slots, "prefill": res["prefill"]}
        else:
            for m in range(n_mb):
                kv = random_kv(shape, ctx, gen, dev)
                P.stage_kv_append(h, m, 0, ctx, kv[0], kv[1])
                del kv
        x = torch.randn(n_mb, 1, shape.hidden, generator=gen, device=dev)
        y = torch.empty_like(x)
        P.stage_decode(h, list(range(n_mb)), 1, x, y)   # warm-up call
        P.stage_sync(h)
        P.stage_get_timeline(h)
        P.stage_set_timing(h, P.STAGE_TIME_CALLS | P.STAGE_TIME_LAYERS)
        t0 = time.perf_counter()
        for _ in range(calls):
            P.stage_decode(h, list(range(n_mb)), 1, x, y)
        P.stage_sync(h)
        wall = time.perf_counter() - t0
        tl = P.stage_get_timeline(h)
        stats = P.stage_get_stats(h)
    finally:
        P.stage_destroy(h)
    seg = last_call(tl)
    if zero_copy:
        call = [(s, e) for k, _, s, e in seg if k == 0][0]
        t_direct = sum(e - s for k, l, s, e in seg if k in (3, 5) and l >= 4)
        return {
            "workload": f"llama70b_offload decode, zero-copy: 16 layers (hidden 8192, 64/8 heads, ffn 28672), 4 "
                        f"resident + 12 read by the decode kernels from pinned host memory, 4 micro-batches of "
                        f"batch 1 per call, context {ctx}",
            "tokens_per_s": n_mb * calls / wall, "ms_per_call": call[1] - call[0],
            "host_read_GB_per_call": streamed / 1e9, "offloaded_layers_ms": t_direct,
            "host_read_GBs": streamed / (t_direct * 1e-3) / 1e9, "h2d_peak_GBs": h2d_gbs,
            "link_util": streamed / (t_direct * 1e-3) / 1e9 / h2d_gbs,
            "layer_loads": stats["layer_loads"], "bytes_direct": stats["bytes_direct"],
        }
    ov = overlap(seg)
    res.update({
        "workload": f"llama70b_offload: 16 layers (hidden 8192, 64/8 heads, ffn 28672), 4 resident + 12 streamed "
                    f"through {slots} HBM slots from pinned host memory on the library's copy stream, 4 micro-batches of "
                    f"batch 1 per call; prefill {ctx} tokens each in one call, then decode calls at context {ctx}",
        "tokens_per_s": n_mb * calls / wall, "streamed_GB_per_call": streamed / 1e9,
        "link_GBs": streamed / (ov["ms_per_call"] * 1e-3) / 1e9, "h2d_peak_GBs": h2d_gbs,
        "link_util": streamed / (ov["ms_per_call"] * 1e-3) / 1e9 / h2d_gbs, "layer_loads": stats["layer_loads"],
        "mha_block_bytes": stats["mha_block_bytes"], "mlp_block_bytes": stats["mlp_block_bytes"],
    })
    res.update(ov)
    return res


def planner_leg(calls: int = 3, ctx: int = 2048, n_steps: int = 6):
    """The 70B-shaped stage, all 16 layers allocated resident, 4 micro-batches of batch 1 decoded
    in one call each step, under the online planner (Eq. (7), stage_plan_offload): the memory left
    for the cache holds the four sequences at context `ctx` plus 64 tokens (so TS^1 = 4*ctx + 64,
    Eq. (6)), each offloaded block frees its bytes once (#Stage = 2) and a block's loading time is
    its bytes.  The cache is grown through stage_kv_append (random K/V) to each of the first
    `n_steps` thresholds in turn; at each, the first decode call applies the step (its extra wall
    time is the switch), then `calls` more calls give the step's call time."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    L, n_mb = shape.n_layers, 4
    kv_token = 2 * shape.kv_dim * 2 * L            # bytes of one token's K and V over the stage
    probe = P.stage_init(P.config_for(shape, max_microbatches=1, max_batch=1, max_context=16, n_resident_max=L,
                                      compute_stream=cstream.cuda_stream))
    try:
        st = P.stage_get_stats(probe)
    finally:
        P.stage_destroy(probe)
    mha, mlp = st["mha_block_bytes"], st["mlp_block_bytes"]
    steps, capacity = P.stage_plan_offload((n_mb * ctx + 64) * kv_token, kv_token, mha, mlp, mha, mlp, L, L, 2)
    steps = steps[:n_steps]
    max_ctx = ctx + (steps[-1][0] - n_mb * ctx) // n_mb + 2 * (calls + 2) + 16
    cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=1, max_context=max_ctx, n_resident_max=L,
                       compute_stream=cstream.cuda_stream, plan=steps)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2514)
    out = []
    try:
        load_random(P, h, shape, gen, dev, lambda l: 1)

        def grow(per_seq):
            if per_seq <= 0:
                return
            for m in range(n_mb):
                kv = random_kv(shape, per_seq, gen, dev)
                P.stage_kv_append(h, m, 0, per_seq, kv[0], kv[1])

        def held():
            return sum(P.stage_get_length(h, m, 0) for m in range(n_mb))

        grow(ctx)
        x = torch.randn(n_mb, 1, shape.hidden, generator=gen, device=dev)
        y = torch.empty_like(x)

        def call():
            t0 = time.perf_counter()
            P.stage_decode(h, list(range(n_mb)), 1, x, y)
            P.stage_sync(h)
            return (time.perf_counter() - t0) * 1e3

        for k, (tokens, alpha, beta) in enumerate(steps):
            if k > 0:
                grow(-(-(tokens - n_mb - held()) // n_mb))
            first = call()
            steady = [call() for _ in range(calls)]
            per = sum(steady) / len(steady)
            out.append({"tokens": held(), "threshold": tokens, "alpha": alpha, "beta": beta,
                        "residency": "".join(map(str, P.stage_get_residency(h, L))), "first_call_ms": first,
                        "call_ms": per,
                        "switch_ms": first - per, "offloaded_GB_per_call": (alpha * mha + beta * mlp) / 1e9})
        log = P.stage_get_residency_log(h)
    finally:
        P.stage_destroy(h)
    return {
        "workload": f"llama70b planner: 16 layers (hidden 8192, 64/8 heads, ffn 28672) allocated resident, 4 "
                    f"micro-batches of batch 1 per decode call, cache grown from context {ctx} through the "
                    f"first {len(steps)} steps of the online planner (Eq. (7), #Stage 2, cost = block bytes)",
        "mha_block_bytes": mha, "mlp_block_bytes": mlp, "kv_bytes_per_token": kv_token,
        "capacity_tokens": capacity, "steps": out, "residency_changes": len(log),
    }


def kvpressure_leg(contexts=(512, 4352, 8192), rounds: int = 2):
    """The KV-pressure workload on the 70B-shaped stage: 8 micro-batches of batch 2, residency
    shrinking 16 -> 8 under the threshold schedule TS_j = 512 + 960 j (one more layer streamed
    through 2 slots per threshold passed).  Sampled: at each context in `contexts` the caches are
    filled to it through stage_kv_append (random K/V), then `rounds` decode rounds are timed (one
    warm-up round first) two ways: round robin, one micro-batch per call (every call streams the
    offloaded layers), and all 8 micro-batches in one call (16 rows; each offloaded layer streams
    once per round).  Reports the round time, tokens/s, the resident layers, and the HBM fraction
    (weights of resident layers, slots read once per call, KV read) when no layer streams."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    wl = synth.WORKLOADS["llama70b_kvpressure"]
    shape = wl.shape
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    L, n_mb, B = shape.n_layers, wl.n_mb, wl.batch
    gen = torch.Generator(device=dev).manual_seed(2516)
    x = torch.randn(n_mb, B, shape.hidden, generator=gen, device=dev)
    ys = [torch.empty_like(x[m:m + 1]) for m in range(n_mb)]
    out = []
    layer = shape.layer_bytes()
    for ctx in contexts:
        cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=B, max_context=ctx + 2 * rounds + 6, n_resident_max=L,
                           n_stream_slots=2, thresholds=wl.thresholds, compute_stream=cstream.cuda_stream)
        h = P.stage_init(cfg)
        try:
            load_random(P, h, shape, gen, dev, lambda l: 1)
            for m in range(n_mb):
                for b in range(B):
                    kv = random_kv(shape, ctx - 1, gen, dev)
                    P.stage_kv_append(h, m, b, ctx - 1, kv[0], kv[1])
                    del kv

            def round_():
                for m in range(n_mb):
                    P.stage_decode(h, [m], B, x[m:m + 1], ys[m])

            round_()                                  # warm-up; applies the thresholds passed
            P.stage_sync(h)
            t0 = time.perf_counter()
            for _ in range(rounds):
                round_()
            P.stage_sync(h)
            dt = (time.perf_counter() - t0) / rounds
            res = P.stage_get_residency(h, L)
            x_all, y_all = x.contiguous(), torch.empty_like(x)
            P.stage_decode(h, list(range(n_mb)), B, x_all, y_all)    # warm-up of the one-call grouping
            P.stage_sync(h)
            t0 = time.perf_counter()
            for _ in range(rounds):
                P.stage_decode(h, list(range(n_mb)), B, x_all, y_all)
            P.stage_sync(h)
            dt1 = (time.perf_counter() - t0) / rounds
            res1 = P.stage_get_residency(h, L)
        finally:
            P.stage_destroy(h)
        resident = sum(1 for c in res if c == 1)
        kv_read = n_mb * B * L * (ctx + rounds) * 2 * shape.kv_dim * 2
        hbm = n_mb * L * layer + kv_read             # every call reads every layer once (slot or HBM)
        entry = {"context": ctx, "resident_layers": resident, "ms_per_round": dt * 1e3,
                 "tokens_per_s": n_mb * B / dt}
        if resident == L:
            entry["hbm_GBs"] = hbm / dt / 1e9
            entry["hbm_frac"] = hbm / dt / 1e9 / HBM_PEAK_GBS
        else:
            entry["streamed_GB_per_round"] = n_mb * (L - resident) * layer / 1e9
        resident1 = sum(1 for c in res1 if c == 1)
        one = {"resident_layers": resident1, "ms_per_round": dt1 * 1e3, "tokens_per_s": n_mb * B / dt1}
        if resident1 == L:
            hbm1 = L * layer + n_mb * B * L * (ctx + 2 * rounds + 1) * 2 * shape.kv_dim * 2
            one["hbm_GBs"] = hbm1 / dt1 / 1e9
            one["hbm_frac"] = hbm1 / dt1 / 1e9 / HBM_PEAK_GBS
        else:
            one["streamed_GB_per_round"] = (L - resident1) * layer / 1e9
        entry["one_call"] = one
        out.append(entry)
    return {"workload": "llama70b_kvpressure decode: 16 layers (hidden 8192, 64/8 heads, ffn 28672), 8 micro-batches "
                        "of batch 2 round robin (one_call: all 8 in one call), residency 16 -> 8 by thresholds "
                        "512 + 960 j, 2 slots; sampled at the listed contexts",
            "samples": out}


def parking_leg(rounds: int = 32, ctx: int = 1024, n_parks=(128, 512)):
    """The KV transfer protocol on one GPU (Alg. 2, pinned host memory as the peer): the
    8B-shaped stage, all 8 layers resident, 4 micro-batches of batch 1 at context `ctx` (filled
    through stage_kv_append with random K/V), decoded round robin, one micro-batch per call.
    Without parking, then with it: before micro-batch m's call the next micro-batch's tail is
    requested back (stage_kv_unpark, copy stream), and after the call m's last n_park tokens
    move out (stage_kv_park), for each n_park in `n_parks`.  Also without parking on two decode
    lanes and on four (micro-batch m on lane m mod n: calls overlap).  Reports the call time each
    way, the bytes each call moves over the host link, and the KV blocks held in HBM after the
    last call."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA8B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    L, n_mb = shape.n_layers, 4
    gen = torch.Generator(device=dev).manual_seed(2515)
    weights = [device_weights(shape, l, gen, dev) for l in range(L)]
    kv = [random_kv(shape, ctx, gen, dev) for _ in range(n_mb)]
    x = torch.randn(n_mb, 1, 1, shape.hidden, generator=gen, device=dev)
    res = {}
    for n_park, lanes in [(0, 1), (0, 2), (0, 4)] + [(n, 1) for n in n_parks]:
        park = n_park > 0
        cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=1, max_context=ctx + rounds + 8, n_resident_max=L,
                           compute_stream=cstream.cuda_stream, kv_park_tokens=n_park, n_lanes=lanes)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                P.stage_load_layer(h, l, weights[l], 1)
            for m in range(n_mb):
                P.stage_kv_append(h, m, 0, ctx, kv[m][0], kv[m][1])
            ys = [torch.empty_like(x[m]) for m in range(n_mb)]

            def step(m):
                if park:
                    P.stage_kv_unpark(h, [(m + 1) % n_mb])
                P.stage_decode_lane(h, m % lanes, [m], 1, x[m], ys[m])
                if park:
                    P.stage_kv_park(h, [m], n_park)

            for m in range(n_mb):          # warm-up round (the first parks)
                step(m)
            P.stage_sync(h)
            t0 = time.perf_counter()
            for i in range(rounds * n_mb):
                step(i % n_mb)
            P.stage_sync(h)
            dt = time.perf_counter() - t0
            st = P.stage_get_stats(h)
        finally:
            P.stage_destroy(h)
        key = f"park_{n_park}" if park else ("plain" if lanes == 1 else f"plain_{lanes}_lanes")
        res[key] = {
            "ms_per_call": dt * 1e3 / (rounds * n_mb), "kv_blocks_in_hbm": st["kv_blocks"] - st["kv_blocks_free"],
            "host_link_MB_per_call": (st["bytes_parked"] + st["bytes_unparked"]) / 1e6 / ((rounds + 1) * n_mb)}
        if park:
            res[key]["overhead"] = res[key]["ms_per_call"] / res["plain"]["ms_per_call"] - 1
    res["workload"] = (f"llama8b_stage decode: 8 layers resident, 4 micro-batches of batch 1 at context {ctx}, round "
                       f"robin one per call (plain_n_lanes: micro-batch m on decode lane m mod n); parking moves the "
                       f"last n tokens of each micro-batch between its calls and fetches the next one's back ahead "
                       f"of its call")
    return res


def eq1_total(n_stage, devices, assigned, retained, offloaded, comm):
    """Eq. (1) for a given spread, whole-layer offloading: sum of compute, the s * |D| hops, and the
    largest loading time a device's overlap window (its retained layers' compute plus every other
    device's compute and the hops) leaves uncovered."""
    comp = [d[1] for d in devices]
    total = sum(c * a for c, a in zip(comp, assigned)) + n_stage * len(devices) * comm
    worst = 0
    for i, d in enumerate(devices):
        window = comp[i] * retained[i] + sum(comp[j] * assigned[j] for j in range(len(devices)) if j != i) \
            + len(devices) * comm
        worst = max(worst, offloaded[i] * (d[2] + d[3]) - window)
    return total + max(0, worst)


def allocation_report(resident_4_in_one_ms: float, offload: dict, device_mem_gb=(32, 24, 20, 16),
                      n_layers: int = 80):
    """The cost model and the allocation scheduler fed with this run's measurements.

    comp = one 70B-shaped layer's decode time for 4 micro-batches in one call (the resident leg),
    load = a block's bytes over the measured pinned host-to-HBM rate (the offload leg).  Eq. (1)
    for one device holding the offload leg's 4 resident + 12 offloaded layers is compared with
    that leg's measured call time; Alg. 1 then allocates an 80-layer model of the same layer
    shape over four devices with the given weight memories (a design study: one GPU is measured,
    the others are assumed identical to it).  Beside Alg. 1's plan, Eq. (1) is evaluated for an
    even spread of the same left-over layers: the printed dynamic program minimises the carried
    sum of uncovered delays, under which every spread that gives each device at least one layer it
    cannot hide ties, and its "<=" update gives the tie to the last device."""
    import paper_2512_21835_amd as P

    layer_ms = resident_4_in_one_ms / 16
    rate = offload["h2d_peak_GBs"] * 1e9 / 1e3            # bytes per ms
    mha, mlp = offload["mha_block_bytes"], offload["mlp_block_bytes"]
    ns = lambda ms: int(round(ms * 1e6))
    comp, load_a, load_m = ns(layer_ms), ns(mha / rate), ns(mlp / rate)
    # Eq. (1), one device, no hops: compute of 16 layers + the loading the 4 resident layers leave uncovered
    predicted = (16 * comp + max(0, 12 * (load_a + load_m) - 4 * comp)) / 1e6
    devices = [(int(g * 1e9), comp, load_a, load_m) for g in device_mem_gb]
    n_stage, t_total, plans = P.stage_allocate(n_layers, mha, mlp, 0, devices)
    cap = [d[0] // (mha + mlp) for d in devices]
    left = n_layers - sum(cap)
    even = [left // len(devices) + (1 if i < left % len(devices) else 0) for i in range(len(devices))]
    t_even = eq1_total(n_stage, devices, [c + e for c, e in zip(cap, even)], cap, even, 0)
    t_plan_whole = eq1_total(n_stage, devices, [p[1] for p in plans], cap, [p[2] for p in plans], 0)
    return {
        "inputs": {"layer_ms_4_microbatches": layer_ms, "load_mha_ms": load_a / 1e6, "load_mlp_ms": load_m / 1e6},
        "eq1_offload_leg": {"predicted_ms_per_call": predicted, "measured_ms_per_call": offload["ms_per_call"],
                            "ratio": offload["ms_per_call"] / predicted},
        "alg1_80_layers": {"device_weight_memory_GB": list(device_mem_gb), "n_stage": n_stage,
                           "t_total_ms": t_total / 1e6,
                           "devices": [dict(zip(("first_layer", "assigned", "offloaded", "mha_only", "mlp_only"), p))
                                       for p in plans],
                           "note": "printed DP: ties between spreads go to the last device"},
        "eq1_same_layers_spread_evenly": {"offloaded": even, "t_total_ms": t_even / 1e6,
                                          "alg1_plan_whole_layers_t_total_ms": t_plan_whole / 1e6},
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1024,
                    help="timed decode steps of the headline (one micro-batch per step, round robin over 4)")
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--prefill", type=int, default=2048, help="prefill tokens per micro-batch of the headline")
    ap.add_argument("--other-rounds", type=int, default=8, help="timed rounds of the other 70B groupings (0 = skip)")
    ap.add_argument("--cpu-layers", type=int, default=8,
                    help="70B-shaped layers the oracle is timed on for cpu_baseline, about 1.2 s each "
                         "(0 = skip)")
    ap.add_argument("--c2-steps", type=int, default=128, help="timed decode steps of the 8B-shaped leg (0 = skip)")
    ap.add_argument("--c1-steps", type=int, default=256, help="timed decode steps of the tiny leg (0 = skip)")
    ap.add_argument("--offload-calls", type=int, default=3, help="timed calls of the offloaded 70B leg (0 = skip)")
    ap.add_argument("--kvpressure-rounds", type=int, default=2,
                    help="timed rounds per sampled context of the 70B KV-pressure leg (0 = skip)")
    ap.add_argument("--parking-rounds", type=int, default=32,
                    help="timed round-robin rounds of the KV parking leg (0 = skip)")
    ap.add_argument("--planner-calls", type=int, default=3,
                    help="timed calls per planner step of the 70B planner leg (0 = skip)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for hardware traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one stage on one GPU; --gpus {args.gpus} is not supported "
              "(the stage does not shard across GPUs).", file=sys.stderr)
        return 2

    import torch

    import synth

    dev = torch.device("cuda", 0)
    stream = torch.cuda.Stream(dev)
    torch.cuda.set_stream(stream)
    K, W, T = args.steps, args.warmup, args.prefill
    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    shape = synth.LLAMA70B_STAGE
    c3 = c3_leg(K, W, T, args.other_rounds)
    ms_step = c3["dt"] * 1e3 / K
    gu_bytes = gateup_bytes(shape, 1)
    achieved = gu_bytes / (c3["gu_ms"] * 1e-3) / 1e9
    out = {
        "metric": "decode tokens/s per stage", "value": K / c3["dt"], "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"llama70b_resident decode: 16 layers (hidden 8192, 64/8 heads x 128, ffn 28672), bf16 "
                               f"weights all resident, bf16 paged KV; 4 interleaved micro-batches of batch 1, prefill "
                               f"{T} each, decode round robin one micro-batch per call, context "
                               f"{c3['ctx'][0]}->{c3['ctx'][1]}",
                   "global_batch": 4, "seq_len": c3["ctx"][1], "parallelism": "none (one stage, one GPU)",
                   "weights": "bf16", "kv_cache": "bf16", "accumulate": "f32"},
        "roofline": {"bound": "hbm", "kernel": "gate/up projection + SwiGLU (gemv, 1 row, 70B-shaped layer)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": gateup_traffic(shape), "bytes_per_launch": gu_bytes,
                     "avg_launch_ms": c3["gu_ms"], "launches": c3["gu_launches"]},
        "step_hbm": {"bytes_per_step": c3["step_bytes"],
                     "achieved_GBs": c3["step_bytes"] / (ms_step * 1e-3) / 1e9,
                     "frac": c3["step_bytes"] / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "kernels_per_step": c3["kernels_per_step"],
        "host_ms_per_call": c3["host_ms_per_call"],
        "prefill": c3["prefill"],
        "weight_setup_s": c3["weight_setup_s"],
    }
    if "other_groupings" in c3 and args.other_rounds > 0:
        out["resident70b"] = c3["other_groupings"]
    if args.c2_steps > 0:
        out["llama8b_stage"] = c2_leg(args.c2_steps, 16, 1024)
    if args.c1_steps > 0:
        out["tiny"] = c1_leg(args.c1_steps)
    if args.kvpressure_rounds > 0:
        out["kvpressure70b"] = kvpressure_leg(rounds=args.kvpressure_rounds)
    if args.parking_rounds > 0:
        out["kv_parking"] = parking_leg(args.parking_rounds)
    if args.planner_calls > 0:
        out["planner"] = planner_leg(args.planner_calls)
    if args.offload_calls > 0:
        out["offload"] = offload_leg(args.offload_calls)
        # the same prefill with more streaming slots: the copy engine no longer waits for a slot
        # while the resident layers compute
        out["offload"]["prefill_more_slots"] = {str(S): offload_leg(0, slots=S, decode=False)["prefill"]
                                                for S in (3, 4)}
        out["offload_zero_copy"] = offload_leg(args.offload_calls, zero_copy=True)
        if "resident70b" in out:
            out["allocation"] = allocation_report(out["resident70b"]["4_in_one_call"]["ms_per_call"], out["offload"])
    if args.cpu_layers > 0:
        out["cpu_baseline"] = cpu_baseline(args.cpu_layers)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
