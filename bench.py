"""Decode throughput of one pipeline stage on one MI355X.

Workload: the LLaMA-3-8B-shaped stage (8 decoder layers, hidden 4096, 32 query /
8 KV heads, head_dim 128, SwiGLU 14336, bf16 weights resident in HBM, bf16 paged
KV cache), batch 1, prefill 1024 tokens, then decode steps.  One timed step is
one decode step of the whole stage (all layers: RMSNorm, QKV, RoPE + KV store,
GQA attention, O + residual, RMSNorm, gate/up + SwiGLU, down + residual) for one
new token, with its input already in HBM.  Inputs are seeded synthetic hidden
states N(0, 1); weights bf16(N(0, 0.02)), gains bf16(1 + N(0, 0.02)).

Prints one JSON line: value = decode tokens/s of the stage, plus the roofline of
the dominant kernel (the gate/up projection, measured with HIP events on the
compute stream over the timed region), whole-step HBM bandwidth, prefill
throughput and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, published
MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak, published

# HBM bytes of one gate/up launch (8B-shaped layer, 1 row), from two rocprofv3 --pmc runs of this
# script (FETCH_SIZE, then WRITE_SIZE, per dispatch, each scaled by what the counter reads for a
# plain 1 GiB device copy in the same run).  Valid for the GEMV source it was taken on: with any
# other source the field is reported as null.
GATEUP_TRAFFIC = {"bytes": 235259002,
                  "source_sha256": "e777833278ae2ff5d75ff4ad83970d5e41d1c0b523fbca1a4a771d884799cd66"}
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


def prefill_flops(shape, T: int):
    """Algorithmic flops of a T-token prefill of one sequence: (projection GEMMs, causal attention)."""
    h, f, qd, kvd = shape.hidden, shape.ffn, shape.q_dim, shape.kv_dim
    params = h * (qd + 2 * kvd) + qd * h + 2 * f * h + f * h
    gemm = 2 * params * T * shape.n_layers
    attn = 4 * (T * (T + 1) // 2) * shape.n_q_heads * shape.head_dim * shape.n_layers
    return gemm, attn


def cpu_baseline(shape, weights, wl, n_tokens: int):
    """The float64 oracle as it stands, decoding n_tokens fresh tokens after a 16-token prefill."""
    import torch

    import synth
    from oracle.stage_oracle import OracleStage
    orc = OracleStage(shape, weights, kv_dtype="bf16")
    orc.forward([("s", synth.prefill_inputs(wl, 7, 0, 16))])
    t0 = time.perf_counter()
    for i in range(n_tokens):
        orc.forward([("s", synth.decode_input(wl, 7, 0, i)[None])])
    dt = time.perf_counter() - t0
    return {"value": n_tokens / dt, "unit": "decode tokens/s", "cores": torch.get_num_threads(),
            "kind": "oracle",
            "sample": f"{n_tokens} decode tokens of the same 8-layer stage after a 16-token prefill "
                      f"(float64 torch CPU; per-token cost is the weight pass, context adds <1%)"}


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


def offload_leg(calls: int, ctx: int = 2048, zero_copy: bool = False):
    """The 70B-shaped stage with 4 resident layers and 12 streamed through 2 HBM slots.

    Four micro-batches at context `ctx` (filled through stage_kv_append with random K/V), each
    decode call carrying all four (streamed layers loaded once per call).  Reports the call time
    and the copy/compute overlap measured from events: slot copies on the copy stream, layer
    compute intervals on the compute stream.  With `zero_copy` the decode kernels of the 12
    offloaded layers read their pinned host blobs directly instead (no slot copies); the report
    then gives the call time and the host-link rate those reads reach.  Weights are random bf16
    generated on the device (timing only; parity of this configuration is covered by the tests).
    """
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    xstream = torch.cuda.Stream(dev)
    n_mb, L = 4, shape.n_layers
    cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=1, max_context=ctx + calls + 2, n_resident_max=4,
                       n_stream_slots=2, compute_stream=cstream.cuda_stream, copy_stream=xstream.cuda_stream,
                       zero_copy=zero_copy)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2512)
    try:
        for l in range(L):
            w = {}
            for name, shp in synth.layer_weight_shapes(shape).items():
                t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
                w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
            P.stage_load_layer(h, l, w, 1 if l < 4 else 0)
            del w
        for m in range(n_mb):
            kv = [torch.randn(L, ctx, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
                  .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)]
            P.stage_kv_append(h, m, 0, ctx, kv[0], kv[1])
        # pinned host -> HBM copy rate of one layer blob, measured on the copy stream
        blob = P.stage_get_stats(h)["layer_bytes"]
        src = torch.empty(blob, dtype=torch.uint8, pin_memory=True)
        dst = torch.empty(blob, dtype=torch.uint8, device=dev)
        with torch.cuda.stream(xstream):
            dst.copy_(src, non_blocking=True)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(xstream)
            for _ in range(3):
                dst.copy_(src, non_blocking=True)
            e1.record(xstream)
        e1.synchronize()
        h2d_gbs = 3 * blob / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del src, dst
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
    # records are in enqueue order; a call's copy and layer records precede its call record
    ends = [i for i, r in enumerate(tl) if r[0] == 0]
    seg = tl[ends[-2] + 1: ends[-1] + 1] if len(ends) > 1 else tl[: ends[-1] + 1]
    last = [(s, e) for k, _, s, e in seg if k == 0][0]
    streamed = 12 * blob
    if zero_copy:
        t_call = last[1] - last[0]
        direct = [(l, e - s) for k, l, s, e in seg if k in (3, 5) and l >= 4]
        t_direct = sum(d for _, d in direct)
        return {
            "workload": f"llama70b_offload decode, zero-copy: 16 layers (hidden 8192, 64/8 heads, ffn 28672), 4 "
                        f"resident + 12 read by the decode kernels from pinned host memory, 4 micro-batches of "
                        f"batch 1 per call, context {ctx}",
            "tokens_per_s": n_mb * calls / wall, "ms_per_call": t_call, "host_read_GB_per_call": streamed / 1e9,
            "offloaded_layers_ms": t_direct, "host_read_GBs": streamed / (t_direct * 1e-3) / 1e9,
            "h2d_peak_GBs": h2d_gbs, "link_util": streamed / (t_direct * 1e-3) / 1e9 / h2d_gbs,
            "layer_loads": stats["layer_loads"], "bytes_direct": stats["bytes_direct"],
        }
    copies = _union([(s, e) for k, _, s, e in seg if k in (1, 4)])
    comp = _union([(s, e) for k, _, s, e in seg if k in (3, 5)])
    t_copy, t_comp = _length(copies), _length(comp)
    t_call = max(last[1], copies[-1][1]) - min(last[0], copies[0][0])
    both = _intersect(copies, comp)
    return {
        "workload": f"llama70b_offload decode: 16 layers (hidden 8192, 64/8 heads, ffn 28672), 4 resident + 12 "
                    f"streamed through 2 HBM slots from pinned host memory, 4 micro-batches of batch 1 per call, "
                    f"context {ctx}",
        "tokens_per_s": n_mb * calls / wall, "ms_per_call": t_call, "streamed_GB_per_call": streamed / 1e9,
        "copy_ms": t_copy, "compute_ms": t_comp,
        "hidden_copy_frac": both / t_copy, "hidden_copy_ceiling": min(1.0, t_comp / t_copy),
        "hidden_shorter_frac": both / min(t_copy, t_comp),
        "link_GBs": streamed / (t_call * 1e-3) / 1e9, "h2d_peak_GBs": h2d_gbs,
        "link_util": streamed / (t_call * 1e-3) / 1e9 / h2d_gbs,
        "exposed_copy_ms": t_call - t_comp, "layer_loads": stats["layer_loads"],
        "mha_block_bytes": stats["mha_block_bytes"], "mlp_block_bytes": stats["mlp_block_bytes"],
    }


def prefill_report(shape, T: int, seconds: float):
    gemm, attn = prefill_flops(shape, T)
    peak = MFMA_BF16_PEAK_TFLOPS * 1e12 * seconds
    return {"tokens": T, "tokens_per_s": T / seconds, "ms": seconds * 1e3,
            "tflop_algorithmic": (gemm + attn) / 1e12,
            # algorithmic flops against the bf16 matrix peak; the projections issue two MFMAs per
            # product (the fp32 activation as a bf16 hi/lo pair), attention runs on the vector units
            "mfma_frac_algorithmic": (gemm + attn) / peak, "mfma_frac_issued": 2 * gemm / peak}


def resident70b_leg(rounds: int, ctx: int = 2048):
    """The 70B-shaped stage with all 16 layers resident and sequences at context `ctx` (filled
    through stage_kv_append with random K/V), decoded four ways: 4 micro-batches of batch 1
    round-robin, one micro-batch per call (every call streams all weights for one token); the same
    round robin on two and on four decode lanes (micro-batch m on lane m mod n: calls overlap); the same
    4 in one call (weights read once for 4 tokens); 8 micro-batches of batch 2 in one call (16 rows,
    matrix cores).  Weights are random bf16 generated on the device (timing only;
    parity of these configurations is covered by the tests)."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    L = shape.n_layers
    lane_streams = [None] + [torch.cuda.Stream(dev).cuda_stream for _ in range(3)]
    cfg = P.config_for(shape, max_microbatches=8, max_batch=2, max_context=ctx + 5 * (rounds + 1) + 8,
                       n_resident_max=L, compute_stream=cstream.cuda_stream, n_lanes=4, lane_streams=lane_streams)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2513)
    res = {}
    try:
        for l in range(L):
            w = {}
            for name, shp in synth.layer_weight_shapes(shape).items():
                t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
                w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
            P.stage_load_layer(h, l, w, 1)
            del w
        for m in range(8):
            for b in range(2):
                kv = [torch.randn(L, ctx, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
                      .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)]
                P.stage_kv_append(h, m, b, ctx, kv[0], kv[1])
        x = torch.randn(8, 2, shape.hidden, generator=gen, device=dev)
        y = torch.empty_like(x)
        layer = shape.layer_bytes()
        modes = {"round_robin": ([[m] for m in range(4)], 1, 1), "round_robin_2_lanes": ([[m] for m in range(4)], 1, 2),
                 "round_robin_4_lanes": ([[m] for m in range(4)], 1, 4),
                 "4_in_one_call": ([list(range(4))], 1, 1), "16_rows_in_one_call": ([list(range(8))], 2, 1)}
        for mode, (groups, B, lanes) in modes.items():
            xs = [x[g[0]: g[0] + len(g), :B].contiguous() for g in groups]
            ys = [torch.empty_like(xi) for xi in xs]
            torch.cuda.synchronize()

            def one_round():
                for i, (g, xi, yi) in enumerate(zip(groups, xs, ys)):
                    P.stage_decode_lane(h, i % lanes, g, B, xi, yi)
            one_round()                              # warm-up round
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(rounds):
                one_round()
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            calls = rounds * len(groups)
            tokens = rounds * sum(len(g) for g in groups) * B
            hbm = calls * L * layer + tokens * L * (ctx + 5 * rounds) * 2 * shape.kv_dim * 2
            res[mode] = {"tokens_per_s": tokens / dt, "ms_per_call": dt * 1e3 / calls,
                         "hbm_GBs": hbm / dt / 1e9, "hbm_frac": hbm / dt / 1e9 / HBM_PEAK_GBS}
    finally:
        P.stage_destroy(h)
    res["workload"] = (f"llama70b_resident decode: 16 layers (hidden 8192, 64/8 heads, ffn 28672) resident, "
                       f"context {ctx}; 4 micro-batches of batch 1 (round robin on one, two or four decode lanes, or "
                       f"one call), or 8 of batch 2 in one call")
    return res


def planner_leg(calls: int = 3, ctx: int = 2048, n_steps: int = 6):
    """The 70B-shaped stage, all 16 layers allocated resident, 4 micro-batches of batch 1 decoded
    in one call each step, under the online planner (Eq. (7), stage_plan_offload): the memory left
    for the cache holds the four sequences at context `ctx` plus 64 tokens (so TS^1 = 4*ctx + 64,
    Eq. (6)), each offloaded block frees its bytes once (#Stage = 2) and a block's loading time is
    its bytes.  The cache is grown through stage_kv_append (random K/V) to each of the first
    `n_steps` thresholds in turn; at each, the first decode call applies the step (its extra wall
    time is the switch), then `calls` more calls give the step's call time.  Weights are random
    bf16 generated on the device (timing only; parity of planner-driven residency is covered by
    the tests)."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA70B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    xstream = torch.cuda.Stream(dev)
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
                       compute_stream=cstream.cuda_stream, copy_stream=xstream.cuda_stream, plan=steps)
    h = P.stage_init(cfg)
    gen = torch.Generator(device=dev).manual_seed(2514)
    out = []
    try:
        for l in range(L):
            w = {}
            for name, shp in synth.layer_weight_shapes(shape).items():
                t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
                w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
            P.stage_load_layer(h, l, w, 1)
            del w

        def grow(per_seq):
            if per_seq <= 0:
                return
            for m in range(n_mb):
                kv = [torch.randn(L, per_seq, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
                      .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)]
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
    xstream = torch.cuda.Stream(dev)
    L, n_mb, B = shape.n_layers, wl.n_mb, wl.batch
    gen = torch.Generator(device=dev).manual_seed(2516)
    x = torch.randn(n_mb, B, shape.hidden, generator=gen, device=dev)
    ys = [torch.empty_like(x[m:m + 1]) for m in range(n_mb)]
    out = []
    layer = shape.layer_bytes()
    for ctx in contexts:
        cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=B, max_context=ctx + 2 * rounds + 6, n_resident_max=L,
                           n_stream_slots=2, thresholds=wl.thresholds, compute_stream=cstream.cuda_stream,
                           copy_stream=xstream.cuda_stream)
        h = P.stage_init(cfg)
        try:
            for l in range(L):
                w = {}
                for name, shp in synth.layer_weight_shapes(shape).items():
                    t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
                    w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
                P.stage_load_layer(h, l, w, 1)
                del w
            for m in range(n_mb):
                for b in range(B):
                    kv = [torch.randn(L, ctx - 1, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
                          .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)]
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
    lanes and on four (micro-batch m on lane m mod n: calls overlap).  Reports the call time each way, the
    bytes each call moves over the host link, and the KV blocks held in HBM after the last call."""
    import torch

    import synth
    import paper_2512_21835_amd as P

    shape = synth.LLAMA8B_STAGE
    dev = torch.device("cuda", 0)
    cstream = torch.cuda.current_stream(dev)
    xstream = torch.cuda.Stream(dev)
    L, n_mb = shape.n_layers, 4
    gen = torch.Generator(device=dev).manual_seed(2515)
    weights = []
    for l in range(L):
        w = {}
        for name, shp in synth.layer_weight_shapes(shape).items():
            t = torch.randn(shp, generator=gen, device=dev) * 0.02 + (1.0 if name in ("g1", "g2") else 0.0)
            w[name] = t.to(torch.bfloat16).view(torch.int16).contiguous()
        weights.append(w)
    kv = [[torch.randn(L, ctx, shape.n_kv_heads, shape.head_dim, generator=gen, device=dev)
           .to(torch.bfloat16).view(torch.int16).contiguous() for _ in range(2)] for _ in range(n_mb)]
    x = torch.randn(n_mb, 1, 1, shape.hidden, generator=gen, device=dev)
    res = {}
    lane_streams = [None] + [torch.cuda.Stream(dev).cuda_stream for _ in range(3)]
    for n_park, lanes in [(0, 1), (0, 2), (0, 4)] + [(n, 1) for n in n_parks]:
        park = n_park > 0
        cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=1, max_context=ctx + rounds + 8, n_resident_max=L,
                           compute_stream=cstream.cuda_stream, copy_stream=xstream.cuda_stream,
                           kv_park_tokens=n_park, n_lanes=lanes, lane_streams=lane_streams)
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


def allocation_report(resident: dict, offload: dict, device_mem_gb=(32, 24, 20, 16), n_layers: int = 80):
    """The cost model and the allocation scheduler fed with this run's measurements.

    comp = one 70B-shaped layer's decode time for 4 micro-batches in one call (the resident leg),
    load = a block's bytes over the measured pinned host-to-HBM rate (the offload leg).  Eq. (1)
    for one device holding the offload leg's 4 resident + 12 offloaded layers is compared with
    that leg's measured call time; Alg. 1 then allocates an 80-layer model of the same layer
    shape over four devices with the given weight memories (a design study: one GPU is
    measured, the others are assumed identical to it)."""
    import paper_2512_21835_amd as P

    layer_ms = resident["4_in_one_call"]["ms_per_call"] / 16
    rate = offload["h2d_peak_GBs"] * 1e9 / 1e3            # bytes per ms
    mha, mlp = offload["mha_block_bytes"], offload["mlp_block_bytes"]
    ns = lambda ms: int(round(ms * 1e6))
    comp, load_a, load_m = ns(layer_ms), ns(mha / rate), ns(mlp / rate)
    # Eq. (1), one device, no hops: compute of 16 layers + the loading the 4 resident layers leave uncovered
    predicted = (16 * comp + max(0, 12 * (load_a + load_m) - 4 * comp)) / 1e6
    devices = [(int(g * 1e9), comp, load_a, load_m) for g in device_mem_gb]
    n_stage, t_total, plans = P.stage_allocate(n_layers, mha, mlp, 0, devices)
    return {
        "inputs": {"layer_ms_4_microbatches": layer_ms, "load_mha_ms": load_a / 1e6, "load_mlp_ms": load_m / 1e6},
        "eq1_offload_leg": {"predicted_ms_per_call": predicted, "measured_ms_per_call": offload["ms_per_call"],
                            "ratio": offload["ms_per_call"] / predicted},
        "alg1_80_layers": {"device_weight_memory_GB": list(device_mem_gb), "n_stage": n_stage,
                           "t_total_ms": t_total / 1e6,
                           "devices": [dict(zip(("first_layer", "assigned", "offloaded", "mha_only", "mlp_only"), p))
                                       for p in plans]},
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--prefill", type=int, default=1024)
    ap.add_argument("--cpu-tokens", type=int, default=4, help="oracle decode tokens for cpu_baseline (0 = skip)")
    ap.add_argument("--offload-calls", type=int, default=3, help="timed calls of the offloaded 70B leg (0 = skip)")
    ap.add_argument("--kvpressure-rounds", type=int, default=2,
                    help="timed rounds per sampled context of the 70B KV-pressure leg (0 = skip)")
    ap.add_argument("--parking-rounds", type=int, default=32,
                    help="timed round-robin rounds of the KV parking leg (0 = skip)")
    ap.add_argument("--planner-calls", type=int, default=3,
                    help="timed calls per planner step of the 70B planner leg (0 = skip)")
    ap.add_argument("--resident70b-rounds", type=int, default=8,
                    help="timed decode rounds of the resident 70B leg (0 = skip)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for hardware traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one stage on one GPU; --gpus {args.gpus} is not supported "
              "(the stage does not shard across GPUs).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    import paper_2512_21835_amd as P

    wl = synth.WORKLOADS["llama8b_stage"]
    shape = wl.shape
    dev = torch.device("cuda", 0)
    stream = torch.cuda.Stream(dev)
    torch.cuda.set_stream(stream)
    K, W, T = args.steps, args.warmup, args.prefill
    ctx = T + max(K, W)

    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    t_gen = time.perf_counter()
    weights = [synth.layer_weights(shape, l) for l in range(shape.n_layers)]
    t_gen = time.perf_counter() - t_gen
    cfg = P.config_for(shape, max_microbatches=2, max_batch=1, max_context=ctx, n_resident_max=shape.n_layers,
                       compute_stream=stream.cuda_stream)
    h = P.stage_init(cfg)
    try:
        for l, w in enumerate(weights):
            P.stage_load_layer(h, l, w, 1)
        H = shape.hidden
        # prefill both sequences (mb 0: warmup, mb 1: timed); time the second prefill
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
        P.stage_get_timeline(h)                       # clear
        P.stage_set_timing(h, P.STAGE_TIME_GATEUP)   # HIP events around every gate/up launch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(K):
            P.stage_decode(h, [1], 1, xd[s:s + 1], yd[s:s + 1])
        t_enq = time.perf_counter() - t0
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        P.stage_set_timing(h, 0)
        tl = P.stage_get_timeline(h)
        assert bool(torch.isfinite(yd).all()), "non-finite decode output"
    finally:
        P.stage_destroy(h)

    step_bytes = sum(decode_step_bytes(shape, T + s) for s in range(K)) / K
    traffic = GATEUP_TRAFFIC["bytes"] if GATEUP_TRAFFIC["source_sha256"] == kernel_source_sha256() else None
    kname = "gate/up projection + SwiGLU (gemv, 1 row)"
    gu = [e - s for kind, _, s, e in tl if kind == 2]
    gu_bytes = gateup_bytes(shape, 1)
    gu_ms = sum(gu) / len(gu)
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    ms_step = dt * 1e3 / K
    out = {
        "metric": "decode tokens/s per stage", "value": K / dt, "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"llama8b_stage decode: 8 layers, hidden 4096, 32/8 heads x 128, ffn 14336, "
                               f"bf16 weights resident, bf16 paged KV, batch 1, context {T}->{T + K}",
                   "global_batch": 1, "seq_len": T + K, "parallelism": "none (one stage, one GPU)",
                   "weights": "bf16", "kv_cache": "bf16", "accumulate": "f32"},
        "roofline": {"bound": "hbm", "kernel": kname,
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "bytes_per_launch": gu_bytes, "avg_launch_ms": gu_ms, "launches": len(gu)},
        "step_hbm": {"bytes_per_step": step_bytes, "achieved_GBs": step_bytes / (ms_step * 1e-3) / 1e9,
                     "frac": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "host_enqueue_ms_per_step": t_enq * 1e3 / K,
        "prefill": prefill_report(shape, T, prefill_s),
        "weight_gen_s": t_gen,
    }
    if args.resident70b_rounds > 0:
        out["resident70b"] = resident70b_leg(args.resident70b_rounds)
    if args.kvpressure_rounds > 0:
        out["kvpressure70b"] = kvpressure_leg(rounds=args.kvpressure_rounds)
    if args.parking_rounds > 0:
        out["kv_parking"] = parking_leg(args.parking_rounds)
    if args.planner_calls > 0:
        out["planner"] = planner_leg(args.planner_calls)
    if args.offload_calls > 0:
        out["offload"] = offload_leg(args.offload_calls)
        out["offload_zero_copy"] = offload_leg(args.offload_calls, zero_copy=True)
        if "resident70b" in out:
            out["allocation"] = allocation_report(out["resident70b"], out["offload"])
    if args.cpu_tokens > 0:
        out["cpu_baseline"] = cpu_baseline(shape, lambda l: weights[l], wl, args.cpu_tokens)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
