"""Drives one call sequence through the HIP stage (C ABI) and through the CPU oracle.

Used by the GPU parity tests, bench.py's correctness-free timing helpers do not
use it.  The oracle side never receives a value produced by the GPU: with
feedback decoding, each side feeds back its own outputs.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth

_WEIGHTS: Dict[int, Dict[int, Dict[str, np.ndarray]]] = {}


def weights_of(shape) -> Callable[[int], Dict[str, np.ndarray]]:
    """Cached seeded bf16 weights of a stage shape, generated on first use per layer."""
    cache = _WEIGHTS.setdefault(shape.shape_id, {})

    def get(layer: int):
        if layer not in cache:
            cache[layer] = synth.layer_weights(shape, layer)
            if shape.hidden >= 4096:
                print(f"  [weights] {shape.name} layer {layer} generated", flush=True)
        return cache[layer]
    return get


def _progress(weights, tag: str):
    """Wraps a weights callable so that long oracle passes print one line per layer."""
    def get(layer: int):
        print(f"  [{tag}] layer {layer}", flush=True)
        return weights(layer)
    return get


def drop_weights(shape) -> None:
    _WEIGHTS.pop(shape.shape_id, None)


@dataclass
class Scenario:
    """A call sequence on one stage.

    prefill: tokens per sequence in the (single) prefill of each micro-batch.
    decode_steps: decode rounds; each round visits every micro-batch.
    calls: "one" = one micro-batch per call, round-robin (the interleaved pipeline's order);
           "all" = one call carrying every micro-batch.
    """
    wl: synth.Workload
    prefill: int
    decode_steps: int
    calls: str = "one"
    kv_fp32: bool = False
    n_resident: Optional[int] = None
    slots: int = 2
    thresholds: Tuple[int, ...] = ()
    max_context: Optional[int] = None
    timing: int = 0
    zero_copy: bool = False
    residency: Optional[Tuple[int, ...]] = None   # per-layer STAGE_RES_* codes (block granularity)
    plan: Optional[Tuple[Tuple[int, int, int], ...]] = None   # planner steps (tokens, alpha, beta)
    slot_check: int = 0   # stage_config.slot_check

    @property
    def shape(self):
        return self.wl.shape

    def resident_layers(self) -> int:
        """The weight budget in layers: enough for every block the scenario keeps resident."""
        if self.residency is not None:
            return sum(1 for c in self.residency if c != 0)
        return self.shape.n_layers if self.n_resident is None else self.n_resident

    def codes(self) -> List[int]:
        if self.residency is not None:
            return list(self.residency)
        r = self.resident_layers()
        return [1 if l < r else 0 for l in range(self.shape.n_layers)]

    def ctx(self) -> int:
        return self.max_context or (self.prefill + self.decode_steps)

    def call_plan(self) -> List[Tuple[str, List[int], int]]:
        """[(kind, mb_ids, step)] in call order; step = decode step index (-1 for prefill)."""
        mbs = list(range(self.wl.n_mb))
        groups = [[m] for m in mbs] if self.calls == "one" else [mbs]
        plan = [("prefill", g, -1) for g in groups]
        for s in range(self.decode_steps):
            plan += [("decode", g, s) for g in groups]
        return plan


@dataclass
class RunResult:
    outputs: List[np.ndarray] = field(default_factory=list)   # per call [n_mb, B, T, H]
    layer_rows: list = field(default_factory=list)             # oracle only, see run_oracle
    inputs: List[np.ndarray] = field(default_factory=list)
    block_tables: Dict[Tuple[int, int], List[int]] = field(default_factory=dict)
    slot_log: List[Tuple[int, int, int]] = field(default_factory=list)
    demotion_log: List[Tuple[int, int]] = field(default_factory=list)
    residency_log: List[Tuple[int, int, int]] = field(default_factory=list)
    residency: List[int] = field(default_factory=list)
    stats: dict = field(default_factory=dict)
    timeline: list = field(default_factory=list)

    def flat_out(self) -> np.ndarray:
        return np.concatenate([o.reshape(-1, o.shape[-1]) for o in self.outputs])

    def flat_in(self) -> np.ndarray:
        return np.concatenate([o.reshape(-1, o.shape[-1]) for o in self.inputs])


def _inputs(sc: Scenario, kind: str, mbs: Sequence[int], step: int, prev: Dict) -> np.ndarray:
    wl, B, H = sc.wl, sc.wl.batch, sc.shape.hidden
    if kind == "prefill":
        return np.stack([np.stack([synth.prefill_inputs(wl, m, b, sc.prefill) for b in range(B)]) for m in mbs])
    if wl.feedback:
        return np.stack([np.stack([prev[(m, b)] for b in range(B)]) for m in mbs])[:, :, None, :]
    return np.stack([np.stack([synth.decode_input(wl, m, b, step) for b in range(B)]) for m in mbs])[:, :, None, :]


class compute_stream:
    """Context: a fresh (default-priority) torch stream made current, shared with the library.

    torch's default stream has handle 0, which the C ABI reads as "create your own"; running
    torch's copies and the stage's kernels on one explicit stream keeps them ordered.
    """

    def __init__(self, device: int = 0):
        import torch
        self.torch = torch
        self.stream = torch.cuda.Stream(torch.device("cuda", device))
        self.ctx = torch.cuda.stream(self.stream)

    @property
    def handle(self):
        return self.stream.cuda_stream

    def __enter__(self):
        self.ctx.__enter__()
        return self

    def __exit__(self, *exc):
        self.stream.synchronize()
        return self.ctx.__exit__(*exc)


def run_gpu(sc: Scenario, device: int = 0, weights=None, feed=None) -> RunResult:
    """The stage's outputs for the scenario's call plan.  ``feed(kind, mbs, T)``, if given, supplies
    each call's input [len(mbs), B, T, H] instead of the workload's seeded inputs."""
    with compute_stream(device) as cs:
        return _run_gpu(sc, device, weights, cs.handle, feed)


def _run_gpu(sc: Scenario, device: int, weights, cs_handle, feed=None) -> RunResult:
    import torch
    import paper_2512_21835_amd as P

    shape, wl = sc.shape, sc.wl
    weights = weights or weights_of(shape)
    dev = torch.device("cuda", device)
    # copy_stream None: the library's own copy stream, on a hardware queue of its own
    cfg = P.config_for(shape, max_microbatches=wl.n_mb, max_batch=wl.batch, max_context=sc.ctx(),
                       n_resident_max=sc.resident_layers(), n_stream_slots=sc.slots, kv_fp32=sc.kv_fp32,
                       thresholds=sc.thresholds, device=device, compute_stream=cs_handle,
                       copy_stream=None, timing=sc.timing, zero_copy=sc.zero_copy,
                       plan=sc.plan, slot_check=sc.slot_check)
    h = P.stage_init(cfg)
    res = RunResult()
    try:
        for l, code in enumerate(sc.codes()):
            P.stage_load_layer(h, l, weights(l), code)
        prev: Dict[Tuple[int, int], np.ndarray] = {}
        outs = []
        for kind, mbs, step in sc.call_plan():
            if feed is not None:
                x = feed(kind, mbs, sc.prefill if kind == "prefill" else 1)
            else:
                x = _inputs(sc, kind, mbs, step, prev)
            x_in = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)
            x_out = torch.empty_like(x_in)
            if kind == "prefill":
                P.stage_prefill(h, mbs, wl.batch, x.shape[2], x_in, x_out)
            else:
                P.stage_decode(h, mbs, wl.batch, x_in, x_out)
            outs.append(x_out)
            res.inputs.append(x)
            if wl.feedback:
                o = x_out.cpu().numpy()
                for i, m in enumerate(mbs):
                    for b in range(wl.batch):
                        prev[(m, b)] = o[i, b, -1]
        P.stage_sync(h)
        res.outputs = [o.cpu().numpy() for o in outs]
        for m in range(wl.n_mb):
            for b in range(wl.batch):
                res.block_tables[(m, b)] = P.stage_get_block_table(h, m, b)
        res.slot_log = P.stage_get_slot_log(h)
        res.demotion_log = P.stage_get_demotion_log(h)
        res.residency_log = P.stage_get_residency_log(h)
        res.residency = P.stage_get_residency(h, shape.n_layers)
        res.stats = P.stage_get_stats(h)
        if sc.timing:
            res.timeline = P.stage_get_timeline(h)
    finally:
        P.stage_destroy(h)
    return res


def run_oracle(sc: Scenario, weights=None, floats: bool = True, kv_jitter: float = 0.0,
               trace: bool = False) -> RunResult:
    """The oracle's outputs (floats=True) and its integer policies for the call sequence.

    With ``trace`` (workloads without feedback), ``res.layer_rows[l][(m, b)]`` holds the rows that
    entered layer l for sequence (m, b), in call order; entry n_layers holds the stage outputs."""
    from oracle.policies import BlockAllocator, ResidencySchedule, SlotSchedule
    from oracle.stage_oracle import OracleStage

    shape, wl = sc.shape, sc.wl
    weights = weights or weights_of(shape)
    if shape.hidden >= 4096:
        weights = _progress(weights, "oracle")
    orc = OracleStage(shape, weights, kv_dtype="f32" if sc.kv_fp32 else "bf16", kv_jitter=kv_jitter, jitter_seed=1)
    n_blocks = wl.n_mb * wl.batch * math.ceil(sc.ctx() / 16)
    alloc = BlockAllocator(n_blocks, 16)
    slots = SlotSchedule(sc.slots)
    resid = ResidencySchedule(shape.n_layers, thresholds=sc.thresholds, codes=sc.codes(), plan=sc.plan)
    res = RunResult()
    prev: Dict[Tuple[int, int], np.ndarray] = {}
    # Without feedback every call's inputs are known up front, so the oracle runs once over each
    # sequence's rows in call order (a decode step equals the matching row of one causal pass)
    # instead of widening every layer's weights again for every call.
    batched = floats and not wl.feedback
    calls = []
    for call_no, (kind, mbs, step) in enumerate(sc.call_plan()):
        x = _inputs(sc, kind, mbs, step, prev)
        T = x.shape[2]
        keys = [(m, b) for m in mbs for b in range(wl.batch)]
        longest = max([alloc.lengths.get(k, 0) for k in alloc.lengths] + [alloc.lengths.get(k, 0) + T for k in keys])
        if sc.plan is not None:
            resid.before_call_planned(call_no, sum(alloc.lengths.values()) + T * len(keys))
        else:
            resid.before_call(call_no, longest)
        alloc.call([(k, T) for k in keys])
        # zero-copy access (Section III-C): a call with one token per sequence reads offloaded
        # layers where they are, in host memory, so it stages nothing through the slots
        slots.call(call_no, [] if (sc.zero_copy and T == 1) else resid.streamed())
        if not floats:
            continue
        res.inputs.append(x)
        if batched:
            calls.append((mbs, x))
            continue
        outs = orc.forward([((m, b), x[i, b]) for i, m in enumerate(mbs) for b in range(wl.batch)])
        o = np.stack(outs).reshape(x.shape)
        res.outputs.append(o)
        if wl.feedback:
            for i, m in enumerate(mbs):
                for b in range(wl.batch):
                    prev[(m, b)] = o[i, b, -1].astype(np.float32)
    if batched:
        rows: Dict[Tuple[int, int], list] = {}
        for mbs, x in calls:
            for i, m in enumerate(mbs):
                for b in range(wl.batch):
                    rows.setdefault((m, b), []).append(x[i, b])
        keys = sorted(rows)
        tr = [] if trace else None
        outs = orc.forward([(k, np.concatenate(rows[k])) for k in keys], trace=tr)
        if trace:
            res.layer_rows = [dict(zip(keys, layer)) for layer in tr] + [dict(zip(keys, outs))]
        done = {k: 0 for k in keys}
        by_key = dict(zip(keys, outs))
        for mbs, x in calls:
            o = np.empty(x.shape, dtype=np.float64)
            for i, m in enumerate(mbs):
                for b in range(wl.batch):
                    t0 = done[(m, b)]
                    o[i, b] = by_key[(m, b)][t0: t0 + x.shape[2]]
                    done[(m, b)] = t0 + x.shape[2]
            res.outputs.append(o)
    for m in range(wl.n_mb):
        for b in range(wl.batch):
            res.block_tables[(m, b)] = alloc.table((m, b))
    res.slot_log = list(slots.log)
    res.demotion_log = list(resid.log)
    res.residency_log = list(resid.changes)
    res.residency = list(resid.codes)
    res._oracle = orc
    return res


def teacher_forced(sc: Scenario, ref: RunResult, weights=None, runner=None) -> List[dict]:
    """Per-layer teacher forcing: layer l runs on the GPU alone (a one-layer stage holding layer l's
    weights), through the scenario's call plan, fed the rows that entered layer l in the oracle
    (rounded to fp32, the stage's input type), and its outputs are compared with the rows that
    entered layer l + 1 there.  Each layer's K/V cache is then built from the same inputs on both
    sides, so K/V rounding flips stay inside the layer instead of compounding through the stage.
    ``ref`` comes from run_oracle(sc, trace=True).  ``runner(sc, weights, feed)`` runs the one-layer
    stage (default: the GPU through run_gpu).  Returns one compare() dict per layer."""
    shape = sc.shape
    weights = weights or weights_of(shape)
    one = dataclasses.replace(shape, n_layers=1)
    sc1 = dataclasses.replace(sc, wl=dataclasses.replace(sc.wl, shape=one, resident=None, thresholds=()),
                              n_resident=None, thresholds=())
    results = []
    for layer in range(shape.n_layers):
        rows_in, rows_out = ref.layer_rows[layer], ref.layer_rows[layer + 1]
        taken = {k: 0 for k in rows_in}

        def feed(kind, mbs, T):
            x = np.empty((len(mbs), sc.wl.batch, T, shape.hidden), dtype=np.float32)
            for i, m in enumerate(mbs):
                for b in range(sc.wl.batch):
                    t0 = taken[(m, b)]
                    x[i, b] = rows_in[(m, b)][t0: t0 + T]
                    taken[(m, b)] = t0 + T
            return x
        run = runner or (lambda s1, w, f: run_gpu(s1, weights=w, feed=f))
        got = run(sc1, lambda _l, _w=weights(layer): _w, feed)
        # oracle rows of the same calls, in the same order
        done = {k: 0 for k in rows_out}
        want, given = [], []
        for (kind, mbs, _), x in zip(sc.call_plan(), got.inputs):
            T = x.shape[2]
            for i, m in enumerate(mbs):
                for b in range(sc.wl.batch):
                    t0 = done[(m, b)]
                    want.append(rows_out[(m, b)][t0: t0 + T])
                    given.append(rows_in[(m, b)][t0: t0 + T])
                    done[(m, b)] = t0 + T
        results.append(compare(got.flat_out(), np.concatenate(want), got.flat_in(), np.concatenate(given)))
    return results


# Relative accuracy of the GPU arithmetic up to the KV store: the prefill projections take the fp32
# activation as a bf16 hi + lo pair, whose residual is below 2^-17 relative.
KV_JITTER = 2.0 ** -16


def bf16_kv_tolerance(sc: Scenario, ref: RunResult, base: float = 2e-2) -> tuple:
    """Tolerance of the stage output with a bf16 KV cache.

    K and V are rounded to bf16 at store; wherever two correct arithmetics (the GPU's fp32 and the
    oracle's float64) straddle a rounding boundary they store neighbouring bf16 values, and the
    flips compound through the layers.  The spread this allows is measured on the oracle alone:
    the same stage with its pre-rounding K/V jittered by KV_JITTER (relative).  Tolerance = base
    + 2 x spread.  Returns (tolerance, spread).
    """
    jit = run_oracle(sc, kv_jitter=KV_JITTER)
    spread = float(np.abs(jit.flat_out() - ref.flat_out()).max())
    return base + 2.0 * spread, spread


def compare(got: np.ndarray, ref: np.ndarray, x_got: np.ndarray, x_ref: np.ndarray) -> dict:
    """max |d|, cosine of the outputs and cosine of the stage contribution out - in."""
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    dg = g - x_got.astype(np.float64)
    dr = r - x_ref.astype(np.float64)

    def cos(a, b):
        return float((a * b).sum() / math.sqrt((a * a).sum() * (b * b).sum()))
    d = np.abs(g - r)
    worst = int(np.argmax(d))
    row, col = divmod(worst, g.shape[-1]) if g.ndim > 1 else (0, worst)
    return {"max_abs": float(d.flat[worst]), "cos": cos(g, r), "cos_delta": cos(dg, dr),
            "rms_ref": float(np.sqrt((r * r).mean())), "n": int(g.size), "worst_row": row, "worst_col": col,
            "worst_ref": float(r.flat[worst])}


def row_origin(sc: Scenario, row: int) -> Tuple[int, str, int, int, int]:
    """Where flat output row `row` of a run of the scenario comes from: (call index, kind, mb, b,
    position in the sequence); rows are in call order, each call's rows [mb][b][t]."""
    pos: Dict[Tuple[int, int], int] = {}
    for call, (kind, mbs, _) in enumerate(sc.call_plan()):
        T = sc.prefill if kind == "prefill" else 1
        n = len(mbs) * sc.wl.batch * T
        if row < n:
            i, rest = divmod(row, sc.wl.batch * T)
            b, t = divmod(rest, T)
            return call, kind, mbs[i], b, pos.get((mbs[i], b), 0) + t
        row -= n
        for m in mbs:
            for b in range(sc.wl.batch):
                pos[(m, b)] = pos.get((m, b), 0) + T
    raise IndexError("row beyond the scenario's calls")


def overlap_of_last_call(timeline) -> dict:
    """Copy/compute overlap of the last call in a stage timeline (records kind, layer, start, end):
    the union of slot copies (kinds 1, 4) and of layer kernels (kinds 3, 5) of that call, their
    intersection, hidden-copy = |copy & compute| / |copy| and hidden-shorter = |copy & compute| /
    min(|copy|, |compute|)."""
    def union(iv):
        out = []
        for s, e in sorted(iv):
            if out and s <= out[-1][1]:
                out[-1][1] = max(out[-1][1], e)
            else:
                out.append([s, e])
        return out

    def inter(a, b):
        i = j = 0
        tot = 0.0
        while i < len(a) and j < len(b):
            tot += max(0.0, min(a[i][1], b[j][1]) - max(a[i][0], b[j][0]))
            if a[i][1] < b[j][1]:
                i += 1
            else:
                j += 1
        return tot

    ends = [i for i, r in enumerate(timeline) if r[0] == 0]
    seg = timeline[ends[-2] + 1: ends[-1] + 1] if len(ends) > 1 else timeline[: ends[-1] + 1]
    copies = union([(a, b) for k, _, a, b in seg if k in (1, 4)])
    comp = union([(a, b) for k, _, a, b in seg if k in (3, 5)])
    t_copy = sum(e - s for s, e in copies)
    t_comp = sum(e - s for s, e in comp)
    both = inter(copies, comp)
    return {"copy_ms": t_copy, "compute_ms": t_comp, "hidden_copy": both / t_copy,
            "hidden_shorter": both / min(t_copy, t_comp)}
