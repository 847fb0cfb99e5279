"""ctypes binding of libstage.so: the same entry points as include/stage.h.

Argument marshalling only -- every step of the stage forward runs in the HIP
kernels behind the C ABI.  There is no fallback: if libstage.so is missing the
import fails with the command that builds it.

torch is imported first on purpose: it loads the process's HIP runtime
(libamdhip64.so.7), which libstage.so then binds to, so torch tensors, torch
streams and the library share one runtime.
"""
from __future__ import annotations

import ctypes
import json
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_void_p
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch  # noqa: F401  (must precede loading libstage.so)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstage.so")

STAGE_OK, STAGE_EINVAL, STAGE_ENOMEM, STAGE_EHIP, STAGE_ESTATE, STAGE_ERANGE, STAGE_ESLOT = 0, -1, -2, -3, -4, -5, -6
STAGE_MAX_THRESHOLDS = 32
STAGE_MAX_SEQS_PER_CALL = 64
STAGE_MAX_CONTEXT = 16384
STAGE_MAX_LANES = 4
STAGE_TIME_CALLS = 1
STAGE_TIME_GATEUP = 2
STAGE_TIME_LAYERS = 4
STAGE_RES_OFFLOADED, STAGE_RES_RESIDENT, STAGE_RES_MHA_OFFLOADED, STAGE_RES_MLP_OFFLOADED = 0, 1, 2, 3

EXPORTED = (
    "stage_config_default", "stage_init", "stage_destroy", "stage_load_layer", "stage_prefill",
    "stage_decode", "stage_decode_lane", "stage_prefill_lane", "stage_kv_append", "stage_kv_export_tail", "stage_reset_sequence", "stage_sync",
    "stage_get_block_table", "stage_get_length", "stage_get_residency", "stage_get_slot_log",
    "stage_get_demotion_log", "stage_get_residency_log", "stage_get_timeline", "stage_set_timing", "stage_get_stats",
    "stage_last_error", "stage_strerror", "stage_plan_offload", "stage_allocate", "stage_kv_park", "stage_kv_unpark",
    "stage_decode_noalloc",
)
STAGE_NOALLOC_SCRATCH_BYTES = 67108864
STAGE_ALLOC_MAX_DEVICES = 64
STAGE_ALLOC_MAX_LAYERS = 4096


class StageConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", c_int32), ("hidden", c_int32), ("n_q_heads", c_int32), ("n_kv_heads", c_int32),
        ("head_dim", c_int32), ("ffn", c_int32),
        ("rope_theta", c_float), ("rms_eps", c_float),
        ("max_microbatches", c_int32), ("max_batch", c_int32), ("max_context", c_int32),
        ("kv_block_tokens", c_int32), ("kv_pool_blocks", c_int32), ("kv_fp32", c_int32),
        ("n_resident_max", c_int32), ("n_stream_slots", c_int32),
        ("n_thresholds", c_int32), ("thresholds", c_int32 * STAGE_MAX_THRESHOLDS),
        ("device", c_int32), ("compute_stream", c_void_p), ("copy_stream", c_void_p),
        ("timing", c_int32), ("zero_copy", c_int32),
        ("plan_mode", c_int32), ("plan_alpha", c_int32 * STAGE_MAX_THRESHOLDS),
        ("plan_beta", c_int32 * STAGE_MAX_THRESHOLDS), ("kv_park_tokens", c_int32),
        ("n_lanes", c_int32), ("lane_streams", c_void_p * STAGE_MAX_LANES),
        ("slot_check", c_int32),
    ]


class StagePlanInput(ctypes.Structure):
    """stage_plan_input of include/stage_planner.h."""
    _fields_ = [
        ("mem_left", c_int64), ("kv_bytes_per_token", c_int64), ("mha_bytes", c_int64), ("mlp_bytes", c_int64),
        ("mha_cost", c_int64), ("mlp_cost", c_int64),
        ("mha_free", c_int32), ("mlp_free", c_int32), ("n_stage", c_int32),
    ]


class StagePlanStep(ctypes.Structure):
    _fields_ = [("tokens", c_int64), ("alpha", c_int32), ("beta", c_int32)]


class StageAllocDevice(ctypes.Structure):
    """stage_alloc_device of include/stage_alloc.h."""
    _fields_ = [("mem_bytes", c_int64), ("comp_layer", c_int64), ("load_mha", c_int64), ("load_mlp", c_int64)]


class StageAllocInput(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("mha_bytes", c_int64), ("mlp_bytes", c_int64), ("comm", c_int64),
                ("n_devices", c_int32), ("devices", POINTER(StageAllocDevice))]


class StageAllocPlan(ctypes.Structure):
    _fields_ = [("first_layer", c_int32), ("assigned", c_int32), ("offloaded", c_int32), ("mha_only", c_int32),
                ("mlp_only", c_int32)]


class StageLayerWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g1", "g2")]


class StageError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (status {code})")
        self.code = code


_LIB = None


def lib():
    """The loaded libstage.so; raises if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2512_21835_amd.build` "
                          "(or __graft_entry__.build()); there is no CPU fallback")
    L = ctypes.CDLL(LIB_PATH)
    ip = POINTER(c_int32)
    sig = {
        "stage_config_default": (None, [POINTER(StageConfig)]),
        "stage_init": (c_int32, [POINTER(StageConfig), POINTER(c_void_p)]),
        "stage_destroy": (c_int32, [c_void_p]),
        "stage_load_layer": (c_int32, [c_void_p, c_int32, POINTER(StageLayerWeights), c_int32]),
        "stage_prefill": (c_int32, [c_void_p, c_int32, ip, c_int32, c_int32, c_void_p, c_void_p]),
        "stage_decode": (c_int32, [c_void_p, c_int32, ip, c_int32, c_void_p, c_void_p]),
        "stage_decode_lane": (c_int32, [c_void_p, c_int32, c_int32, ip, c_int32, c_void_p, c_void_p]),
        "stage_decode_noalloc": (c_int32, [c_void_p, c_int32, ip, c_int32, c_void_p, c_void_p]),
        "stage_prefill_lane": (c_int32, [c_void_p, c_int32, c_int32, ip, c_int32, c_int32, c_void_p, c_void_p]),
        "stage_kv_append": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p]),
        "stage_kv_export_tail": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_int32]),
        "stage_reset_sequence": (c_int32, [c_void_p, c_int32, c_int32]),
        "stage_kv_park": (c_int32, [c_void_p, c_int32, ip, c_int32]),
        "stage_kv_unpark": (c_int32, [c_void_p, c_int32, ip]),
        "stage_sync": (c_int32, [c_void_p]),
        "stage_get_block_table": (c_int32, [c_void_p, c_int32, c_int32, ip, c_int32, ip]),
        "stage_get_length": (c_int32, [c_void_p, c_int32, c_int32, ip]),
        "stage_get_residency": (c_int32, [c_void_p, ip]),
        "stage_get_slot_log": (c_int32, [c_void_p, ip, c_int32, ip]),
        "stage_get_demotion_log": (c_int32, [c_void_p, ip, c_int32, ip]),
        "stage_get_residency_log": (c_int32, [c_void_p, ip, c_int32, ip]),
        "stage_plan_offload": (c_int32, [POINTER(StagePlanInput), POINTER(StagePlanStep), c_int32, ip,
                                         POINTER(c_int64)]),
        "stage_allocate": (c_int32, [POINTER(StageAllocInput), POINTER(StageAllocPlan), ip, POINTER(c_int64)]),
        "stage_get_timeline": (c_int32, [c_void_p, POINTER(c_float), c_int32, ip]),
        "stage_set_timing": (c_int32, [c_void_p, c_int32]),
        "stage_get_stats": (c_int32, [c_void_p, c_char_p, c_int32]),
        "stage_last_error": (c_char_p, [c_void_p]),
        "stage_strerror": (c_char_p, [c_int32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _LIB = L
    return L


def _check(rc: int, h=None) -> None:
    if rc != STAGE_OK:
        msg = lib().stage_strerror(rc).decode()
        if h is not None:
            detail = lib().stage_last_error(h).decode()
            if detail:
                msg = f"{msg}: {detail}"
        raise StageError(rc, msg)


def _ptr(x) -> int:
    """Address of a torch tensor or numpy array (contiguous)."""
    if isinstance(x, torch.Tensor):
        if not x.is_contiguous():
            raise ValueError("tensor must be contiguous")
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("array must be C-contiguous")
        return x.ctypes.data
    raise TypeError(f"expected a torch tensor or numpy array, got {type(x)}")


def _ids(mb_ids: Sequence[int]):
    arr = (c_int32 * len(mb_ids))(*[int(m) for m in mb_ids])
    return arr


# ---------------------------------------------------------------------------- entry points
def stage_config_default() -> StageConfig:
    cfg = StageConfig()
    lib().stage_config_default(ctypes.byref(cfg))
    return cfg


def stage_init(cfg: StageConfig) -> c_void_p:
    h = c_void_p()
    _check(lib().stage_init(ctypes.byref(cfg), ctypes.byref(h)))
    return h


def stage_destroy(h) -> None:
    _check(lib().stage_destroy(h))


def stage_load_layer(h, layer: int, weights: Optional[Dict[str, object]], resident: int) -> None:
    """weights: name -> bf16 bits (numpy uint16 or torch int16/bfloat16, host or device), or None."""
    if weights is None:
        _check(lib().stage_load_layer(h, layer, None, int(resident)), h)
        return
    w = StageLayerWeights(*[_ptr(weights[n]) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g1", "g2")])
    _check(lib().stage_load_layer(h, layer, ctypes.byref(w), int(resident)), h)


def stage_prefill(h, mb_ids: Sequence[int], B: int, T: int, x_in: torch.Tensor, x_out: torch.Tensor) -> None:
    _check(lib().stage_prefill(h, len(mb_ids), _ids(mb_ids), B, T, _ptr(x_in), _ptr(x_out)), h)


def stage_decode(h, mb_ids: Sequence[int], B: int, x_in: torch.Tensor, x_out: torch.Tensor) -> None:
    _check(lib().stage_decode(h, len(mb_ids), _ids(mb_ids), B, _ptr(x_in), _ptr(x_out)), h)


def stage_decode_noalloc(h, mb_ids: Sequence[int], B: int, x_in: torch.Tensor, x_out: torch.Tensor) -> None:
    _check(lib().stage_decode_noalloc(h, len(mb_ids), _ids(mb_ids), B, _ptr(x_in), _ptr(x_out)), h)


def stage_decode_lane(h, lane: int, mb_ids: Sequence[int], B: int, x_in: torch.Tensor, x_out: torch.Tensor) -> None:
    _check(lib().stage_decode_lane(h, lane, len(mb_ids), _ids(mb_ids), B, _ptr(x_in), _ptr(x_out)), h)


def stage_prefill_lane(h, lane: int, mb_ids: Sequence[int], B: int, T: int, x_in: torch.Tensor,
                       x_out: torch.Tensor) -> None:
    _check(lib().stage_prefill_lane(h, lane, len(mb_ids), _ids(mb_ids), B, T, _ptr(x_in), _ptr(x_out)), h)


def stage_kv_append(h, mb: int, b: int, n_tokens: int, k, v) -> None:
    _check(lib().stage_kv_append(h, mb, b, n_tokens, _ptr(k), _ptr(v)), h)


def stage_kv_export_tail(h, mb: int, b: int, n_tokens: int, k, v, drop: bool) -> None:
    _check(lib().stage_kv_export_tail(h, mb, b, n_tokens, _ptr(k), _ptr(v), int(bool(drop))), h)


def stage_reset_sequence(h, mb: int, b: int) -> None:
    _check(lib().stage_reset_sequence(h, mb, b), h)


def stage_kv_park(h, mb_ids: Sequence[int], n_tokens: int) -> None:
    _check(lib().stage_kv_park(h, len(mb_ids), _ids(mb_ids), n_tokens), h)


def stage_kv_unpark(h, mb_ids: Sequence[int]) -> None:
    _check(lib().stage_kv_unpark(h, len(mb_ids), _ids(mb_ids)), h)


def stage_sync(h) -> None:
    _check(lib().stage_sync(h), h)


def stage_get_block_table(h, mb: int, b: int) -> List[int]:
    n = c_int32()
    _check(lib().stage_get_block_table(h, mb, b, None, 0, ctypes.byref(n)), h)
    buf = (c_int32 * max(1, n.value))()
    _check(lib().stage_get_block_table(h, mb, b, buf, n.value, ctypes.byref(n)), h)
    return list(buf[: n.value])


def stage_get_length(h, mb: int, b: int) -> int:
    n = c_int32()
    _check(lib().stage_get_length(h, mb, b, ctypes.byref(n)), h)
    return n.value


def stage_get_residency(h, n_layers: int) -> List[int]:
    buf = (c_int32 * n_layers)()
    _check(lib().stage_get_residency(h, buf), h)
    return list(buf)


def _log(fn, h, width: int) -> List[Tuple[int, ...]]:
    n = c_int32()
    _check(fn(h, None, 0, ctypes.byref(n)), h)
    buf = (c_int32 * max(1, n.value * width))()
    _check(fn(h, buf, n.value, ctypes.byref(n)), h)
    return [tuple(buf[i * width:(i + 1) * width]) for i in range(n.value)]


def stage_get_slot_log(h) -> List[Tuple[int, int, int]]:
    return _log(lib().stage_get_slot_log, h, 3)


def stage_get_demotion_log(h) -> List[Tuple[int, int]]:
    return _log(lib().stage_get_demotion_log, h, 2)


def stage_get_residency_log(h) -> List[Tuple[int, int, int]]:
    return _log(lib().stage_get_residency_log, h, 3)


def stage_plan_offload(mem_left: int, kv_bytes_per_token: int, mha_bytes: int, mlp_bytes: int, mha_cost: int,
                       mlp_cost: int, mha_free: int, mlp_free: int, n_stage: int
                       ) -> Tuple[List[Tuple[int, int, int]], int]:
    """The online planner's steps [(tokens, alpha, beta)] and the capacity in tokens."""
    inp = StagePlanInput(mem_left, kv_bytes_per_token, mha_bytes, mlp_bytes, mha_cost, mlp_cost, mha_free, mlp_free,
                         n_stage)
    n, capacity = c_int32(), c_int64()
    _check(lib().stage_plan_offload(ctypes.byref(inp), None, 0, ctypes.byref(n), ctypes.byref(capacity)))
    buf = (StagePlanStep * max(1, n.value))()
    _check(lib().stage_plan_offload(ctypes.byref(inp), buf, n.value, ctypes.byref(n), ctypes.byref(capacity)))
    return [(buf[i].tokens, buf[i].alpha, buf[i].beta) for i in range(n.value)], capacity.value


def stage_allocate(n_layers: int, mha_bytes: int, mlp_bytes: int, comm: int,
                   devices: Sequence[Tuple[int, int, int, int]]) -> Tuple[int, int, List[Tuple[int, ...]]]:
    """Alg. 1: (#Stage, T_total, [(first_layer, assigned, offloaded, mha_only, mlp_only)] per
    device); devices are (mem_bytes, comp_layer, load_mha, load_mlp)."""
    devs = (StageAllocDevice * len(devices))(*[StageAllocDevice(*d) for d in devices])
    inp = StageAllocInput(n_layers, mha_bytes, mlp_bytes, comm, len(devices), devs)
    out = (StageAllocPlan * len(devices))()
    n_stage, t = c_int32(), c_int64()
    _check(lib().stage_allocate(ctypes.byref(inp), out, ctypes.byref(n_stage), ctypes.byref(t)))
    return n_stage.value, t.value, [(o.first_layer, o.assigned, o.offloaded, o.mha_only, o.mlp_only) for o in out]


def stage_get_timeline(h) -> List[Tuple[int, int, float, float]]:
    n = c_int32()
    cap = 1 << 16
    buf = (c_float * (4 * cap))()
    _check(lib().stage_get_timeline(h, buf, cap, ctypes.byref(n)), h)
    return [(int(buf[4 * i]), int(buf[4 * i + 1]), buf[4 * i + 2], buf[4 * i + 3]) for i in range(min(cap, n.value))]


def stage_set_timing(h, flags: int) -> None:
    _check(lib().stage_set_timing(h, flags), h)


def stage_get_stats(h) -> dict:
    buf = ctypes.create_string_buffer(4096)
    _check(lib().stage_get_stats(h, buf, 4096), h)
    return json.loads(buf.value.decode())


def stage_strerror(code: int) -> str:
    return lib().stage_strerror(code).decode()


# ---------------------------------------------------------------------------- helpers
def config_for(shape, *, max_microbatches: int, max_batch: int, max_context: int, n_resident_max: int,
               n_stream_slots: int = 2, kv_fp32: bool = False, thresholds: Sequence[int] = (),
               kv_pool_blocks: int = 0, device: int = 0, compute_stream=None, copy_stream=None,
               timing: int = 0, zero_copy: bool = False,
               plan: Optional[Sequence[Tuple[int, int, int]]] = None, kv_park_tokens: int = 0,
               n_lanes: int = 1, lane_streams: Optional[Sequence] = None, slot_check: int = 0) -> StageConfig:
    """A StageConfig for a stage shape (any object with the StageShape fields).  ``plan``:
    planner steps [(tokens, alpha, beta)] (plan_mode 1), instead of ``thresholds``.
    ``n_lanes`` decode lanes; ``lane_streams[l]``: lane l's stream handle (None: the library's).
    ``slot_check``: the slot tag check mode (0 off, 1 on, 2 self-test)."""
    cfg = stage_config_default()
    cfg.n_layers, cfg.hidden = shape.n_layers, shape.hidden
    cfg.n_q_heads, cfg.n_kv_heads = shape.n_q_heads, shape.n_kv_heads
    cfg.head_dim, cfg.ffn = shape.head_dim, shape.ffn
    cfg.rope_theta, cfg.rms_eps = shape.rope_theta, shape.rms_eps
    cfg.max_microbatches, cfg.max_batch, cfg.max_context = max_microbatches, max_batch, max_context
    cfg.kv_pool_blocks = kv_pool_blocks
    cfg.kv_fp32 = int(bool(kv_fp32))
    cfg.n_resident_max, cfg.n_stream_slots = n_resident_max, n_stream_slots
    if plan is not None:
        if thresholds:
            raise ValueError("give thresholds or a plan, not both")
        cfg.plan_mode = 1
        thresholds = [t for t, _, _ in plan]
        for i, (_, a, b) in enumerate(plan[:STAGE_MAX_THRESHOLDS]):
            cfg.plan_alpha[i], cfg.plan_beta[i] = int(a), int(b)
    if len(thresholds) > STAGE_MAX_THRESHOLDS:
        raise ValueError("too many thresholds")
    cfg.n_thresholds = len(thresholds)
    for i, t in enumerate(thresholds):
        cfg.thresholds[i] = int(t)
    cfg.device = device
    cfg.compute_stream = compute_stream
    cfg.copy_stream = copy_stream
    cfg.timing = timing
    cfg.zero_copy = int(bool(zero_copy))
    cfg.kv_park_tokens = kv_park_tokens
    cfg.n_lanes = n_lanes
    for l, st in enumerate(lane_streams or ()):
        cfg.lane_streams[l] = st
    cfg.slot_check = slot_check
    return cfg
