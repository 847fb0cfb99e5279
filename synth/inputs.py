"""Stage shapes, workloads and seeded generators (no decoder arithmetic here).

Seeds
-----
* Weights of layer ``l`` of a stage shape: ``seed_of(0x57, shape_id, l, tensor_id)``
  with tensor ids wq=0, wk=1, wv=2, wo=3, wg=4, wu=5, wd=6, g1=7, g2=8.  Seeding by
  stage shape (not by workload) lets the three 70B-shaped workloads share one
  weight set, as "the same 70B-shaped 16-layer stage".
* Prefill hidden states of sequence (mb, b): ``seed_of(0xA1, workload_id, 0, mb, b, 0)``,
  a stream of T*H values in row-major [T, H] order.
* Decode hidden state of sequence (mb, b) at decode step s:
  ``seed_of(0xA1, workload_id, 1, mb, b, s)``, H values.

The generator itself (SplitMix64 + Box-Muller) is defined in ``gen.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_MASK = (1 << 64) - 1

TENSOR_IDS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "wg": 4, "wu": 5, "wd": 6, "g1": 7, "g2": 8}


@dataclass(frozen=True)
class StageShape:
    """Shape of one pipeline stage: a contiguous block of LLaMA-style decoder layers."""
    name: str
    shape_id: int
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rope_theta: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_params(self) -> int:
        h = self.hidden
        return (self.q_dim + 2 * self.kv_dim) * h + h * self.q_dim + 3 * self.ffn * h + 2 * h

    def layer_bytes(self) -> int:
        return 2 * self.layer_params()

    def kv_bytes_per_token_layer(self, elem_bytes: int = 2) -> int:
        return 2 * self.kv_dim * elem_bytes


TINY = StageShape("tiny-2L-h256", 0, 2, 256, 4, 2, 64, 688)
LLAMA8B_STAGE = StageShape("llama3-8b-shaped-8L", 1, 8, 4096, 32, 8, 128, 14336)
LLAMA70B_STAGE = StageShape("llama3.3-70b-shaped-16L", 2, 16, 8192, 64, 8, 128, 28672)


@dataclass(frozen=True)
class Workload:
    """A seeded synthetic serving workload for one stage.

    ``resident`` is the number of resident layers (a prefix of layer ids); the
    rest are streamed from pinned host memory through ``stream_slots`` HBM slots.
    ``thresholds`` are context lengths at which one more resident layer is
    demoted (highest id first).  ``feedback`` feeds each decode output back as
    the next decode input; otherwise every decode step takes fresh hidden states.
    """
    name: str
    workload_id: int
    shape: StageShape
    n_mb: int
    batch: int
    prefill: int
    decode_steps: int
    feedback: bool = False
    resident: Optional[int] = None
    stream_slots: int = 2
    kv_block: int = 16
    thresholds: Tuple[int, ...] = field(default_factory=tuple)

    @property
    def n_resident(self) -> int:
        return self.shape.n_layers if self.resident is None else self.resident

    @property
    def max_context(self) -> int:
        return self.prefill + self.decode_steps


WORKLOADS: Dict[str, Workload] = {
    # 2 layers, hidden 256, batch 1, prefill 16 then 16 decode steps fed back.
    "tiny": Workload("tiny", 0, TINY, 1, 1, 16, 16, feedback=True),
    # 8 resident layers, batch 1, prefill 1024 then 128 decode steps.
    "llama8b_stage": Workload("llama8b_stage", 1, LLAMA8B_STAGE, 1, 1, 1024, 128),
    # 16 resident layers, 4 interleaved micro-batches of batch 1.
    "llama70b_resident": Workload("llama70b_resident", 2, LLAMA70B_STAGE, 4, 1, 2048, 256),
    # Same stage, 4 resident layers, 12 streamed through 2 reusable HBM slots.
    "llama70b_offload": Workload("llama70b_offload", 3, LLAMA70B_STAGE, 4, 1, 2048, 256, resident=4),
    # 8 micro-batches of batch 2, context 512 -> 8192, residency 16 -> 8.
    "llama70b_kvpressure": Workload(
        "llama70b_kvpressure", 4, LLAMA70B_STAGE, 8, 2, 512, 7680,
        thresholds=tuple(512 + 960 * j for j in range(1, 9))),
}


def seed_of(*parts: int) -> int:
    """Fold integers into one 64-bit stream seed with the SplitMix64 finaliser."""
    h = 0x243F6A8885A308D3
    for p in parts:
        h = _mix64((h ^ (int(p) & _MASK)) + 0x9E3779B97F4A7C15)
    return h


def _mix64(z: int) -> int:
    z &= _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


# ---------------------------------------------------------------------------
# native generator
# ---------------------------------------------------------------------------
def lib_path() -> str:
    return os.path.join(_HERE, "_libsynth.so")


def build_lib() -> str:
    """Compile gen.c into _libsynth.so (plain C, OpenMP)."""
    out = lib_path()
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC",
                           os.path.join(_HERE, "gen.c"), "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(lib_path()):
            build_lib()
        lib = ctypes.CDLL(lib_path())
        u64, i64, dbl, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        lib.synth_normal_bf16.argtypes = [u64, u64, i64, dbl, dbl, vp]
        lib.synth_normal_f32.argtypes = [u64, u64, i64, dbl, dbl, vp]
        lib.synth_draws.argtypes = [u64, u64, i64, vp]
        for f in (lib.synth_normal_bf16, lib.synth_normal_f32, lib.synth_draws):
            f.restype = None
        _LIB = lib
    return _LIB


def normal_bf16(seed: int, shape, mean: float = 0.0, std: float = 1.0, offset: int = 0) -> np.ndarray:
    """bf16 bits (uint16) of mean + std * N(0,1), element j from counter offset + j."""
    out = np.empty(shape, dtype=np.uint16)
    _lib().synth_normal_bf16(seed, offset, out.size, mean, std, out.ctypes.data)
    return out


def normal_f32(seed: int, shape, mean: float = 0.0, std: float = 1.0, offset: int = 0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _lib().synth_normal_f32(seed, offset, out.size, mean, std, out.ctypes.data)
    return out


def draws(seed: int, n: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    _lib().synth_draws(seed, offset, n, out.ctypes.data)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# workload tensors
# ---------------------------------------------------------------------------
def layer_weight_shapes(shape: StageShape) -> Dict[str, Tuple[int, ...]]:
    h = shape.hidden
    return {
        "wq": (shape.q_dim, h), "wk": (shape.kv_dim, h), "wv": (shape.kv_dim, h),
        "wo": (h, shape.q_dim), "wg": (shape.ffn, h), "wu": (shape.ffn, h), "wd": (h, shape.ffn),
        "g1": (h,), "g2": (h,),
    }


def layer_weights(shape: StageShape, layer: int) -> Dict[str, np.ndarray]:
    """bf16 bits of every tensor of one layer, [out, in] row-major for projections."""
    out = {}
    for name, shp in layer_weight_shapes(shape).items():
        seed = seed_of(0x57, shape.shape_id, layer, TENSOR_IDS[name])
        if name in ("g1", "g2"):
            out[name] = normal_bf16(seed, shp, mean=1.0, std=0.02)
        else:
            out[name] = normal_bf16(seed, shp, mean=0.0, std=0.02)
    return out


def prefill_inputs(wl: Workload, mb: int, b: int, n_tokens: Optional[int] = None) -> np.ndarray:
    """fp32 [T, H] hidden states entering the stage for a prefill of sequence (mb, b)."""
    t = wl.prefill if n_tokens is None else n_tokens
    return normal_f32(seed_of(0xA1, wl.workload_id, 0, mb, b, 0), (t, wl.shape.hidden))


def decode_input(wl: Workload, mb: int, b: int, step: int) -> np.ndarray:
    """fp32 [H] fresh hidden state entering the stage at decode step ``step``."""
    return normal_f32(seed_of(0xA1, wl.workload_id, 1, mb, b, step), (wl.shape.hidden,))
