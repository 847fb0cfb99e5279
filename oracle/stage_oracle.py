"""Float64 CPU oracle of one pipeline stage's forward -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may use this module.  It is deliberately plain: every step is the textbook
definition written out with float64 torch CPU tensors, no blocking, no fusion.

What is computed
----------------
The paper's interleaved pipeline (Section III-A, Fig. 2) gives every device
stages, each a contiguous block of decoder layers, and runs micro-batches
through them in turn; offloading and slot reuse (Section III-C) move weights,
never change the arithmetic, so inference stays lossless (abstract, Section
IV-A "Evaluation Metrics").  The oracle therefore ignores residency and computes
the plain forward of the layer block.  The paper does not spell out the decoder
layer; it serves LLaMA-family checkpoints (Section IV-A "Models", citing the
LLaMA 3 report), so each layer is the LLaMA decoder:

    y   = x / sqrt(mean(x^2) + eps) * g1                      (RMSNorm)
    q, k, v = Wq y, Wk y, Wv y                                 (projections)
    q, k    = RoPE(q, p), RoPE(k, p)                           (rotate-half pairs (i, i+d/2))
    K, V   <- append(round_kv(k), round_kv(v))                 (KV cache store)
    o_h = sum_j softmax_j(q_h . K_{g(h),j} / sqrt(d)) V_{g(h),j},  j <= p   (causal GQA)
    x   = x + Wo concat_h(o_h)
    y2  = x / sqrt(mean(x^2) + eps) * g2
    x   = x + Wd (silu(Wg y2) * (Wu y2)),  silu(z) = z / (1 + e^-z)

with g(h) = floor(h / (Hq / Hkv)).  The stage output is x after its last layer
(no final norm: that belongs to the model's last stage).  ``round_kv`` is the
cache element type: bf16 (value rounded to float32, then to bf16, both nearest
even -- the same precision in which the kernel takes the decision) or float32.

Weights are the exact float64 widening of their bf16 bits.  Everything else is
float64.

Pins (tests/test_oracle_pins.py): RMSNorm unit RMS before the gain; RoPE closed
form on unit vectors, pair-norm preservation and relative-position invariance;
softmax rows sum to 1; one key returns V; zero queries give the causal mean of
V; GQA with Hkv = Hq equals per-head brute force; decode step t equals row t of
one prefill; a pure-Python loop brute force of the tiny layer, which also pins
layer_kv and decoder_layer_rows.
"""
from __future__ import annotations

import math
from typing import Optional, Callable, Dict, Hashable, List, Sequence, Tuple

import numpy as np
import torch

F64 = torch.float64


# ---------------------------------------------------------------------------
# element types
# ---------------------------------------------------------------------------
def widen_bf16(bits) -> torch.Tensor:
    """Exact float64 value of bf16 bit patterns (uint16 numpy array or int16 tensor)."""
    if isinstance(bits, np.ndarray):
        bits = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return bits.view(torch.bfloat16).to(F64)


def round_to_f32(x: torch.Tensor) -> torch.Tensor:
    """Round to the nearest float32 (ties to even) and return it as float64."""
    return x.to(torch.float32).to(F64)


def round_to_bf16(x: torch.Tensor) -> torch.Tensor:
    """Round to float32, then float32 to bf16, both to nearest even; return float64.

    The bf16 step is written on the float32 bit pattern: add 0x7FFF plus the
    lowest kept bit, then clear the 16 dropped bits.
    """
    u = x.to(torch.float32).view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    u = torch.where(u >= 0x80000000, u - (1 << 32), u).to(torch.int32)
    return u.view(torch.float32).to(F64)


def bf16_bits(x: torch.Tensor) -> np.ndarray:
    """bf16 bit patterns (uint16) of values that are already bf16-exact."""
    u = x.to(torch.float32).view(torch.int32).numpy().view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value is not bf16-exact"
    return (u >> 16).astype(np.uint16)


# ---------------------------------------------------------------------------
# the decoder layer, step by step
# ---------------------------------------------------------------------------
def rms_norm(x: torch.Tensor, g: torch.Tensor, eps: float) -> torch.Tensor:
    """x / sqrt(mean over the hidden dimension of x^2 + eps), times the gain g."""
    ms = (x * x).mean(dim=-1, keepdim=True)
    return x / torch.sqrt(ms + eps) * g


def rope_angles(positions: torch.Tensor, head_dim: int, theta: float) -> torch.Tensor:
    """angle[p, i] = p * theta^(-2i/d), i = 0 .. d/2-1, in float64."""
    i = torch.arange(head_dim // 2, dtype=F64)
    inv = theta ** (-2.0 * i / head_dim)
    return positions.to(F64)[:, None] * inv[None, :]


def rope(x: torch.Tensor, positions: torch.Tensor, theta: float) -> torch.Tensor:
    """Rotate-half RoPE: x [T, n_heads, d] at positions [T].

    Pair (i, i + d/2) turns by angle[p, i]:
        x_i'       = x_i cos - x_{i+d/2} sin
        x_{i+d/2}' = x_i sin + x_{i+d/2} cos
    """
    d = x.shape[-1]
    ang = rope_angles(positions, d, theta)          # [T, d/2]
    c = torch.cos(ang)[:, None, :]
    s = torch.sin(ang)[:, None, :]
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return torch.cat([x1 * c - x2 * s, x1 * s + x2 * c], dim=-1)


def softmax(s: torch.Tensor) -> torch.Tensor:
    """Row softmax with the row maximum subtracted first; -inf entries get weight 0."""
    m = s.max(dim=-1, keepdim=True).values
    e = torch.exp(s - m)
    return e / e.sum(dim=-1, keepdim=True)


def gqa_attention(q: torch.Tensor, k_all: torch.Tensor, v_all: torch.Tensor,
                  q_positions: torch.Tensor) -> torch.Tensor:
    """Causal grouped-query attention of one sequence.

    q [T, Hq, d] at positions q_positions [T]; k_all, v_all [N, Hkv, d] hold the
    cache for positions 0..N-1 (new rows included).  Query head h reads KV head
    floor(h / (Hq / Hkv)); row t sees keys j <= q_positions[t].  Returns [T, Hq*d].
    """
    t, hq, d = q.shape
    n, hkv, _ = k_all.shape
    group = hq // hkv
    j = torch.arange(n)
    visible = j[None, :] <= q_positions[:, None]            # [T, N]
    out = torch.empty(t, hq, d, dtype=F64)
    for h in range(hq):
        g = h // group
        s = (q[:, h, :] @ k_all[:, g, :].T) / math.sqrt(d)    # [T, N]
        s = torch.where(visible, s, torch.tensor(-math.inf, dtype=F64))
        out[:, h, :] = softmax(s) @ v_all[:, g, :]
    return out.reshape(t, hq * d)


def silu(z: torch.Tensor) -> torch.Tensor:
    return z / (1.0 + torch.exp(-z))


class LayerWeights:
    """float64 widening of one layer's bf16 weights ([out, in] row-major)."""

    def __init__(self, bits: Dict[str, np.ndarray]):
        self.wq, self.wk, self.wv = (widen_bf16(bits[n]) for n in ("wq", "wk", "wv"))
        self.wo, self.wg, self.wu, self.wd = (widen_bf16(bits[n]) for n in ("wo", "wg", "wu", "wd"))
        self.g1, self.g2 = widen_bf16(bits["g1"]), widen_bf16(bits["g2"])


class LayerCache:
    """Stored K and V of one sequence at one layer: [N, Hkv, d] each (values as stored)."""

    def __init__(self, hkv: int, d: int):
        self.k = torch.zeros(0, hkv, d, dtype=F64)
        self.v = torch.zeros(0, hkv, d, dtype=F64)

    def append(self, k: torch.Tensor, v: torch.Tensor) -> None:
        self.k = torch.cat([self.k, k], dim=0)
        self.v = torch.cat([self.v, v], dim=0)

    def __len__(self) -> int:
        return self.k.shape[0]


def decoder_layer(x: torch.Tensor, w: LayerWeights, cache: LayerCache, shape, kv_round) -> torch.Tensor:
    """One decoder layer on the new rows x [T, H] of one sequence (positions follow the cache)."""
    t = x.shape[0]
    hq, hkv, d = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    p0 = len(cache)
    positions = torch.arange(p0, p0 + t)

    y = rms_norm(x, w.g1, shape.rms_eps)
    q = (y @ w.wq.T).reshape(t, hq, d)
    k = (y @ w.wk.T).reshape(t, hkv, d)
    v = (y @ w.wv.T).reshape(t, hkv, d)
    q = rope(q, positions, shape.rope_theta)
    k = rope(k, positions, shape.rope_theta)
    cache.append(kv_round(k), kv_round(v))
    o = gqa_attention(q, cache.k, cache.v, positions)
    x = x + o @ w.wo.T

    y2 = rms_norm(x, w.g2, shape.rms_eps)
    h = silu(y2 @ w.wg.T) * (y2 @ w.wu.T)
    return x + h @ w.wd.T


def layer_kv(x: torch.Tensor, w: LayerWeights, shape, kv_round) -> Tuple[torch.Tensor, torch.Tensor]:
    """The K and V that one decoder layer stores for the rows x [T, H] of a new sequence
    (positions 0..T-1), as the cache holds them: [T, Hkv, d] each (the first steps of
    decoder_layer)."""
    t = x.shape[0]
    hkv, d = shape.n_kv_heads, shape.head_dim
    positions = torch.arange(t)
    y = rms_norm(x, w.g1, shape.rms_eps)
    k = rope((y @ w.wk.T).reshape(t, hkv, d), positions, shape.rope_theta)
    v = (y @ w.wv.T).reshape(t, hkv, d)
    return kv_round(k), kv_round(v)


def decoder_layer_rows(x: torch.Tensor, w: LayerWeights, shape, rows: Sequence[int],
                       k_all: torch.Tensor, v_all: torch.Tensor) -> torch.Tensor:
    """Outputs of the listed rows of one decoder layer over x [T, H] of a new sequence (positions
    0..T-1), attending over the stored K, V [T, Hkv, d] given: decoder_layer restricted to those
    rows.  Every step but attention acts on each row alone, and attention reads only its own
    query row and the stored K and V, so the restriction changes nothing for the rows kept."""
    hq, d = shape.n_q_heads, shape.head_dim
    idx = torch.as_tensor(list(rows), dtype=torch.long)
    xr = x[idx]
    y = rms_norm(xr, w.g1, shape.rms_eps)
    q = rope((y @ w.wq.T).reshape(len(idx), hq, d), idx, shape.rope_theta)
    o = gqa_attention(q, k_all, v_all, idx)
    xr = xr + o @ w.wo.T
    y2 = rms_norm(xr, w.g2, shape.rms_eps)
    h = silu(y2 @ w.wg.T) * (y2 @ w.wu.T)
    return xr + h @ w.wd.T


# ---------------------------------------------------------------------------
# the stage
# ---------------------------------------------------------------------------
class OracleStage:
    """The plain forward of one stage over many independent sequences.

    ``weights(l)`` returns the bf16 bits of layer l (see ``synth.layer_weights``).
    ``kv_dtype`` is "bf16" or "f32": the element type of the KV cache.
    Sequences are keyed by any hashable (e.g. (mb, b)); each has its own cache
    and positions.  ``forward`` takes a list of (key, new rows [T, H]) and
    returns the stage output rows of each, in float64.
    """

    def __init__(self, shape, weights: Callable[[int], Dict[str, np.ndarray]], kv_dtype: str = "bf16",
                 kv_jitter: float = 0.0, jitter_seed: int = 0):
        if kv_dtype not in ("bf16", "f32"):
            raise ValueError(kv_dtype)
        self.shape = shape
        self.weights = weights
        base = round_to_bf16 if kv_dtype == "bf16" else round_to_f32
        if kv_jitter:
            # Sensitivity of the result to the KV rounding point: every K/V value is scaled by
            # (1 + kv_jitter * u), u uniform in [-1, 1], before it is rounded to the cache type --
            # the stage as computed by an arithmetic that is kv_jitter-accurate (relative) up to
            # the cache store.  Used only to size tolerances; 0 (default) is the plain definition.
            gen = torch.Generator().manual_seed(jitter_seed)

            def jittered(t: torch.Tensor) -> torch.Tensor:
                u = torch.rand(t.shape, generator=gen, dtype=F64) * 2.0 - 1.0
                return base(t * (1.0 + kv_jitter * u))
            self.kv_round = jittered
        else:
            self.kv_round = base
        self.caches: Dict[Hashable, List[LayerCache]] = {}

    def cache(self, key: Hashable) -> List[LayerCache]:
        if key not in self.caches:
            s = self.shape
            self.caches[key] = [LayerCache(s.n_kv_heads, s.head_dim) for _ in range(s.n_layers)]
        return self.caches[key]

    def length(self, key: Hashable) -> int:
        return len(self.cache(key)[0])

    def forward(self, batch: Sequence[Tuple[Hashable, np.ndarray]],
                trace: Optional[List[List[np.ndarray]]] = None) -> List[np.ndarray]:
        """Runs every layer over the batch's new rows.  With ``trace``, appends each layer's input
        rows (one array per batch entry) before running it."""
        xs = [torch.as_tensor(np.asarray(x), dtype=F64).reshape(-1, self.shape.hidden) for _, x in batch]
        for layer in range(self.shape.n_layers):
            if trace is not None:
                trace.append([x.numpy().copy() for x in xs])
            w = LayerWeights(self.weights(layer))
            for i, (key, _) in enumerate(batch):
                xs[i] = decoder_layer(xs[i], w, self.cache(key)[layer], self.shape, self.kv_round)
            del w
        return [x.numpy() for x in xs]

    # --- the KV-tail move of the online KV transfer protocol (Section III-E, Alg. 2) ---
    def export_tail(self, key: Hashable, n: int, drop: bool) -> Tuple[np.ndarray, np.ndarray]:
        """Stored K, V of the last n positions, [L, n, Hkv, d] float64; drop them if asked."""
        c = self.cache(key)
        k = torch.stack([lc.k[len(lc) - n:] for lc in c]).numpy().copy()
        v = torch.stack([lc.v[len(lc) - n:] for lc in c]).numpy().copy()
        if drop:
            for lc in c:
                lc.k, lc.v = lc.k[: len(lc) - n], lc.v[: len(lc) - n]
        return k, v

    def append_kv(self, key: Hashable, k: np.ndarray, v: np.ndarray) -> None:
        """Concatenate received K, V ([L, n, Hkv, d], already rotated) onto the cache."""
        for layer, lc in enumerate(self.cache(key)):
            lc.append(torch.as_tensor(k[layer], dtype=F64), torch.as_tensor(v[layer], dtype=F64))

    def reset(self, key: Hashable) -> None:
        self.caches.pop(key, None)
