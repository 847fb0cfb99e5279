// Device code of the decode projections, shared by the per-projection kernels (gemv.hip) and the
// persistent per-layer decode kernel (decode_layer.hip).  y = W x with bf16 weights W [N, K]
// (row-major) and fp32 activations, fp32 accumulation, for up to 8 activation rows at once.
//
// A wavefront owns R units over the whole K range, a unit being one output row, or a pair of rows
// that its epilogue needs together: (gate row f, up row f) for SwiGLU, (row i, row i + d/2) of one
// head for rotate-half RoPE.  Lane l reads 16 bytes (8 bf16) of every owned row at k = l*8 + 512*i,
// so one load instruction covers 1 KiB of contiguous weights per row; U consecutive k steps are
// loaded before they are used.  Lane partial sums are combined with a butterfly of cross-lane
// shuffles.  Fused: the RMSNorm in front of the QKV and gate/up projections (the sum of squares of
// x is accumulated from the same loads and the 1/rms scale applied to the dot product), RoPE and
// the KV-cache store after the QKV projection, the SwiGLU of the gate/up pair, and the residual
// add after the O and down projections.
//
// Every output element is one fixed sequence of fused multiply-adds in ascending k followed by one
// fixed butterfly, whatever M, R, U or the caller: results do not depend on how many micro-batches
// share a call, nor on which kernel runs the projection.
#pragma once

#include <hip/hip_runtime.h>

#include "stage_kernels.h"

namespace stg {
namespace gemv_dev {

constexpr int kWaves = 4;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte weight load marked non-temporal: weights are streamed once per call.
static __device__ __forceinline__ uint4 load_stream16(const uint16_t *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

static __device__ __forceinline__ float bf16lo(uint32_t u) { return __uint_as_float(u << 16); }
static __device__ __forceinline__ float bf16hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

static __device__ __forceinline__ void unpack8(const uint4 &v, float f[8]) {
    f[0] = bf16lo(v.x); f[1] = bf16hi(v.x);
    f[2] = bf16lo(v.y); f[3] = bf16hi(v.y);
    f[4] = bf16lo(v.z); f[5] = bf16hi(v.z);
    f[6] = bf16lo(v.w); f[7] = bf16hi(v.w);
}

static __device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
static __device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <int MODE> struct Shape {
    static constexpr bool kNorm = MODE != GEMV_PLAIN_RESIDUAL;
    static constexpr int NW = (MODE == GEMV_NORM_SWIGLU || MODE == GEMV_NORM_ROPE_KV) ? 2 : 1;
};

// Weight row w (0 or 1) of unit u; units beyond the last are clamped to it (loads stay in bounds).
template <int MODE>
static __device__ __forceinline__ const uint16_t *unit_row(const GemvArgs &a, int u, int w) {
    if (MODE == GEMV_NORM_ROPE_KV) {
        const int half = a.kv.head_dim / 2;
        const int h = u / half, i = u % half;
        return a.w + (size_t)(h * a.kv.head_dim + i + w * half) * a.K;
    }
    if (MODE == GEMV_NORM_SWIGLU) return (w ? a.w2 : a.w) + (size_t)u * a.K;
    return a.w + (size_t)u * a.K;
}

template <int MODE>
static __device__ __forceinline__ int n_units(const GemvArgs &a) {
    return MODE == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N;
}

static __device__ __forceinline__ void store_kv(void *pool, size_t e, float v, int kv_fp32) {
    if (kv_fp32)
        static_cast<float *>(pool)[e] = v;
    else
        static_cast<uint16_t *>(pool)[e] = to_bf16(v);
}

// RoPE + KV store of one (row i, row i + d/2) pair of head h for activation row m.
static __device__ __forceinline__ void rope_kv_epilogue(const GemvArgs &a, int u, int m, float x1, float x2) {
    const int d = a.kv.head_dim, half = d / 2;
    const int h = u / half, i = u % half;
    const int row = a.row0 + m;
    const int sidx = row / a.meta->rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.meta->rows_per_seq;
    const int hq = a.n_q_heads, hkv = a.kv.n_kv_heads;
    float r1 = x1, r2 = x2;
    if (h < hq + hkv) {
        const float c = a.cos_t[(size_t)pos * half + i], s = a.sin_t[(size_t)pos * half + i];
        r1 = x1 * c - x2 * s;
        r2 = x1 * s + x2 * c;
    }
    if (h < hq) {
        float *q = a.out + m * a.out_ld + h * d;
        q[i] = r1;
        q[i + half] = r2;
        return;
    }
    const int slot = a.meta->seq_slot[sidx];
    const int block = a.kv.block_table[(size_t)slot * a.kv.max_blocks + pos / kBlockTokens];
    const int kv = h < hq + hkv ? 0 : 1;
    const int g = h - hq - kv * hkv;
    const size_t e = (((size_t)block * 2 + kv) * hkv + g) * kBlockTokens * d +
                     (size_t)(pos % kBlockTokens) * d + i;
    store_kv(a.kv.pool, e, r1, a.kv_fp32);
    store_kv(a.kv.pool, e + half, r2, a.kv_fp32);
}

template <int MODE, int R, int U>
struct Prefetch {
    uint4 w[U][Shape<MODE>::NW][R];
};

// Issues the weight loads of the first U k steps of units unit0 .. unit0+R-1; needs no activation.
template <int MODE, int R, int U>
static __device__ __forceinline__ void gemv_prefetch(const GemvArgs &a, int unit0, Prefetch<MODE, R, U> &p) {
    constexpr int NW = Shape<MODE>::NW;
    const int lane = threadIdx.x & 63;
    const int units = n_units<MODE>(a);
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint16_t *row = unit_row<MODE>(a, min(unit0 + r, units - 1), w);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int k = lane * 8 + u * 512;
                p.w[u][w][r] = k < a.K ? load_stream16(row + k) : make_uint4(0, 0, 0, 0);
            }
        }
}

// One wavefront's units unit0 .. unit0+R-1 (over all of K) and their epilogue.  With `use_pre`, the
// first U k steps come from `pre` (loaded earlier by gemv_prefetch for the same units).
template <int M, int R, int MODE, int U>
static __device__ __forceinline__ void gemv_wave(const GemvArgs &a, int unit0, bool use_pre,
                                                 const Prefetch<MODE, R, U> &pre) {
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    const int lane = threadIdx.x & 63;
    const int units = n_units<MODE>(a);
    if (unit0 >= units) return;

    const uint16_t *wrow[NW][R];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int r = 0; r < R; ++r) wrow[w][r] = unit_row<MODE>(a, min(unit0 + r, units - 1), w);

    float acc[NW][R][M];
    float ss[M];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        ss[m] = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int r = 0; r < R; ++r) acc[w][r][m] = 0.f;
    }

    for (int kb = lane * 8; kb < a.K; kb += 512 * U) {
        uint4 wv[U][NW][R];
        if (use_pre && kb == lane * 8) {
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int w = 0; w < NW; ++w)
#pragma unroll
                    for (int r = 0; r < R; ++r) wv[u][w][r] = pre.w[u][w][r];
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int w = 0; w < NW; ++w)
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        const int k = kb + u * 512;
                        wv[u][w][r] = k < a.K ? load_stream16(wrow[w][r] + k) : make_uint4(0, 0, 0, 0);
                    }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = kb + u * 512;
            if (k >= a.K) break;
            float g[8];
            if (kNorm) unpack8(*reinterpret_cast<const uint4 *>(a.gain + k), g);
#pragma unroll
            for (int m = 0; m < M; ++m) {
                if (m >= a.rows) break;
                const float4 *xp = reinterpret_cast<const float4 *>(a.act + m * a.act_ld + k);
                const float4 x0 = xp[0], x1 = xp[1];
                float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
                if (kNorm) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        ss[m] = fmaf(x[j], x[j], ss[m]);
                        x[j] = x[j] * g[j];
                    }
                }
#pragma unroll
                for (int w = 0; w < NW; ++w)
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        float f[8];
                        unpack8(wv[u][w][r], f);
#pragma unroll
                        for (int j = 0; j < 8; ++j) acc[w][r][m] = fmaf(f[j], x[j], acc[w][r][m]);
                    }
            }
        }
    }

#pragma unroll
    for (int m = 0; m < M; ++m) {
        if (kNorm) ss[m] = wave_sum(ss[m]);
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int r = 0; r < R; ++r) acc[w][r][m] = wave_sum(acc[w][r][m]);
    }

    // Epilogue: lane (r * M + m) finishes unit unit0 + r of activation row m.
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int m = 0; m < M; ++m) {
            if (lane != r * M + m) continue;
            const int u = unit0 + r;
            if (u >= units || m >= a.rows) continue;
            float scale = 1.f;
            if (kNorm) scale = 1.f / sqrtf(ss[m] / (float)a.K + a.eps);
            if (MODE == GEMV_NORM_ROPE_KV) {
                rope_kv_epilogue(a, u, m, acc[0][r][m] * scale, acc[NW - 1][r][m] * scale);
                continue;
            }
            float *o = a.out + m * a.out_ld + u;
            if (MODE == GEMV_NORM_STORE) {
                *o = acc[0][r][m] * scale;
            } else if (MODE == GEMV_PLAIN_RESIDUAL) {
                *o = a.res[m * a.out_ld + u] + acc[0][r][m];
            } else {
                const float gt = acc[0][r][m] * scale;
                const float up = acc[NW - 1][r][m] * scale;
                *o = gt / (1.f + expf(-gt)) * up;
            }
        }
    }
}

}  // namespace gemv_dev
}  // namespace stg
