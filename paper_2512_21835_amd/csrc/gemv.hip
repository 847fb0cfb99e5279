// Decode projections: y = W x with bf16 weights W [N, K] (row-major), fp32 activations and fp32
// accumulation, for up to 8 activation rows per launch.
//
// Work split.  A workgroup of four wavefronts owns R units over the whole K range.  A unit is one
// output row, or a pair of rows that the epilogue needs together: (gate row f, up row f) for
// SwiGLU, (row i, row i + d/2) of one head for rotate-half RoPE.  K is cut into steps of 512
// (1 KiB of bf16 per row); wavefront w takes steps w, w + 4, w + 8, ... of every owned row, lane l
// reading 16 bytes at k = 512 s + 8 l of step s.  Splitting K across the wavefronts (instead of
// giving each wavefront whole rows) lets one activation load serve all R units and leaves each
// wavefront a quarter of the dependent load round trips; U steps are loaded before they are used.
// Each wavefront reduces its lane partial sums with a butterfly of shuffles, the four wavefront
// partials meet in LDS, and wavefront 0 runs the epilogue.
//
// Fused: the RMSNorm in front of the QKV and gate/up projections (the sum of squares of x comes
// from the same activation loads; the 1/rms scale is applied to the finished dot product), RoPE and
// the KV-cache store after the QKV projection, SwiGLU of the gate/up pair, and the residual add
// after the O and down projections.
//
// Arithmetic of one output element (and of one row's sum of squares): per wavefront, per lane, a
// chain of fused multiply-adds over the wavefront's steps in ascending k; one fixed butterfly; then
// the partials of wavefronts 0, 1, 2, 3 added in that order.  R, U and M only decide which
// workgroup computes what and how loads are batched, so results do not depend on how many
// micro-batches share a call.
//
// Matrix-core engine (gemv_mfma_kernel), for launches of 5 to 16 activation rows, where the
// vector kernel becomes bound by its multiply-adds (one per row per weight element): the rows
// are the A operand of v_mfma_f32_16x16x32_bf16 (padded to 16, the fp32 activation as a bf16
// hi + lo pair, two MFMAs), 16 weight rows of a block the B operand, read straight from memory
// (lane l: row l % 16, 16 bytes at k = 32 s + 8 (l / 16)).  The same K split across the four
// wavefronts (128-wide k chunks, chunk c to wavefront c % 4), the same wavefront-order sum in
// LDS and the same epilogues.  Its results are independent of the row count too, but differ in
// rounding from the vector kernel's (by ~1e-5 relative).  With a workspace, the QKV, O and down
// projections run it split: 64 units per workgroup (each workgroup then re-reads the activation
// rows, 64 bytes per k at 16 rows, for four times as many weight rows) and K cut into up to 8
// ranges across workgroups so the grid still covers the GPU; a second launch adds the ranges in
// ascending order and applies the epilogue.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "stage_kernels.h"

namespace stg {
namespace {

constexpr int kWaves = 4;
constexpr int kStep = 512;  // k per wavefront step (64 lanes x 8 bf16)
constexpr int kMaxRowsPerLaunch = 8;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte weight load marked non-temporal: weights are streamed once per call.
__device__ __forceinline__ uint4 load_stream16(const uint16_t *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float bf16lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

__device__ __forceinline__ void unpack8(const uint4 &v, float f[8]) {
    f[0] = bf16lo(v.x); f[1] = bf16hi(v.x);
    f[2] = bf16lo(v.y); f[3] = bf16hi(v.y);
    f[4] = bf16lo(v.z); f[5] = bf16hi(v.z);
    f[6] = bf16lo(v.w); f[7] = bf16hi(v.w);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <int MODE> struct Shape {
    static constexpr bool kNorm = MODE != GEMV_PLAIN_RESIDUAL;
    static constexpr int NW = MODE == GEMV_PLAIN_RESIDUAL ? 1 : 2;  // weight rows per unit
};

template <int MODE>
__device__ __forceinline__ int n_units(const GemvArgs &a) {
    return MODE == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N;
}

// Weight row w (0 or 1) of unit u.
template <int MODE>
__device__ __forceinline__ const uint16_t *unit_row(const GemvArgs &a, int u, int w) {
    if (MODE == GEMV_NORM_ROPE_KV) {
        const int half = a.kv.head_dim / 2;
        const int h = u / half, i = u % half;
        return a.w + (size_t)(h * a.kv.head_dim + i + w * half) * a.K;
    }
    if (MODE == GEMV_NORM_SWIGLU) return (w ? a.w2 : a.w) + (size_t)u * a.K;
    return a.w + (size_t)u * a.K;
}

__device__ __forceinline__ void store_kv(void *pool, size_t e, float v, int kv_fp32) {
    if (kv_fp32)
        static_cast<float *>(pool)[e] = v;
    else
        static_cast<uint16_t *>(pool)[e] = to_bf16(v);
}

// RoPE + KV store of one (row i, row i + d/2) pair of head h for activation row m.  Heads below Hq
// are queries (rotated, to out), the next Hkv keys (rotated, to the cache), the last Hkv values.
__device__ __forceinline__ void rope_kv_epilogue(const GemvArgs &a, int u, int m, float x1, float x2) {
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

// One workgroup: units blockIdx.x * R .. + R - 1 for the launch's a.rows (<= M) activation rows.
template <int M, int R, int U, int MODE>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    constexpr int NP = NW * R * M + (kNorm ? M : 0);  // partials per wavefront
    __shared__ float part[kWaves][NP];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int units = n_units<MODE>(a);
    const int unit0 = blockIdx.x * R;
    const int K = a.K, steps = (K + kStep - 1) / kStep, rows = a.rows;

    // rows of units past the last are clamped to it: their loads stay in bounds, results are dropped
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

    for (int s0 = wave; s0 < steps; s0 += kWaves * U) {
        uint4 wv[U][NW][R];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = s0 + kWaves * u, k = s * kStep + lane * 8;
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int r = 0; r < R; ++r)
                    wv[u][w][r] = (s < steps && k < K) ? load_stream16(wrow[w][r] + k) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = s0 + kWaves * u, k = s * kStep + lane * 8;
            if (s >= steps || k >= K) break;
            float g[8];
            if (kNorm) unpack8(*reinterpret_cast<const uint4 *>(a.gain + k), g);
#pragma unroll
            for (int m = 0; m < M; ++m) {
                if (m >= rows) break;
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

    // wavefront partials -> LDS, laid out [w][r][m] then the sums of squares [m]
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int m = 0; m < M; ++m) {
                const float v = wave_sum(acc[w][r][m]);
                if (lane == 0) part[wave][(w * R + r) * M + m] = v;
            }
    if (kNorm) {
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const float v = wave_sum(ss[m]);
            if (lane == 0) part[wave][NW * R * M + m] = v;
        }
    }
    __syncthreads();

    // epilogue: lane r * M + m of wavefront 0 finishes unit unit0 + r of activation row m
    if (wave != 0 || lane >= R * M) return;
    const int r = lane / M, m = lane % M, u = unit0 + r;
    if (u >= units || m >= rows) return;
    auto total = [&](int i) { return ((part[0][i] + part[1][i]) + part[2][i]) + part[3][i]; };
    float scale = 1.f;
    if (kNorm) scale = 1.f / sqrtf(total(NW * R * M + m) / (float)K + a.eps);
    const float y0 = total(r * M + m) * scale;
    if (MODE == GEMV_NORM_ROPE_KV) {
        rope_kv_epilogue(a, u, m, y0, total((R + r) * M + m) * scale);
    } else if (MODE == GEMV_PLAIN_RESIDUAL) {
        a.out[m * a.out_ld + u] = a.res[m * a.out_ld + u] + y0;
    } else {
        const float up = total((R + r) * M + m) * scale;
        a.out[m * a.out_ld + u] = y0 / (1.f + expf(-y0)) * up;
    }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kMfmaRows = 16;     // activation rows per matrix-core launch
constexpr int kMfmaMinRows = 5;   // fewer rows: the vector kernel is faster
constexpr int kChunkK = 128;      // k per wavefront chunk (4 MFMA k steps of 32)

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4 &v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// One workgroup: RB blocks of 16 units (units blockIdx.x * 16 RB ..) for up to 16 activation rows;
// SPLIT: k chunks [blockIdx.y * cps, (blockIdx.y + 1) * cps) only, partial results to the
// workspace.
template <int MODE, int RB, bool SPLIT = false>
__global__ __launch_bounds__(256) void gemv_mfma_kernel(GemvArgs a, int cps) {
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    __shared__ float part[kWaves][NW * RB][16][17];   // wavefront partial D[m][n] per weight block
    __shared__ float ssp[kWaves][16];                  // wavefront partial sums of squares per row
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int units = n_units<MODE>(a);
    const int unit0 = blockIdx.x * 16 * RB;
    const int K = a.K, chunks = K / kChunkK, rows = a.rows;
    const int nl = lane & 15, kq = lane >> 4;
    const bool mvalid = nl < rows;   // this lane's A row (activation row nl)

    const uint16_t *wrow[NW][RB];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int b = 0; b < RB; ++b)
            wrow[w][b] = unit_row<MODE>(a, min(unit0 + 16 * b + nl, units - 1), w) + 8 * kq;
    const float *xr = a.act + (size_t)(mvalid ? nl : 0) * a.act_ld + 8 * kq;

    f32x4 d[NW][RB];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int b = 0; b < RB; ++b) d[w][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;
    const int c_beg = SPLIT ? blockIdx.y * cps : 0;
    const int c_end = SPLIT ? min(c_beg + cps, chunks) : chunks;
    for (int c = c_beg + wave; c < c_end; c += kWaves) {
        uint4 wv[4][NW][RB];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int b = 0; b < RB; ++b) wv[s4][w][b] = load_stream16(wrow[w][b] + kChunkK * c + 32 * s4);
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const int k = kChunkK * c + 32 * s4;
            const float4 x0 = *reinterpret_cast<const float4 *>(xr + k);
            const float4 x1 = *reinterpret_cast<const float4 *>(xr + k + 4);
            float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            float g[8];
            if (kNorm) unpack8(*reinterpret_cast<const uint4 *>(a.gain + k + 8 * kq), g);
            bf16x8 xh, xl;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                float v = mvalid ? x[j] : 0.f;
                if (kNorm) {
                    ss = fmaf(v, v, ss);
                    v = v * g[j];
                }
                xh[j] = (__bf16)v;                       // nearest even
                xl[j] = (__bf16)(v - (float)xh[j]);
            }
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int b = 0; b < RB; ++b) {
                    d[w][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, as_bf16x8(wv[s4][w][b]), d[w][b], 0, 0, 0);
                    d[w][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl, as_bf16x8(wv[s4][w][b]), d[w][b], 0, 0, 0);
                }
        }
    }
    // result register i of lane l: D[m = 4 (l / 16) + i][n = l % 16]
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int b = 0; b < RB; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) part[wave][w * RB + b][4 * kq + i][nl] = d[w][b][i];
    if (kNorm) {
        ss += __shfl_xor(ss, 16, 64);
        ss += __shfl_xor(ss, 32, 64);
        if (lane < 16) ssp[wave][lane] = ss;
    }
    __syncthreads();

    if (SPLIT) {  // workspace [split][w][m][units], wavefront-order sums
        const int split = blockIdx.y;
        for (int e = threadIdx.x; e < NW * 16 * RB * kMfmaRows; e += 256) {
            const int m = e % kMfmaRows, r = e / kMfmaRows, ub = r % (16 * RB), w = r / (16 * RB);
            const int u = unit0 + ub, wb = w * RB + ub / 16, n = ub % 16;
            if (m >= rows || u >= units) continue;
            a.split_part[(((size_t)split * NW + w) * kMfmaRows + m) * units + u] =
                ((part[0][wb][m][n] + part[1][wb][m][n]) + part[2][wb][m][n]) + part[3][wb][m][n];
        }
        if (kNorm && blockIdx.x == 0 && threadIdx.x < rows)
            a.split_ss[split * kMfmaRows + threadIdx.x] =
                ((ssp[0][threadIdx.x] + ssp[1][threadIdx.x]) + ssp[2][threadIdx.x]) + ssp[3][threadIdx.x];
        return;
    }
    for (int e = threadIdx.x; e < 16 * RB * kMfmaRows; e += 256) {
        const int m = e % kMfmaRows, ub = e / kMfmaRows, b = ub / 16, n = ub % 16;
        const int u = unit0 + ub;
        if (m >= rows || u >= units) continue;
        auto total = [&](int wb) { return ((part[0][wb][m][n] + part[1][wb][m][n]) + part[2][wb][m][n]) + part[3][wb][m][n]; };
        float scale = 1.f;
        if (kNorm) scale = 1.f / sqrtf((((ssp[0][m] + ssp[1][m]) + ssp[2][m]) + ssp[3][m]) / (float)K + a.eps);
        const float y0 = total(b) * scale;
        if (MODE == GEMV_NORM_ROPE_KV) {
            rope_kv_epilogue(a, u, m, y0, total(RB + b) * scale);
        } else if (MODE == GEMV_PLAIN_RESIDUAL) {
            a.out[m * a.out_ld + u] = a.res[m * a.out_ld + u] + y0;
        } else {
            const float up = total(RB + b) * scale;
            a.out[m * a.out_ld + u] = y0 / (1.f + expf(-y0)) * up;
        }
    }
}

// Adds the k ranges of a split matrix-core launch in ascending order and applies the epilogue:
// one thread per (row, unit).
template <int MODE>
__global__ __launch_bounds__(256) void gemv_split_epilogue(GemvArgs a, int splits) {
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    const int units = n_units<MODE>(a);
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= a.rows * units) return;
    const int m = e / units, u = e % units;
    float t[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        float acc = a.split_part[((size_t)w * kMfmaRows + m) * units + u];
        for (int sp = 1; sp < splits; ++sp) acc += a.split_part[(((size_t)sp * NW + w) * kMfmaRows + m) * units + u];
        t[w] = acc;
    }
    float scale = 1.f;
    if (kNorm) {
        float sq = a.split_ss[m];
        for (int sp = 1; sp < splits; ++sp) sq += a.split_ss[sp * kMfmaRows + m];
        scale = 1.f / sqrtf(sq / (float)a.K + a.eps);
    }
    const float y0 = t[0] * scale;
    if (MODE == GEMV_NORM_ROPE_KV) {
        rope_kv_epilogue(a, u, m, y0, t[NW - 1] * scale);
    } else if (MODE == GEMV_PLAIN_RESIDUAL) {
        a.out[m * a.out_ld + u] = a.res[m * a.out_ld + u] + y0;
    } else {
        const float up = t[NW - 1] * scale;
        a.out[m * a.out_ld + u] = y0 / (1.f + expf(-y0)) * up;
    }
}

int host_units(int mode, const GemvArgs &a) { return mode == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N; }

template <int MODE, int RB>
void launch_mfma_rb(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const int grid = (host_units(MODE, c) + 16 * RB - 1) / (16 * RB);
    if (e0 || e1)
        hipExtLaunchKernelGGL((gemv_mfma_kernel<MODE, RB>), dim3(grid), dim3(256), 0, st, e0, e1, 0, c, 0);
    else
        hipLaunchKernelGGL((gemv_mfma_kernel<MODE, RB>), dim3(grid), dim3(256), 0, st, c, 0);
}

// Split launch: 64 units per workgroup, k ranges so that the grid has about 256 workgroups (up to
// 8; swept on the 8B- and 70B-shaped QKV, O and down projections), then the epilogue launch.
template <int MODE>
void launch_mfma_split(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const int units = host_units(MODE, c), chunks = c.K / kChunkK;
    const int blocks = (units + 63) / 64;
    int splits = (256 + blocks - 1) / blocks;
    splits = max(1, min(splits, min(kGemvMaxSplits, chunks)));
    const int cps = (chunks + splits - 1) / splits;
    splits = (chunks + cps - 1) / cps;  // no empty range
    if (e0)
        hipExtLaunchKernelGGL((gemv_mfma_kernel<MODE, 4, true>), dim3(blocks, splits), dim3(256), 0, st, e0, nullptr, 0,
                              c, cps);
    else
        hipLaunchKernelGGL((gemv_mfma_kernel<MODE, 4, true>), dim3(blocks, splits), dim3(256), 0, st, c, cps);
    const int eg = (c.rows * units + 255) / 256;
    if (e1)
        hipExtLaunchKernelGGL((gemv_split_epilogue<MODE>), dim3(eg), dim3(256), 0, st, nullptr, e1, 0, c, splits);
    else
        hipLaunchKernelGGL((gemv_split_epilogue<MODE>), dim3(eg), dim3(256), 0, st, c, splits);
}

// Two 16-unit blocks per workgroup where that still gives at least 256 workgroups (swept on the
// 8B- and 70B-shaped layers: fewer workgroups than compute units cost more than the block pair
// saves), one otherwise; the split launch for the QKV, O and down projections given a workspace.
template <int MODE>
void launch_mfma(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    if (MODE != GEMV_NORM_SWIGLU && c.split_part && c.split_ss) launch_mfma_split<MODE>(c, st, e0, e1);
    else if (host_units(MODE, c) >= 32 * 256) launch_mfma_rb<MODE, 2>(c, st, e0, e1);
    else launch_mfma_rb<MODE, 1>(c, st, e0, e1);
}

template <int M, int R, int U, int MODE>
void launch_one(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const int grid = (host_units(MODE, c) + R - 1) / R;
    if (e0 || e1)
        hipExtLaunchKernelGGL((gemv_kernel<M, R, U, MODE>), dim3(grid), dim3(256), 0, st, e0, e1, 0, c);
    else
        hipLaunchKernelGGL((gemv_kernel<M, R, U, MODE>), dim3(grid), dim3(256), 0, st, c);
}

// Units per workgroup and steps in flight, by mode and rows (swept on the 8B- and 70B-shaped
// layers): one row: gate/up 4 units x 1 step, O and down 4 x 2, QKV 2 x 1 (2 x 2 on the larger
// shape); two rows: O and down 4 x 1 (8 x 1 for the 70B down projection), QKV 4 x 1 (2 x 1 on the
// larger shape); fewer as the rows multiply the registers.
template <int M, int MODE>
void launch_rows(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const long work = (long)host_units(MODE, c) * c.K;
    if (MODE == GEMV_PLAIN_RESIDUAL) {
        if (M == 1) launch_one<M, 4, 2, MODE>(c, st, e0, e1);
        else if (M == 2 && work >= 200L * 1000 * 1000) launch_one<M, 8, 1, MODE>(c, st, e0, e1);
        else launch_one<M, 4, 1, MODE>(c, st, e0, e1);
    } else if (MODE == GEMV_NORM_SWIGLU) {
        if (M <= 4) launch_one<M, 4, 1, MODE>(c, st, e0, e1);
        else launch_one<M, 2, 1, MODE>(c, st, e0, e1);
    } else {
        const bool big = work >= 40L * 1000 * 1000;
        if (M == 1 && big) launch_one<M, 2, 2, MODE>(c, st, e0, e1);
        else if (M == 2 && !big) launch_one<M, 4, 1, MODE>(c, st, e0, e1);
        else launch_one<M, 2, 1, MODE>(c, st, e0, e1);
    }
}

template <int MODE>
hipError_t launch_mode(const GemvArgs &a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    // 16-unit blocks must not straddle the two halves of a RoPE head
    const bool mfma_ok = a.K % kChunkK == 0 && (MODE != GEMV_NORM_ROPE_KV || (a.kv.head_dim / 2) % 16 == 0);
    for (int r0 = 0, n = 0; r0 < a.rows; r0 += n) {
        const int left = a.rows - r0;
        const bool mfma = mfma_ok && left >= kMfmaMinRows;
        n = min(left, mfma ? kMfmaRows : kMaxRowsPerLaunch);
        GemvArgs c = a;
        c.rows = n;
        c.row0 = a.row0 + r0;
        c.act = a.act + (size_t)r0 * a.act_ld;
        c.out = a.out + (size_t)r0 * a.out_ld;
        if (a.res) c.res = a.res + (size_t)r0 * a.out_ld;
        hipEvent_t e0 = r0 == 0 ? ev_start : nullptr;
        hipEvent_t e1 = r0 + n >= a.rows ? ev_stop : nullptr;
        if (mfma)
            launch_mfma<MODE>(c, st, e0, e1);
        else if (c.rows == 1)
            launch_rows<1, MODE>(c, st, e0, e1);
        else if (c.rows == 2)
            launch_rows<2, MODE>(c, st, e0, e1);
        else if (c.rows <= 4)
            launch_rows<4, MODE>(c, st, e0, e1);
        else
            launch_rows<8, MODE>(c, st, e0, e1);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_gemv(int mode, GemvArgs a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    if (a.rows <= 0) return hipSuccess;
    if (a.K <= 0 || a.K % 8 != 0 || a.N <= 0) return hipErrorInvalidValue;
    switch (mode) {
        case GEMV_PLAIN_RESIDUAL: return launch_mode<GEMV_PLAIN_RESIDUAL>(a, st, ev_start, ev_stop);
        case GEMV_NORM_SWIGLU: return launch_mode<GEMV_NORM_SWIGLU>(a, st, ev_start, ev_stop);
        case GEMV_NORM_ROPE_KV: return launch_mode<GEMV_NORM_ROPE_KV>(a, st, ev_start, ev_stop);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace stg
