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
// Matrix-core engine (gemv_mfma_kernel), for launches of 3 to 16 activation rows (5 to 16 for
// the square O projection), where the vector kernel falls behind (one multiply-add per row per
// weight element): the rows are the A operand of v_mfma_f32_16x16x32_bf16 (padded to 16, the
// fp32 activation as a bf16 hi + lo pair, two MFMAs), up to 16 weight rows the B operand.  A workgroup
// of four wavefronts owns 4 x 16 units (4 x 14 in unsplit launches where that evens out the grid),
// each wavefront its share over the workgroup's K range, in chunks of 128 k taken two at a time.  The
// B layout wants 16 rows x 64 bytes per load instruction, which streams HBM poorly (~4 TB/s; 4
// rows x 256 bytes ~5.7 TB/s), so a wavefront loads a pair of chunks as 2 rows x 512 contiguous
// bytes per instruction, stores both chunks in its own LDS tiles (the 16-byte k segments
// XOR-swizzled by row, so the stores are contiguous and the MFMA-layout reads are free of bank
// conflicts) and reads them back as B fragments.  The A fragments of a pair are converted once per
// workgroup (two per thread) into an LDS tile; two barriers per pair.  The next pair's weights and
// activations are loaded before the current pair is multiplied.  Per output element: MFMA
// accumulation over the chunks in ascending k.  K is cut into up to 8 ranges of whole chunk pairs
// across workgroups where the grid would leave compute units idle (partial products to a
// workspace) and a second launch adds the ranges in ascending order and applies the epilogue.
// Which of the two runs depends on the layer shape only, so results are independent of the row
// count; they differ in rounding from the vector kernel's (by ~1e-5 relative).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <atomic>

#include "lanes.h"
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
    for (int o = 32; o >= 1; o >>= 1) v += lane_xor(v, o);
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

// Epilogue inputs that do not depend on the dot products: the residual (O and down projections),
// or for a RoPE unit (row i, row i + d/2 of head h) the rotation at the row's position and the
// unit's place in the KV cache.  The vector kernel loads them before its weight stream, so their
// dependent round trips (row metadata, then tables) overlap it instead of following it.
struct EpiIn {
    float res = 0.f;
    float c = 1.f, s = 0.f;
    size_t kv_e = 0;
};

template <int MODE>
__device__ __forceinline__ EpiIn epi_load(const GemvArgs &a, int u, int m) {
    EpiIn e;
    if (MODE == GEMV_PLAIN_RESIDUAL) {
        e.res = a.res[m * a.out_ld + u];
    } else if (MODE == GEMV_NORM_ROPE_KV) {
        const int d = a.kv.head_dim, half = d / 2;
        const int h = u / half, i = u % half;
        const int row = a.row0 + m;
        const int sidx = row / a.meta->rows_per_seq;
        const int pos = a.meta->pos0[sidx] + row % a.meta->rows_per_seq;
        const int hq = a.n_q_heads, hkv = a.kv.n_kv_heads;
        if (h < hq + hkv) {
            e.c = a.cos_t[(size_t)pos * half + i];
            e.s = a.sin_t[(size_t)pos * half + i];
        }
        if (h >= hq) {
            const int slot = a.meta->seq_slot[sidx];
            const int block = a.kv.block_table[(size_t)slot * a.kv.max_blocks + pos / kBlockTokens];
            const int kv = h < hq + hkv ? 0 : 1;
            const int g = h - hq - kv * hkv;
            e.kv_e = (((size_t)block * 2 + kv) * hkv + g) * kBlockTokens * d + (size_t)(pos % kBlockTokens) * d + i;
        }
    }
    return e;
}

// Finishes unit u of activation row m from its (scaled) dot products y0 and y1 (second row of the
// unit: up projection, or row i + d/2): SwiGLU; residual add; or RoPE, then queries to `out`
// and keys/values (heads Hq .. Hq + Hkv - 1, then the last Hkv) to the cache.
template <int MODE>
__device__ __forceinline__ void epi_store(const GemvArgs &a, const EpiIn &e, int u, int m, float y0, float y1) {
    if (MODE == GEMV_PLAIN_RESIDUAL) {
        a.out[m * a.out_ld + u] = e.res + y0;
    } else if (MODE == GEMV_NORM_SWIGLU) {
        a.out[m * a.out_ld + u] = y0 / (1.f + expf(-y0)) * y1;
    } else {
        const int d = a.kv.head_dim, half = d / 2;
        const int h = u / half, i = u % half;
        const int hq = a.n_q_heads, hkv = a.kv.n_kv_heads;
        float r1 = y0, r2 = y1;
        if (h < hq + hkv) {
            r1 = y0 * e.c - y1 * e.s;
            r2 = y0 * e.s + y1 * e.c;
        }
        if (h < hq) {
            float *q = a.out + m * a.out_ld + h * d;
            q[i] = r1;
            q[i + half] = r2;
            return;
        }
        store_kv(a.kv.pool, e.kv_e, r1, a.kv_fp32);
        store_kv(a.kv.pool, e.kv_e + half, r2, a.kv_fp32);
    }
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

    // epilogue inputs of lane r * M + m of wavefront 0 (unit unit0 + r, row m), ahead of the weights
    const int er = lane / M, em = lane % M, eu = unit0 + er;
    const bool epi_lane = wave == 0 && lane < R * M && eu < units && em < rows;
    EpiIn epi;
    if (epi_lane) epi = epi_load<MODE>(a, eu, em);

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
    if (!epi_lane) return;
    auto total = [&](int i) { return ((part[0][i] + part[1][i]) + part[2][i]) + part[3][i]; };
    float scale = 1.f;
    if (kNorm) scale = 1.f / sqrtf(total(NW * R * M + em) / (float)K + a.eps);
    const float y0 = total(er * M + em) * scale;
    const float y1 = NW == 2 ? total((R + er) * M + em) * scale : 0.f;
    epi_store<MODE>(a, epi, eu, em, y0, y1);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kMfmaRows = 16;     // activation rows per matrix-core launch
constexpr int kChunkK = 128;      // k per wavefront chunk (4 MFMA k steps of 32)

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4 &v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// One workgroup: units 4 UW blockIdx.x .. + 4 UW - 1 (wavefront w: UW <= 16 of them, the MFMA's
// other B columns unused) for up to 16 activation rows.  SPLIT: k chunks [blockIdx.y * cps,
// (blockIdx.y + 1) * cps) only, partial products and sums of squares to the workspace
// [split][w][m][units], [split][m].  LDS: 80 KB with two weight rows per unit (two workgroups per
// compute unit), 48 KB with one (three).
template <int MODE, bool SPLIT, int UW>
__global__ __launch_bounds__(256) void gemv_mfma_kernel(GemvArgs a, int cps) {
    static_assert(UW % 2 == 0 && UW >= 2 && UW <= 16, "units per wavefront: an even number up to 16");
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    // wavefront B tiles of a chunk pair: [wave][matrix][chunk], row r, k segment s at 16 r + (s ^ r)
    __shared__ uint4 bt[kWaves][NW][2][256];
    __shared__ uint4 at[2][4][2][64];       // A fragments [chunk][k step][hi, lo][lane]
    float *const ssp = reinterpret_cast<float *>(&at[0][0][0][0]);   // [wave][lane], after the k loop
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int units = n_units<MODE>(a);
    const int u0 = blockIdx.x * 4 * UW + UW * wave;
    const int K = a.K, chunks = K / kChunkK, rows = a.rows;
    const int c_beg = SPLIT ? blockIdx.y * cps : 0;
    const int c_end = SPLIT ? min(c_beg + cps, chunks) : chunks;

    // load instruction i < UW / 2 of matrix w: lane l reads row 2 i + l / 32 of the block, 16-byte k
    // segment l % 16 of chunk (l / 16) % 2 of the pair, i.e. 512 contiguous bytes per row; rows
    // past the last unit are clamped to it, and a missing second chunk of a range to its first
    // (in bounds, results dropped)
    const int pr = lane >> 5, ph = (lane >> 4) & 1, ps = lane & 15;
    const int lr = lane >> 4, lk = lane & 15;
    const uint16_t *wp[NW][8];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int i = 0; i < 8; ++i) wp[w][i] = unit_row<MODE>(a, min(u0 + 2 * i + pr, units - 1), w) + 8 * ps;
    // this thread's A fragments: k step `wave` of each chunk, lane `lane` (row l % 16, k 8 (l / 16))
    const int am = lane & 15, ak = 32 * wave + 8 * (lane >> 4);
    const bool avalid = am < rows;
    const float *xp = a.act + (size_t)(avalid ? am : 0) * a.act_ld + ak;
    const uint16_t *gp = a.gain + ak;

    f32x4 d[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) d[w] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;

    struct Pair {
        uint4 w[NW][8];
        float4 x[2][2];
        uint4 g[2];
    };
    auto load = [&](int c, Pair &b) {
        const int kc = kChunkK * min(c + ph, c_end - 1);
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (2 * i < UW) b.w[w][i] = load_stream16(wp[w][i] + kc);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int k = kChunkK * min(c + h, c_end - 1);
            b.x[h][0] = *reinterpret_cast<const float4 *>(xp + k);
            b.x[h][1] = *reinterpret_cast<const float4 *>(xp + k + 4);
            if (kNorm) b.g[h] = *reinterpret_cast<const uint4 *>(gp + k);
        }
    };
    auto convert = [&](const Pair &b, int h) {
        const float x[8] = {b.x[h][0].x, b.x[h][0].y, b.x[h][0].z, b.x[h][0].w,
                            b.x[h][1].x, b.x[h][1].y, b.x[h][1].z, b.x[h][1].w};
        float g[8];
        if (kNorm) unpack8(b.g[h], g);
        bf16x8 xh, xl;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float v = avalid ? x[j] : 0.f;
            if (kNorm) {
                ss = fmaf(v, v, ss);
                v = v * g[j];
            }
            xh[j] = (__bf16)v;                       // nearest even
            xl[j] = (__bf16)(v - (float)xh[j]);
        }
        uint4 h4, l4;
        __builtin_memcpy(&h4, &xh, 16);
        __builtin_memcpy(&l4, &xl, 16);
        at[h][wave][0][lane] = h4;
        at[h][wave][1][lane] = l4;
    };
    auto multiply = [&](int h) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const bf16x8 ah = as_bf16x8(at[h][t][0][lane]);
            const bf16x8 al = as_bf16x8(at[h][t][1][lane]);
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const bf16x8 bw = as_bf16x8(bt[wave][w][h][16 * lk + ((4 * t + lr) ^ lk)]);
                d[w] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw, d[w], 0, 0, 0);
                d[w] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw, d[w], 0, 0, 0);
            }
        }
    };
    Pair b;
    if (c_beg < c_end) load(c_beg, b);
    for (int c = c_beg; c < c_end; c += 2) {
        const bool two = c + 1 < c_end;
        convert(b, 0);
        if (two) convert(b, 1);
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int r = 2 * i + pr;
                if (2 * i < UW) bt[wave][w][ph][16 * r + (ps ^ r)] = b.w[w][i];
            }
        if (c + 2 < c_end) load(c + 2, b);
        // A tiles complete for every wavefront (each wavefront reads only its own B tiles)
        __syncthreads();
        multiply(0);
        if (two) multiply(1);
        // the A tiles and the sums-of-squares array are written next by other wavefronts
        __syncthreads();
    }

    // a row's sum of squares: 16 thread partials (4 k steps x 4 k blocks) in a fixed order
    if (kNorm) ssp[wave * 64 + lane] = ss;
    __syncthreads();
    auto row_ss = [&](int m) {
        float t = 0.f;
        for (int w = 0; w < kWaves; ++w)
            for (int q = 0; q < 4; ++q) t += ssp[w * 64 + 16 * q + m];
        return t;
    };
    if (SPLIT && kNorm && blockIdx.x == 0 && threadIdx.x < kMfmaRows)
        a.split_ss[blockIdx.y * kMfmaRows + threadIdx.x] = row_ss(threadIdx.x);
    // result register i of lane l: D[m = 4 (l / 16) + i][n = l % 16]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = 4 * lr + i, u = u0 + lk;
        if (m >= rows || lk >= UW || u >= units) continue;
        if (SPLIT) {
#pragma unroll
            for (int w = 0; w < NW; ++w)
                a.split_part[(((size_t)blockIdx.y * NW + w) * kMfmaRows + m) * units + u] = d[w][i];
            continue;
        }
        const float scale = kNorm ? 1.f / sqrtf(row_ss(m) / (float)K + a.eps) : 1.f;
        epi_store<MODE>(a, epi_load<MODE>(a, u, m), u, m, d[0][i] * scale, d[NW - 1][i] * scale);
    }
}

// Adds the k ranges of a split matrix-core launch in ascending order and applies the epilogue:
// one thread per (row, unit).  Every load (each range's partials and sums of squares, indices past
// the last range clamped to it, then the epilogue inputs) is issued before the first sum, so the
// partials cost one round trip to memory.
template <int MODE>
__global__ __launch_bounds__(256) void gemv_split_epilogue(GemvArgs a, int splits) {
    constexpr bool kNorm = Shape<MODE>::kNorm;
    constexpr int NW = Shape<MODE>::NW;
    const int units = n_units<MODE>(a);
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= a.rows * units) return;
    const int m = e / units, u = e % units;
    float p[NW][kGemvMaxSplits], q[kGemvMaxSplits];
#pragma unroll
    for (int sp = 0; sp < kGemvMaxSplits; ++sp) {
        const int c = min(sp, splits - 1);
#pragma unroll
        for (int w = 0; w < NW; ++w) p[w][sp] = a.split_part[(((size_t)c * NW + w) * kMfmaRows + m) * units + u];
        if (kNorm) q[sp] = a.split_ss[c * kMfmaRows + m];
    }
    const EpiIn epi = epi_load<MODE>(a, u, m);   // (RoPE/KV: dependent metadata loads, after the partials')
    float t[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        float acc = p[w][0];
#pragma unroll
        for (int sp = 1; sp < kGemvMaxSplits; ++sp) acc = sp < splits ? acc + p[w][sp] : acc;
        t[w] = acc;
    }
    float scale = 1.f;
    if (kNorm) {
        float sq = q[0];
#pragma unroll
        for (int sp = 1; sp < kGemvMaxSplits; ++sp) sq = sp < splits ? sq + q[sp] : sq;
        scale = 1.f / sqrtf(sq / (float)a.K + a.eps);
    }
    epi_store<MODE>(a, epi, u, m, t[0] * scale, t[NW - 1] * scale);
}

int host_units(int mode, const GemvArgs &a) { return mode == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N; }

// K ranges of whole chunk pairs, at most 8 and at most one per four chunks, as many as keep the
// grid within one even layer of workgroups: two per compute unit (512 on MI355X) with one weight
// row per unit, 7/6 per compute unit (298) with two, whose 80 KB of LDS leave room for two but
// whose split epilogue costs more than a second, partial layer gains.  Swept at 4, 8 and 16 rows on the
// 8B- and 70B-shaped layers (16 rows, with the epilogue): 70B gate/up unsplit (448 workgroups)
// 155 us against 165 with 4 ranges; 70B QKV 3 ranges 36.7 us, 4 ranges 44.6, 6 ranges 39.7; 70B
// down 4 ranges 78 us against 92 for 8 and 95 for 2; 70B O 4 ranges 28 us against 31 for 8; 8B
// gate/up unsplit 48.7 us against 52.1 with 2 ranges; 8B QKV 6 ranges 17.4 us against 18.1 for 4;
// 8B down and O 8 ranges.  Without a workspace, unsplit.
//
// An unsplit launch of the SwiGLU or residual form takes 14 units per wavefront instead of 16
// where that leaves the most loaded compute unit fewer units (ceil(workgroups / compute units) x
// units per wavefront): the 70B gate/up projection (F = 28672 = 7 x 2^12) then runs 512 workgroups, two on
// every compute unit, where 16 leaves 448 and a quarter of the compute units half idle (153 ->
// 143 us at 4 to 16 rows); the 8B one (F = 14336) 256 workgroups instead of 224 (48.5 -> 46.7
// us).  12 units per wavefront (597 and 299 workgroups) took 171 and 56 us.
bool fewer_units_per_wave(int units, int cus) {
    const long b16 = (units + 63) / 64, b14 = (units + 55) / 56;
    return (b14 + cus - 1) / cus * 14 < (b16 + cus - 1) / cus * 16;
}

template <int MODE>
void launch_mfma(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const int units = host_units(MODE, c), chunks = c.K / kChunkK;
    const int blocks = (units + 63) / 64;
    const int cus = device_compute_units();
    const int grid_max = Shape<MODE>::NW == 1 ? 2 * cus : cus * 7 / 6;
    int splits = max(1, min(min(kGemvMaxSplits, chunks / 4), grid_max / blocks));
    if (!c.split_part || !c.split_ss) splits = 1;
    if constexpr (MODE != GEMV_NORM_ROPE_KV) {
        if (splits == 1 && fewer_units_per_wave(units, cus)) {
            const dim3 grid((units + 55) / 56);
            if (e0 || e1)
                STG_EXT_LAUNCH((gemv_mfma_kernel<MODE, false, 14>), grid, dim3(256), 0, st, e0, e1, 0, c, 0);
            else
                STG_LAUNCH((gemv_mfma_kernel<MODE, false, 14>), grid, dim3(256), 0, st, c, 0);
            return;
        }
    }
    if (splits == 1) {
        if (e0 || e1)
            STG_EXT_LAUNCH((gemv_mfma_kernel<MODE, false, 16>), dim3(blocks), dim3(256), 0, st, e0, e1, 0, c, 0);
        else
            STG_LAUNCH((gemv_mfma_kernel<MODE, false, 16>), dim3(blocks), dim3(256), 0, st, c, 0);
        return;
    }
    const int cps = ((chunks + splits - 1) / splits + 1) & ~1;   // whole chunk pairs
    splits = (chunks + cps - 1) / cps;  // no empty range
    if (e0)
        STG_EXT_LAUNCH((gemv_mfma_kernel<MODE, true, 16>), dim3(blocks, splits), dim3(256), 0, st, e0, nullptr,
                              0, c, cps);
    else
        STG_LAUNCH((gemv_mfma_kernel<MODE, true, 16>), dim3(blocks, splits), dim3(256), 0, st, c, cps);
    const int eg = (c.rows * units + 255) / 256;
    if (e1)
        STG_EXT_LAUNCH((gemv_split_epilogue<MODE>), dim3(eg), dim3(256), 0, st, nullptr, e1, 0, c, splits);
    else
        STG_LAUNCH((gemv_split_epilogue<MODE>), dim3(eg), dim3(256), 0, st, c, splits);
}

template <int M, int R, int U, int MODE>
void launch_one(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const int grid = (host_units(MODE, c) + R - 1) / R;
    if (e0 || e1)
        STG_EXT_LAUNCH((gemv_kernel<M, R, U, MODE>), dim3(grid), dim3(256), 0, st, e0, e1, 0, c);
    else
        STG_LAUNCH((gemv_kernel<M, R, U, MODE>), dim3(grid), dim3(256), 0, st, c);
}

// Units per workgroup and steps in flight, by mode and rows (swept on the 8B- and 70B-shaped
// layers): one row: gate/up 4 units x 1 step, O 4 x 2, down (K >= 2N) and the 70B O projection
// 8 x 1 (70B down: 70.4 us against 75.4 us for 4 x 2; O: 23.9 against 24.6), QKV 2 x 1 (2 x 2 on
// the larger shape); two rows: O and down 4 x 1 (8 x 1 for the 70B down projection), QKV 4 x 1
// (2 x 1 on the larger shape); fewer as the rows multiply the registers.
template <int M, int MODE>
void launch_rows(const GemvArgs &c, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const long work = (long)host_units(MODE, c) * c.K;
    if (MODE == GEMV_PLAIN_RESIDUAL) {
        if (M == 1 && (c.K >= 2 * c.N || work >= 60L * 1000 * 1000)) launch_one<M, 8, 1, MODE>(c, st, e0, e1);
        else if (M == 1) launch_one<M, 4, 2, MODE>(c, st, e0, e1);
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
    // rows from which the matrix cores are faster (measured on the 8B- and 70B-shaped layers):
    // 3, except for square plain projections (the O projection), where the vector kernel keeps up
    // to 4 rows
    const int mfma_min_rows = MODE == GEMV_PLAIN_RESIDUAL && a.K <= a.N ? 5 : 3;
    for (int r0 = 0, n = 0; r0 < a.rows; r0 += n) {
        const int left = a.rows - r0;
        const bool mfma = mfma_ok && left >= mfma_min_rows;
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

// (256, the count of a whole MI355X, if the runtime cannot tell)
int device_compute_units() {
    constexpr int kDevices = 64;
    static std::atomic<int> cached[kDevices];
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) {
        (void)hipGetLastError();   // a failed query must not surface as a launch error
        return 256;
    }
    n = cached[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return 256;
    }
    cached[dev].store(n, std::memory_order_relaxed);
    return n;
}

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
