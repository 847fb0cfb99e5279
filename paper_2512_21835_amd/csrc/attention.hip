// Causal grouped-query attention over the paged KV cache, fp32 arithmetic.
//
// One workgroup handles one (row, KV head, key split): the G = Hq/Hkv query heads that share the
// KV head, over a range of keys.  Keys are walked in chunks of 64.  Inside a chunk, 128-bit loads
// fetch one K row per D/8 lanes (a 16-token block of one head is 4 KiB contiguous in the pool);
// the lanes of a key reduce their partial dot products with shuffles, scores go to LDS, one
// wavefront per head takes the chunk maximum and exponentials (online softmax across chunks), and
// the same lanes then accumulate P.V from V rows fetched the same way.
//
// Prefill (split_keys == 0): with a bf16 cache, attn_prefill_mfma runs the products on the matrix
// cores (flash-attention tiling, below); with an fp32 cache (the parity mode), attn_kernel: one
// workgroup per (row, KV head) walks all of the row's keys.  Decode (split_keys > 0): the context is
// cut into splits of split_keys keys so that one token's attention still fills the GPU, and a
// second launch (attn_merge) merges each row's splits.  With a bf16 cache and 128-wide heads the
// splits run on the matrix cores (attn_decode_mfma: the G query heads of a KV head are the N
// dimension of S^T = K Q^T, then O = P V; with G = 8 the vector form spends 16 multiply-adds per
// cached element and is bound by them); otherwise attn_decode_kernel.
#include <hip/hip_runtime.h>

#include "lanes.h"
#include "pair.h"
#include "stage_kernels.h"

namespace stg {
namespace {

constexpr int kChunk = 64;
constexpr int kMaxDecodeSplits = 256;  // splits one row may have (max_context / split_keys)

__device__ __forceinline__ float bf16lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

template <bool F32KV>
__device__ __forceinline__ void load8(const void *pool, size_t elem, float f[8]) {
    if (F32KV) {
        const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(pool) + elem);
        const float4 a = p[0], b = p[1];
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
        f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    } else {
        const uint4 v = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(pool) + elem);
        f[0] = bf16lo(v.x); f[1] = bf16hi(v.x);
        f[2] = bf16lo(v.y); f[3] = bf16hi(v.y);
        f[4] = bf16lo(v.z); f[5] = bf16hi(v.z);
        f[6] = bf16lo(v.w); f[7] = bf16hi(v.w);
    }
}

template <int G, int D>
struct DecodeSmem {
    float wm[4][G], wl[4][G];
    float o[4][G][D];
};

// Decode: one workgroup per (key split, KV head, row); a split holds at most kChunk keys.  K and V
// of the lane's keys are fetched together up front, scores are reduced across the D/8 lanes of a
// key, the split's maximum and sum across the workgroup through LDS once, and the partial output
// (unnormalised, with its max and sum) goes to global memory for attn_merge.  FINAL (every
// row of the call within one split): the output o / l directly, the value the merge would compute
// from the single split (weight exp(m - m) = 1), so no merge launch follows.
template <int G, int D, bool F32KV, bool FINAL>
__device__ __forceinline__ void attn_decode_task(const AttnArgs &a, int split, int g, int row,
                                                 DecodeSmem<G, D> &sm) {
    constexpr int LPK = D / 8;
    constexpr int KPW = 64 / LPK;
    constexpr int KPS = 4 * KPW;
    constexpr int STEPS = kChunk / KPS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kl = lane / LPK, sub = lane % LPK, c0 = sub * 8;
    const int hq_total = a.n_q_heads;
    const size_t q_ld = (size_t)hq_total * D;
    // the queries first: they depend on the row only
    const float scale = 1.f / sqrtf((float)D);
    float q[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float *qp = a.q + row * q_ld + (size_t)(g * G + h) * D + c0;
#pragma unroll
        for (int j = 0; j < 8; ++j) q[h][j] = qp[j] * scale;
    }
    const int sidx = row / a.rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.rows_per_seq;
    const int slot = a.meta->seq_slot[sidx];
    const int ctx = pos + 1;
    const int kbeg = split * a.split_keys;
    if (kbeg >= ctx || slot < 0) return;  // (slot tested so that both metadata loads go out together)
    const int n = min(a.split_keys, ctx - kbeg);

    const int hkv = a.kv.n_kv_heads;
    const int *table = a.kv.block_table + (size_t)slot * a.kv.max_blocks;
    const size_t blk_stride = (size_t)2 * hkv * kBlockTokens * D;

    // keys of this lane: kk = st * KPS + wave * KPW + kl.  Slots past the split's last key load that
    // key again (in bounds; their scores are masked below), so that the loads carry no branches and
    // all block-table loads, then all K/V loads, are in flight together: two round trips in all.
    int blk[STEPS];
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const int key = kbeg + min(st * KPS + wave * KPW + kl, n - 1);
        blk[st] = table[key / kBlockTokens];
    }
    float kf[STEPS][8], vf[STEPS][8];
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const int key = kbeg + min(st * KPS + wave * KPW + kl, n - 1);
        const size_t e = (size_t)blk[st] * blk_stride + ((size_t)g * kBlockTokens + key % kBlockTokens) * D + c0;
        load8<F32KV>(a.kv.pool, e, kf[st]);
        load8<F32KV>(a.kv.pool, e + (size_t)hkv * kBlockTokens * D, vf[st]);
    }
    __builtin_amdgcn_sched_barrier(0);  // every K and V load in flight before any is used

    float sc[STEPS][G];
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const bool valid = st * KPS + wave * KPW + kl < n;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float p = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) p = fmaf(q[h][j], kf[st][j], p);
#pragma unroll
            for (int o2 = LPK / 2; o2 >= 1; o2 >>= 1) p += lane_xor(p, o2);
            sc[st][h] = valid ? p : -INFINITY;
        }
    }
    // split maximum per head
#pragma unroll
    for (int h = 0; h < G; ++h) {
        float m = sc[0][h];
#pragma unroll
        for (int st = 1; st < STEPS; ++st) m = fmaxf(m, sc[st][h]);
#pragma unroll
        for (int o2 = 32; o2 >= LPK; o2 >>= 1) m = fmaxf(m, lane_xor(m, o2));
        if (lane == 0) sm.wm[wave][h] = m;
    }
    __syncthreads();
    float mh[G];
#pragma unroll
    for (int h = 0; h < G; ++h) mh[h] = fmaxf(fmaxf(sm.wm[0][h], sm.wm[1][h]), fmaxf(sm.wm[2][h], sm.wm[3][h]));

    float l[G], o[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        l[h] = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[h][j] = 0.f;
    }
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float p = sc[st][h] == -INFINITY ? 0.f : expf(sc[st][h] - mh[h]);
            l[h] += p;
#pragma unroll
            for (int j = 0; j < 8; ++j) o[h][j] = fmaf(p, vf[st][j], o[h][j]);
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
        for (int o2 = 32; o2 >= LPK; o2 >>= 1) l[h] += lane_xor(l[h], o2);
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int o2 = 32; o2 >= LPK; o2 >>= 1)   // G >= 8: the VALU is the bound, the LDS crossbar is idle
                o[h][j] += G >= 8 ? __shfl_xor(o[h][j], o2, 64) : lane_xor(o[h][j], o2);
    }
    if (kl == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int j = 0; j < 8; ++j) sm.o[wave][h][c0 + j] = o[h][j];
    }
    if (lane == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) sm.wl[wave][h] = l[h];
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, c = i % D;
        if (FINAL) {
            const float o_sum = ((sm.o[0][h][c] + sm.o[1][h][c]) + sm.o[2][h][c]) + sm.o[3][h][c];
            const float l_sum = ((sm.wl[0][h] + sm.wl[1][h]) + sm.wl[2][h]) + sm.wl[3][h];
            a.out[row * q_ld + (size_t)(g * G + h) * D + c] = o_sum / l_sum;
            continue;
        }
        const size_t pi = ((size_t)row * hq_total + g * G + h) * a.max_splits + split;
        a.part_o[pi * D + c] = ((sm.o[0][h][c] + sm.o[1][h][c]) + sm.o[2][h][c]) + sm.o[3][h][c];
        if (c == 0) {
            a.part_ml[pi * 2 + 0] = fmaxf(fmaxf(sm.wm[0][h], sm.wm[1][h]), fmaxf(sm.wm[2][h], sm.wm[3][h]));
            a.part_ml[pi * 2 + 1] = ((sm.wl[0][h] + sm.wl[1][h]) + sm.wl[2][h]) + sm.wl[3][h];
        }
    }
}


template <int G, int D, bool F32KV>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    constexpr int LPK = D / 8;        // lanes per key row
    constexpr int KPW = 64 / LPK;     // keys per wavefront per step
    constexpr int KPS = 4 * KPW;      // keys per workgroup per step
    static_assert(kChunk % KPS == 0, "chunk must be a multiple of keys per step");
    const int g = blockIdx.y, row = blockIdx.z;
    const int sidx = row / a.meta->rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.meta->rows_per_seq;
    const int slot = a.meta->seq_slot[sidx];
    const int ctx = pos + 1;
    const int kbeg = 0, kend = ctx;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kl = lane / LPK;        // key slot of this lane within the wavefront step
    const int sub = lane % LPK;
    const int c0 = sub * 8;
    const int hq_total = a.n_q_heads;
    const size_t q_ld = (size_t)hq_total * D;
    const int hkv = a.kv.n_kv_heads;
    const int *table = a.kv.block_table + (size_t)slot * a.kv.max_blocks;
    const size_t blk_stride = (size_t)2 * hkv * kBlockTokens * D;

    __shared__ float s_p[G][kChunk];
    __shared__ float s_m[G], s_l[G], s_alpha[G];
    __shared__ float s_o[4][G][D];

    const float scale = 1.f / sqrtf((float)D);
    float q[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float *qp = a.q + row * q_ld + (size_t)(g * G + h) * D + c0;
#pragma unroll
        for (int j = 0; j < 8; ++j) q[h][j] = qp[j] * scale;
    }
    if (tid < G) { s_m[tid] = -INFINITY; s_l[tid] = 0.f; }
    float o[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int j = 0; j < 8; ++j) o[h][j] = 0.f;
    __syncthreads();

    for (int kc = kbeg; kc < kend; kc += kChunk) {
        const int n = min(kChunk, kend - kc);
        // scores of this chunk
        for (int base = 0; base < kChunk; base += KPS) {
            const int kk = base + wave * KPW + kl;
            float part[G];
#pragma unroll
            for (int h = 0; h < G; ++h) part[h] = 0.f;
            if (kk < n) {
                const int key = kc + kk;
                const size_t e = (size_t)table[key / kBlockTokens] * blk_stride +
                                 ((size_t)g * kBlockTokens + key % kBlockTokens) * D + c0;
                float kf[8];
                load8<F32KV>(a.kv.pool, e, kf);
#pragma unroll
                for (int h = 0; h < G; ++h)
#pragma unroll
                    for (int j = 0; j < 8; ++j) part[h] = fmaf(q[h][j], kf[j], part[h]);
            }
#pragma unroll
            for (int h = 0; h < G; ++h)
#pragma unroll
                for (int o2 = LPK / 2; o2 >= 1; o2 >>= 1) part[h] += lane_xor(part[h], o2);
            if (kk < n && sub == 0) {
#pragma unroll
                for (int h = 0; h < G; ++h) s_p[h][kk] = part[h];
            }
        }
        __syncthreads();
        // online softmax update, one wavefront per head
        for (int h = wave; h < G; h += 4) {
            const float sv = lane < n ? s_p[h][lane] : -INFINITY;
            float mx = sv;
#pragma unroll
            for (int o2 = 32; o2 >= 1; o2 >>= 1) mx = fmaxf(mx, lane_xor(mx, o2));
            const float m_old = s_m[h];
            const float m_new = fmaxf(m_old, mx);
            const float p = lane < n ? expf(sv - m_new) : 0.f;
            float sum = p;
#pragma unroll
            for (int o2 = 32; o2 >= 1; o2 >>= 1) sum += lane_xor(sum, o2);
            s_p[h][lane] = p;
            if (lane == 0) {
                const float alpha = expf(m_old - m_new);  // 0 on the first chunk (m_old = -inf)
                s_alpha[h] = alpha;
                s_l[h] = s_l[h] * alpha + sum;
                s_m[h] = m_new;
            }
        }
        __syncthreads();
        // P.V
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float al = s_alpha[h];
#pragma unroll
            for (int j = 0; j < 8; ++j) o[h][j] *= al;
        }
        for (int base = 0; base < kChunk; base += KPS) {
            const int kk = base + wave * KPW + kl;
            if (kk < n) {
                const int key = kc + kk;
                const size_t e = (size_t)table[key / kBlockTokens] * blk_stride +
                                 ((size_t)(hkv + g) * kBlockTokens + key % kBlockTokens) * D + c0;
                float vf[8];
                load8<F32KV>(a.kv.pool, e, vf);
#pragma unroll
                for (int h = 0; h < G; ++h) {
                    const float p = s_p[h][kk];
#pragma unroll
                    for (int j = 0; j < 8; ++j) o[h][j] = fmaf(p, vf[j], o[h][j]);
                }
            }
        }
        __syncthreads();
    }

    // reduce the key slots: lanes with equal `sub` inside a wavefront, then across wavefronts
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int o2 = 32; o2 >= LPK; o2 >>= 1) o[h][j] += lane_xor(o[h][j], o2);
    if (kl == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int j = 0; j < 8; ++j) s_o[wave][h][c0 + j] = o[h][j];
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, c = i % D;
        const float v = ((s_o[0][h][c] + s_o[1][h][c]) + s_o[2][h][c]) + s_o[3][h][c];
        a.out[row * q_ld + (size_t)(g * G + h) * D + c] = v / s_l[h];
    }
}

template <int G, int D, bool F32KV, bool FINAL>
__global__ __launch_bounds__(256) void attn_decode_kernel(AttnArgs a) {
    __shared__ DecodeSmem<G, D> sm;
    attn_decode_task<G, D, F32KV, FINAL>(a, blockIdx.x, blockIdx.y, blockIdx.z, sm);
}

// Merge of the decode splits: one workgroup per (row, query head).  Thread t owns the 4 output
// columns 4 (t % (D/4)) .. + 3 and the splits s with s % SL == t / (D/4) (SL = 1024 / D split
// lanes: 8 for 128-wide heads, 16 for 64-wide).  Per round of kMergePer splits per lane it issues
// the loads of all of them at once (addresses clamped to the call's longest row, a.grid_splits),
// before the row's own split count arrives from the metadata: one round trip for contexts up to
// kMergePer * SL splits.  A lane merges its splits in ascending order (online: rescaled to the
// running maximum; weight exp(m_s - max)); the SL lane states then meet in LDS and are added in
// lane order.  The order depends on the row's split count only, never on the other rows of the
// call; for a single split the result is exactly o / l (weights exp(0) = 1, empty lanes add 0).
constexpr int kMergePer = 8;
template <int D>
__global__ __launch_bounds__(256) void attn_merge(AttnArgs a) {
    constexpr int CG = D / 4, SL = 256 / CG;
    __shared__ float s_m[SL][CG], s_l[SL][CG];
    __shared__ float4 s_o[SL][CG];
    const int cg = threadIdx.x % CG, sl = threadIdx.x / CG;
    const int hq = blockIdx.x, row = blockIdx.y, hq_total = a.n_q_heads;
    const size_t pi0 = ((size_t)row * hq_total + hq) * a.max_splits;
    const float2 *ml = reinterpret_cast<const float2 *>(a.part_ml) + pi0;
    const float4 *po = reinterpret_cast<const float4 *>(a.part_o + pi0 * D) + cg;
    const int lim = a.grid_splits;
    float mx = -INFINITY, den = 0.f;
    float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
    int nsp = -1;
    for (int s0 = 0; s0 < lim; s0 += kMergePer * SL) {
        const int nper = min(kMergePer, (lim - s0 + SL - 1) / SL);  // same for every thread
        float2 v[kMergePer];
        float4 o[kMergePer];
#pragma unroll
        for (int j = 0; j < kMergePer; ++j)
            if (j < nper) {
                const int s = min(s0 + j * SL + sl, lim - 1);
                v[j] = ml[s];
                o[j] = po[(size_t)s * (D / 4)];
            }
        if (nsp < 0) {
            const int sidx = row / a.rows_per_seq;
            const int ctx = a.meta->pos0[sidx] + row % a.rows_per_seq + 1;
            nsp = min((ctx + a.split_keys - 1) / a.split_keys, lim);
        }
        if (s0 >= nsp) break;
        float m = mx;
#pragma unroll
        for (int j = 0; j < kMergePer; ++j)
            if (j < nper && s0 + j * SL + sl < nsp) m = fmaxf(m, v[j].x);
        if (m > -INFINITY) {  // this lane holds a split of the row
            const float r = expf(mx - m);  // 0 on the lane's first split (mx = -inf)
            den *= r;
            num.x *= r;
            num.y *= r;
            num.z *= r;
            num.w *= r;
#pragma unroll
            for (int j = 0; j < kMergePer; ++j)
                if (j < nper && s0 + j * SL + sl < nsp) {
                    const float w = expf(v[j].x - m);
                    den = fmaf(w, v[j].y, den);
                    num.x = fmaf(w, o[j].x, num.x);
                    num.y = fmaf(w, o[j].y, num.y);
                    num.z = fmaf(w, o[j].z, num.z);
                    num.w = fmaf(w, o[j].w, num.w);
                }
            mx = m;
        }
    }
    s_m[sl][cg] = mx;
    s_l[sl][cg] = den;
    s_o[sl][cg] = num;
    __syncthreads();
    if (sl != 0) return;
    float M = -INFINITY;
#pragma unroll
    for (int i = 0; i < SL; ++i) M = fmaxf(M, s_m[i][cg]);
    float L = 0.f;
    float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int i = 0; i < SL; ++i) {
        const float mi = s_m[i][cg];
        if (mi > -INFINITY) {
            const float w = expf(mi - M);
            const float4 oi = s_o[i][cg];
            L = fmaf(w, s_l[i][cg], L);
            O.x = fmaf(w, oi.x, O.x);
            O.y = fmaf(w, oi.y, O.y);
            O.z = fmaf(w, oi.z, O.z);
            O.w = fmaf(w, oi.w, O.w);
        }
    }
    *reinterpret_cast<float4 *>(a.out + (size_t)row * hq_total * D + (size_t)hq * D + 4 * cg) =
        make_float4(O.x / L, O.y / L, O.z / L, O.w / L);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8_t as_bf(uint4 v) {
    bf16x8_t r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}
// x as an exact-sum pair of bf16 vectors: hi = bf16(x), lo = bf16(x - hi), both nearest even.
__device__ __forceinline__ void split8(const float *x, bf16x8_t &hi, bf16x8_t &lo) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        hi[j] = (__bf16)x[j];                   // v_cvt_pk_bf16_f32: nearest even
        lo[j] = (__bf16)(x[j] - (float)hi[j]);
    }
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));
// Decode attention of one (64-key split, KV head g, row) on the matrix cores (bf16 KV, D = 128,
// G <= 16): S^T = K Q^T with the K rows of the split's cache blocks as the A operand (one 16-key
// block per wavefront) and Q as a bf16 hi/lo pair; softmax statistics per head from the MFMA
// layout; O = P V with P (hi/lo) from LDS and V read transposed from an LDS tile.  Partial
// outputs as attn_decode_task writes them, or with FINAL the output o / l.
template <int G, int D, bool FINAL>
__global__ __launch_bounds__(256) void attn_decode_mfma(AttnArgs a) {
    static_assert(D == 128 && G <= 16, "one 128-wide head, up to 16 query heads per KV head");
    constexpr int VROW = D + 8;                     // V tile row stride in bf16 (272 bytes)
    // one LDS area for the K tile (until the first barrier: each wavefront reads only its own 16
    // keys) and then the V tile
    __shared__ uint4 kv_tile[kChunk * VROW * 2 / 16];
    uint4 (*const ks)[D / 8] = reinterpret_cast<uint4 (*)[D / 8]>(kv_tile);    // [key][chunk ^ key % 16]
    uint16_t (*const vs)[VROW] = reinterpret_cast<uint16_t (*)[VROW]>(kv_tile);
    __shared__ uint4 pf[2][2][64];                  // P A-fragments [key step][hi, lo][lane]
    __shared__ float wm[4][16], wl[4][16];
    const int split = blockIdx.x, g = blockIdx.y, row = blockIdx.z;
    const int lane = threadIdx.x & 63, l16 = lane & 15, lq = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int hq_total = a.n_q_heads, hkv = a.kv.n_kv_heads;
    // Q^T fragments first (they depend on the row only): head l16 (heads past G load head G - 1 and
    // are zeroed below), d 32 s + 8 lq
    const float *qp = a.q + (size_t)row * hq_total * D + (size_t)(g * G + min(l16, G - 1)) * D + 8 * lq;
    float4 qv[4][2];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        qv[s][0] = *reinterpret_cast<const float4 *>(qp + 32 * s);
        qv[s][1] = *reinterpret_cast<const float4 *>(qp + 32 * s + 4);
    }
    const int sidx = row / a.rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.rows_per_seq;
    const int slot = a.meta->seq_slot[sidx];
    const int ctx = pos + 1, kbeg = split * a.split_keys;
    if (kbeg >= ctx || slot < 0) return;  // (slot tested so that both metadata loads go out together)
    const int n = min(a.split_keys, ctx - kbeg);
    const size_t blk_stride = (size_t)2 * hkv * kBlockTokens * D;
    const uint16_t *pool = static_cast<const uint16_t *>(a.kv.pool);
    // every key of wavefront w (16 w .. 16 w + 15 of the split, clamped into it) lies in one cache
    // block (splits start on a block boundary): one block-table entry per wavefront
    const int blk = a.kv.block_table[(size_t)slot * a.kv.max_blocks + (kbeg + min(16 * wave, n - 1)) / kBlockTokens];
    const uint16_t *kb = pool + (size_t)blk * blk_stride + (size_t)g * kBlockTokens * D;
    const uint16_t *vb = pool + (size_t)blk * blk_stride + (size_t)(hkv + g) * kBlockTokens * D;
    // K and V rows, 4 keys x 256 contiguous bytes per load instruction (16 keys x 64 bytes, the
    // MFMA fragment layout read straight from memory, streams poorly): instruction i, lane l: key
    // 16 wave + 4 i + lq of the split (clamped into it); K: 16-byte d chunk l16 ^ (4 i + lq),
    // stored in the K tile at [key][l16]; V: chunk l16
    auto krow = [&](int i) {
        const int key = kbeg + min(16 * wave + 4 * i + lq, n - 1);
        return *reinterpret_cast<const uint4 *>(kb + (size_t)(key % kBlockTokens) * D + 8 * (l16 ^ (4 * i + lq)));
    };
    auto vrow = [&](int i) {
        const int key = kbeg + min(16 * wave + 4 * i + lq, n - 1);
        return *reinterpret_cast<const uint4 *>(vb + (size_t)(key % kBlockTokens) * D + 8 * l16);
    };
    const uint4 kr0 = krow(0), kr1 = krow(1), kr2 = krow(2), kr3 = krow(3);
    const uint4 vr0 = vrow(0), vr1 = vrow(1), vr2 = vrow(2), vr3 = vrow(3);
    // every K and V load in flight before any is used (left alone, the scheduler issues half of
    // them after the first products, a second round trip to memory)
    __builtin_amdgcn_sched_barrier(0);
    // Q^T as a bf16 hi/lo pair, scaled by 1/sqrt(d)
    const float scale = 1.f / sqrtf((float)D);
    bf16x8_t qh[4], ql[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const float q8[8] = {qv[s][0].x, qv[s][0].y, qv[s][0].z, qv[s][0].w,
                             qv[s][1].x, qv[s][1].y, qv[s][1].z, qv[s][1].w};
        float x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = l16 < G ? q8[j] * scale : 0.f;
        split8(x, qh[s], ql[s]);
    }
    ks[16 * wave + lq][l16] = kr0;
    ks[16 * wave + 4 + lq][l16] = kr1;
    ks[16 * wave + 8 + lq][l16] = kr2;
    ks[16 * wave + 12 + lq][l16] = kr3;
    // K fragments: key 16 wave + l16, d 32 s + 8 lq, i.e. chunk 4 s + lq (the tile holds chunk c of
    // key k at c ^ k % 16: every 16 lanes of a read meet distinct banks)
    f32x4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const bf16x8_t kf = as_bf(ks[16 * wave + l16][(4 * s + lq) ^ l16]);
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qh[s], sc, 0, 0, 0);
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, ql[s], sc, 0, 0, 0);
    }
    // sc[i]: score of key 16 wave + 4 lq + i for head l16
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (16 * wave + 4 * lq + i >= n) sc[i] = -INFINITY;
        mx = fmaxf(mx, sc[i]);
    }
    mx = fmaxf(mx, lane_xor(mx, 16));
    mx = fmaxf(mx, lane_xor(mx, 32));
    if (lane < 16) wm[wave][lane] = mx;
    __syncthreads();   // every wavefront's K reads done: the tile takes V
    *reinterpret_cast<uint4 *>(&vs[16 * wave + lq][8 * l16]) = vr0;
    *reinterpret_cast<uint4 *>(&vs[16 * wave + 4 + lq][8 * l16]) = vr1;
    *reinterpret_cast<uint4 *>(&vs[16 * wave + 8 + lq][8 * l16]) = vr2;
    *reinterpret_cast<uint4 *>(&vs[16 * wave + 12 + lq][8 * l16]) = vr3;
    const float mh = fmaxf(fmaxf(wm[0][l16], wm[1][l16]), fmaxf(wm[2][l16], wm[3][l16]));
    float p[4], ls = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        p[i] = sc[i] == -INFINITY ? 0.f : expf(sc[i] - mh);
        ls += p[i];
    }
    ls += lane_xor(ls, 16);
    ls += lane_xor(ls, 32);
    if (lane < 16) wl[wave][lane] = ls;
    // P fragment slot of key 16 wave + 4 lq + i: key step wave / 2, lane l16 + 16 (2 (wave % 2) + lq / 2),
    // elements 4 (lq % 2) + i
    {
        uint16_t hb[4], lb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const __bf16 h = (__bf16)p[i];
            const __bf16 l = (__bf16)(p[i] - (float)h);
            hb[i] = __builtin_bit_cast(uint16_t, h);
            lb[i] = __builtin_bit_cast(uint16_t, l);
        }
        const int L = l16 + 16 * (2 * (wave & 1) + (lq >> 1));
        uint2 h2 = make_uint2(hb[0] | ((uint32_t)hb[1] << 16), hb[2] | ((uint32_t)hb[3] << 16));
        uint2 l2 = make_uint2(lb[0] | ((uint32_t)lb[1] << 16), lb[2] | ((uint32_t)lb[3] << 16));
        reinterpret_cast<uint2 *>(&pf[wave >> 1][0][L])[lq & 1] = h2;
        reinterpret_cast<uint2 *>(&pf[wave >> 1][1][L])[lq & 1] = l2;
    }
    __syncthreads();
    // O block (heads 0..15) x (d 32 wave + 16 nb .. + 15), K = the split's 64 keys in two steps
    f32x4_t o[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t ph = as_bf(pf[ks][0][lane]), pl = as_bf(pf[ks][1][lane]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            const int d = 32 * wave + 16 * nb + l16;
            bf16x8_t vb;
#pragma unroll
            for (int j = 0; j < 8; ++j) vb[j] = __builtin_bit_cast(__bf16, vs[32 * ks + 8 * lq + j][d]);
            o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vb, o[nb], 0, 0, 0);
            o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vb, o[nb], 0, 0, 0);
        }
    }
    // o[nb][i]: head 4 lq + i, d 32 wave + 16 nb + l16
    if (FINAL) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int h = 4 * lq + i;
            if (h >= G) continue;
            const float l_sum = ((wl[0][h] + wl[1][h]) + wl[2][h]) + wl[3][h];
            float *op = a.out + (size_t)row * hq_total * D + (size_t)(g * G + h) * D;
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) op[32 * wave + 16 * nb + l16] = o[nb][i] / l_sum;
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = 4 * lq + i;
        if (h >= G) continue;
        const size_t pi = ((size_t)row * hq_total + g * G + h) * a.max_splits + split;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) a.part_o[pi * D + 32 * wave + 16 * nb + l16] = o[nb][i];
    }
    if (wave == 0 && lane < G) {
        const size_t pi = ((size_t)row * hq_total + g * G + lane) * a.max_splits + split;
        a.part_ml[pi * 2 + 0] = fmaxf(fmaxf(wm[0][lane], wm[1][lane]), fmaxf(wm[2][lane], wm[3][lane]));
        a.part_ml[pi * 2 + 1] = ((wl[0][lane] + wl[1][lane]) + wl[2][lane]) + wl[3][lane];
    }
}

constexpr int KT = 32;                 // keys per tile of the prefill kernel
constexpr int VROW = KT + 8;           // transposed V tile row stride in bf16 (padding)

// One workgroup: 128 query rows = G heads x (128 / G) consecutive positions of one sequence, one
// KV head.  Wave w owns rows 32 w .. 32 w + 31 (row r: head r / BQ, position offset r % BQ).
// Per 32-key tile: S^T = K Q^T (lane = one query column, 16 keys), online softmax in-lane,
// O^T += V^T P^T with V transposed in LDS.  q and p enter the MFMAs as bf16 hi + lo pairs.
// Bounded to two wavefronts per SIMD (205 registers): left to itself the compiler takes 276 (the
// O^T and S^T accumulators in AGPRs), which admits one, and a tile's dependent MFMA chain and
// softmax then run with nothing to overlap them.
template <int G, int D>
__global__ __launch_bounds__(256, 2) void attn_prefill_mfma(AttnArgs a) {
    constexpr int KROW = D + 8;         // K tile row stride in bf16 (padding)
    constexpr int BQ = 128 / G;
    constexpr int KK = D / 16;          // k16 steps over d
    constexpr int NB = D / 32;          // 32-row blocks of d in O^T
    __shared__ uint16_t sk[KT * KROW];
    __shared__ uint16_t sv[D * VROW];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5, col = lane & 31;
    const int qb = gridDim.x - 1 - blockIdx.x, g = blockIdx.y, sidx = blockIdx.z;  // longest first
    const int T = a.meta->rows_per_seq;
    const int pos0 = a.meta->pos0[sidx], slot = a.meta->seq_slot[sidx];
    const int hkv = a.kv.n_kv_heads, hq_total = a.n_q_heads;
    const size_t q_ld = (size_t)hq_total * D;
    const int *table = a.kv.block_table + (size_t)slot * a.kv.max_blocks;
    const uint16_t *pool = static_cast<const uint16_t *>(a.kv.pool);
    const size_t blk_stride = (size_t)2 * hkv * kBlockTokens * D;

    // this lane's query (column) and its position
    const int r = wave * 32 + col, hh = r / BQ, t = qb * BQ + r % BQ;
    const bool qvalid = t < T;
    const int qpos = pos0 + (qvalid ? t : T - 1);
    const size_t qrow = (size_t)(sidx * T + (qvalid ? t : T - 1));
    // Q^T fragments: B[k = d 16 kk + 8 half + j][query col]
    bf16x8_t qh[KK], ql[KK];
    {
        const float scale = 1.4426950408889634f / sqrtf((float)D);   // log2(e) / sqrt(d): scores in base 2
        const float *qp = a.q + qrow * q_ld + (size_t)(g * G + hh) * D + 8 * half;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            float x[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = qp[16 * kk + j] * scale;
            split8(x, qh[kk], ql[kk]);
        }
    }
    f32x16_t o[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[b][i] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    const int last_t = min(T, (qb + 1) * BQ) - 1;
    const int n_keys = pos0 + last_t + 1;
    const int n_tiles = (n_keys + KT - 1) / KT;
    // wave's largest query position (tiles past it are fully masked for the wave)
    int wave_max = 0;
    {
        const int r_lo = wave * 32, r_hi = wave * 32 + 31;
        for (int rr = r_lo; rr <= r_hi; rr += 1) {
            const int tt = qb * BQ + rr % BQ;
            if (tt < T) wave_max = max(wave_max, pos0 + tt);
        }
    }

    // tile loads: 32 keys x (D / 8) 16-byte chunks (512 for D = 128), PER_T per thread; chunk
    // c = tid + 256 i.  K: key c / (D / 8), d chunk c % (D / 8) (a wavefront reads 4 whole key
    // rows).  V: key c % 32, d chunk c / 32, so that one transposed store instruction writes 32
    // consecutive keys of one V^T row (the K mapping would put a wavefront's 16 rows 8 apart: on
    // two LDS bank offsets)
    constexpr int CHUNKS = KT * D / 8;          // 16-byte chunks per K (or V) tile
    constexpr int PER_T = CHUNKS / 256;         // per thread (2 for D = 128, 1 for D = 64)
    uint4 kr0, kr1, vr0, vr1;
#define STG_GLOAD(TILE, I, KR, VR)                                                                        \
    do {                                                                                                  \
        const int c_ = tid + 256 * (I);                                                                   \
        const int kp_ = min((TILE) * KT + c_ / (D / 8), n_keys - 1);                                      \
        const size_t b_ = (size_t)table[kp_ / kBlockTokens] * blk_stride +                                \
                          (size_t)(kp_ % kBlockTokens) * D + (c_ % (D / 8)) * 8;                          \
        KR = *reinterpret_cast<const uint4 *>(pool + b_ + (size_t)g * kBlockTokens * D);                 \
        const int vp_ = min((TILE) * KT + c_ % KT, n_keys - 1);                                           \
        const size_t v_ = (size_t)table[vp_ / kBlockTokens] * blk_stride +                                \
                          (size_t)(vp_ % kBlockTokens) * D + (c_ / KT) * 8;                               \
        VR = *reinterpret_cast<const uint4 *>(pool + v_ + (size_t)(hkv + g) * kBlockTokens * D);         \
    } while (0)
#define STG_LSTORE(I, KR, VR)                                                                             \
    do {                                                                                                  \
        const int c_ = tid + 256 * (I);                                                                   \
        const int key_ = c_ / (D / 8), d_ = (c_ % (D / 8)) * 8;                                           \
        *reinterpret_cast<uint4 *>(sk + key_ * KROW + d_) = KR;                                           \
        const int vkey_ = c_ % KT, vd_ = (c_ / KT) * 8;                                                   \
        const uint32_t w_[4] = {VR.x, VR.y, VR.z, VR.w};                                                  \
        _Pragma("unroll") for (int j_ = 0; j_ < 4; ++j_) {                                                \
            sv[(vd_ + 2 * j_) * VROW + vkey_] = (uint16_t)(w_[j_] & 0xFFFFu);                             \
            sv[(vd_ + 2 * j_ + 1) * VROW + vkey_] = (uint16_t)(w_[j_] >> 16);                             \
        }                                                                                                 \
    } while (0)
    auto gload = [&](int tile) {
        STG_GLOAD(tile, 0, kr0, vr0);
        if (PER_T > 1) STG_GLOAD(tile, 1, kr1, vr1);
    };
    auto lstore = [&]() {
        STG_LSTORE(0, kr0, vr0);
        if (PER_T > 1) STG_LSTORE(1, kr1, vr1);
    };

    gload(0);
    for (int tile = 0; tile < n_tiles; ++tile) {
        __syncthreads();            // previous tile's LDS reads done
        lstore();
        __syncthreads();
        if (tile + 1 < n_tiles) gload(tile + 1);
        const int k0 = tile * KT;
        if (k0 <= wave_max) {           // wave-uniform: past it every key of the tile is masked
        // S^T[key][query] = sum_d K[key][d] Q[query][d]: A = K (lane: key col, d 16kk + 8 half)
        f32x16_t s;
#pragma unroll
        for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8_t kf = as_bf(*reinterpret_cast<const uint4 *>(sk + col * KROW + 16 * kk + 8 * half));
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qh[kk], s, 0, 0, 0);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, ql[kk], s, 0, 0, 0);
        }
        // lane holds keys k0 + 8 (i / 4) + 4 half + i % 4 for query column col
        float mt = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int kp = k0 + 8 * (i / 4) + 4 * half + (i % 4);
            if (kp > qpos) s[i] = -INFINITY;
            mt = fmaxf(mt, s[i]);
        }
        mt = fmaxf(mt, lane_xor(mt, 32));
        const float m_new = fmaxf(m_run, mt);
        const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
        float p[16], ps = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            p[i] = s[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s[i] - m_new);
            ps += p[i];
        }
        ps += lane_xor(ps, 32);
        l_run = l_run * alpha + ps;
        m_run = m_new;
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {   // some lane's maximum moved
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int i = 0; i < 16; ++i) o[b][i] *= alpha;
        }
        // O^T[d][query] += sum_key V[key][d] P[query][key]; k index (8 half + j) of MFMA m is the
        // lane's key 16 m + 8 (j / 4) + 4 half + j % 4 = its p[8 m + j]
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            bf16x8_t ph, pl;
            split8(p + 8 * m, ph, pl);
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint16_t *vr = sv + (32 * b + col) * VROW + 16 * m + 4 * half;
                const uint2 v0 = *reinterpret_cast<const uint2 *>(vr), v1 = *reinterpret_cast<const uint2 *>(vr + 8);
                const bf16x8_t vf = as_bf(make_uint4(v0.x, v0.y, v1.x, v1.y));
                o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, ph, o[b], 0, 0, 0);
                o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pl, o[b], 0, 0, 0);
            }
        }
        }
    }
    if (!qvalid) return;
    // O^T[d = 32 b + 8 (i / 4) + 4 half + i % 4][query col]
    const float inv = 1.f / l_run;
    if (a.out_pair) {   // four consecutive d of one 32-wide block per store
        uint16_t *prow = a.out_pair + qrow * a.out_pair_ld;
        const int k0 = (g * G + hh) * D;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                store_pair4(prow + pair_at(k0 + 32 * b + 8 * j + 4 * half),
                            make_float4(o[b][4 * j] * inv, o[b][4 * j + 1] * inv, o[b][4 * j + 2] * inv,
                                        o[b][4 * j + 3] * inv));
        return;
    }
    float *orow = a.out + qrow * q_ld + (size_t)(g * G + hh) * D;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) orow[32 * b + 8 * (i / 4) + 4 * half + (i % 4)] = o[b][i] * inv;
}

template <int G, int D>
hipError_t launch_gd(const AttnArgs &a, hipStream_t st) {
    const int hkv = a.kv.n_kv_heads;
    if (a.split_keys == 0) {
        if (a.kv_fp32) {
            STG_LAUNCH((attn_kernel<G, D, true>), dim3(1, hkv, a.rows), dim3(256), 0, st, a);
        } else {
            if (a.n_seqs * a.rows_per_seq != a.rows) return hipErrorInvalidValue;
            constexpr int BQ = 128 / G;
            dim3 grid((a.rows_per_seq + BQ - 1) / BQ, hkv, a.n_seqs);
            STG_LAUNCH((attn_prefill_mfma<G, D>), grid, dim3(256), 0, st, a);
        }
        return hipGetLastError();
    }
    if (a.split_keys > kChunk || a.split_keys % kBlockTokens || a.max_splits > kMaxDecodeSplits ||
        a.rows_per_seq <= 0)
        return hipErrorInvalidValue;
    dim3 grid(a.grid_splits, hkv, a.rows);
    if (a.grid_splits == 1) {   // every row within one split: its output directly, no merge
        if (a.kv_fp32)
            STG_LAUNCH((attn_decode_kernel<G, D, true, true>), grid, dim3(256), 0, st, a);
        else if constexpr (D == 128)
            STG_LAUNCH((attn_decode_mfma<G, D, true>), grid, dim3(256), 0, st, a);
        else
            STG_LAUNCH((attn_decode_kernel<G, D, false, true>), grid, dim3(256), 0, st, a);
        return hipGetLastError();
    }
    if (a.kv_fp32)
        STG_LAUNCH((attn_decode_kernel<G, D, true, false>), grid, dim3(256), 0, st, a);
    else if constexpr (D == 128)
        STG_LAUNCH((attn_decode_mfma<G, D, false>), grid, dim3(256), 0, st, a);
    else
        STG_LAUNCH((attn_decode_kernel<G, D, false, false>), grid, dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    STG_LAUNCH((attn_merge<D>), dim3((unsigned)a.n_q_heads, (unsigned)a.rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs &a, hipStream_t st) {
    if (a.rows <= 0) return hipSuccess;
    const int G = a.n_q_heads / a.kv.n_kv_heads;
    const int D = a.kv.head_dim;
#define STG_ATTN_CASE(GG, DD) \
    if (G == GG && D == DD) return launch_gd<GG, DD>(a, st);
    STG_ATTN_CASE(1, 64) STG_ATTN_CASE(2, 64) STG_ATTN_CASE(4, 64) STG_ATTN_CASE(8, 64)
    STG_ATTN_CASE(1, 128) STG_ATTN_CASE(2, 128) STG_ATTN_CASE(4, 128) STG_ATTN_CASE(8, 128)
#undef STG_ATTN_CASE
    return hipErrorInvalidValue;
}

bool attention_supported(int group, int head_dim) {
    return (group == 1 || group == 2 || group == 4 || group == 8) && (head_dim == 64 || head_dim == 128);
}

}  // namespace stg
