// Device code of decode attention, shared by the attention kernel (attention.hip) and the persistent
// per-layer decode kernel (decode_layer.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "stage_kernels.h"

namespace stg {
namespace attn_dev {

constexpr int kChunk = 64;
constexpr int kMaxDecodeSplits = 256;  // splits one row may have (max_context / split_keys)

static __device__ __forceinline__ float bf16lo(uint32_t u) { return __uint_as_float(u << 16); }
static __device__ __forceinline__ float bf16hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

template <bool F32KV>
static __device__ __forceinline__ void load8(const void *pool, size_t elem, float f[8]) {
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

// Decode: one workgroup per (key split, KV head, row); a split holds at most kChunk keys.  K and V
// of the lane's keys are fetched together up front, scores are reduced across the D/8 lanes of a
// key, the split's maximum and sum across the workgroup through LDS once, and the partial output
// (unnormalised, with its max and sum) goes to global memory.  The last workgroup of a (row, KV
// head) to finish -- counted with a device-scope atomic -- merges the row's splits in ascending
// order and resets the counter, so no separate combine launch is needed.
template <int G, int D>
struct DecodeSmem {
    float wm[4][G], wl[4][G];
    float o[4][G][D];
    float cm[G][kMaxDecodeSplits], cl[G][kMaxDecodeSplits], den[G];
    int last;
};

// Merges the nsp splits of (row, KV head g) in ascending order: the weight of split s for head h
// is exp(m_s - max_s m_s) / sum_s(...) of its max m_s and sum l_s.
template <int G, int D>
static __device__ __forceinline__ void attn_merge_group(const AttnArgs &a, int g, int row, int nsp,
                                                        DecodeSmem<G, D> &sm) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hq_total = a.n_q_heads;
    const size_t q_ld = (size_t)hq_total * D;
    for (int i = tid; i < G * nsp; i += 256) {
        const int h = i / nsp, sp = i % nsp;
        const size_t pi = ((size_t)row * hq_total + g * G + h) * a.max_splits + sp;
        sm.cm[h][sp] = a.part_ml[pi * 2 + 0];
        sm.cl[h][sp] = a.part_ml[pi * 2 + 1];
    }
    __syncthreads();
    for (int h = wave; h < G; h += 4) {
        float mx = -INFINITY;
        for (int sp = lane; sp < nsp; sp += 64) mx = fmaxf(mx, sm.cm[h][sp]);
#pragma unroll
        for (int o2 = 32; o2 >= 1; o2 >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o2, 64));
        float den = 0.f;
        for (int sp = lane; sp < nsp; sp += 64) {
            const float w = expf(sm.cm[h][sp] - mx);
            sm.cm[h][sp] = w;
            den = fmaf(w, sm.cl[h][sp], den);
        }
#pragma unroll
        for (int o2 = 32; o2 >= 1; o2 >>= 1) den += __shfl_xor(den, o2, 64);
        if (lane == 0) sm.den[h] = den;
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, c = i % D;
        const int hq = g * G + h;
        const float *po = a.part_o + ((size_t)row * hq_total + hq) * a.max_splits * D + c;
        float num = 0.f;
#pragma unroll 8
        for (int sp = 0; sp < nsp; ++sp) num = fmaf(sm.cm[h][sp], po[(size_t)sp * D], num);
        a.out[row * q_ld + (size_t)hq * D + c] = num / sm.den[h];
    }
}

// Returns true in the workgroup that merged the splits of (row, g) (it wrote the final output).
template <int G, int D, bool F32KV>
static __device__ __forceinline__ bool attn_decode_task(const AttnArgs &a, int split, int g, int row,
                                                       DecodeSmem<G, D> &sm) {
    constexpr int LPK = D / 8;
    constexpr int KPW = 64 / LPK;
    constexpr int KPS = 4 * KPW;
    constexpr int STEPS = kChunk / KPS;
    const int sidx = row / a.meta->rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.meta->rows_per_seq;
    const int slot = a.meta->seq_slot[sidx];
    const int ctx = pos + 1;
    const int kbeg = split * a.split_keys;
    if (kbeg >= ctx) return false;
    const int n = min(a.split_keys, ctx - kbeg);
    const int nsp = (ctx + a.split_keys - 1) / a.split_keys;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kl = lane / LPK, sub = lane % LPK, c0 = sub * 8;
    const int hq_total = a.n_q_heads;
    const size_t q_ld = (size_t)hq_total * D;
    const int hkv = a.kv.n_kv_heads;
    const int *table = a.kv.block_table + (size_t)slot * a.kv.max_blocks;
    const size_t blk_stride = (size_t)2 * hkv * kBlockTokens * D;


    // keys of this lane: kk = st * KPS + wave * KPW + kl
    float kf[STEPS][8], vf[STEPS][8];
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const int kk = st * KPS + wave * KPW + kl;
        if (kk < n) {
            const int key = kbeg + kk;
            const size_t e = (size_t)table[key / kBlockTokens] * blk_stride +
                             ((size_t)g * kBlockTokens + key % kBlockTokens) * D + c0;
            load8<F32KV>(a.kv.pool, e, kf[st]);
            load8<F32KV>(a.kv.pool, e + (size_t)hkv * kBlockTokens * D, vf[st]);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) kf[st][j] = vf[st][j] = 0.f;
        }
    }
    const float scale = 1.f / sqrtf((float)D);
    float q[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float *qp = a.q + row * q_ld + (size_t)(g * G + h) * D + c0;
#pragma unroll
        for (int j = 0; j < 8; ++j) q[h][j] = qp[j] * scale;
    }

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
            for (int o2 = LPK / 2; o2 >= 1; o2 >>= 1) p += __shfl_xor(p, o2, 64);
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
        for (int o2 = 32; o2 >= LPK; o2 >>= 1) m = fmaxf(m, __shfl_xor(m, o2, 64));
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
        for (int o2 = 32; o2 >= LPK; o2 >>= 1) l[h] += __shfl_xor(l[h], o2, 64);
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int o2 = 32; o2 >= LPK; o2 >>= 1) o[h][j] += __shfl_xor(o[h][j], o2, 64);
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
        const size_t pi = ((size_t)row * hq_total + g * G + h) * a.max_splits + split;
        a.part_o[pi * D + c] = ((sm.o[0][h][c] + sm.o[1][h][c]) + sm.o[2][h][c]) + sm.o[3][h][c];
        if (c == 0) {
            a.part_ml[pi * 2 + 0] = fmaxf(fmaxf(sm.wm[0][h], sm.wm[1][h]), fmaxf(sm.wm[2][h], sm.wm[3][h]));
            a.part_ml[pi * 2 + 1] = ((sm.wl[0][h] + sm.wl[1][h]) + sm.wl[2][h]) + sm.wl[3][h];
        }
    }
    if (a.done == nullptr) return false;   // merged by a separate launch (attn_merge_group)
    __threadfence();
    __syncthreads();
    if (tid == 0) sm.last = (atomicAdd(&a.done[row * hkv + g], 1) == nsp - 1);
    __syncthreads();
    if (!sm.last) return false;
    __threadfence();
    attn_merge_group<G, D>(a, g, row, nsp, sm);
    if (tid == 0) a.done[row * hkv + g] = 0;
    return true;
}

}  // namespace attn_dev
}  // namespace stg
