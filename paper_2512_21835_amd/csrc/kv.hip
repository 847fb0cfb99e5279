// RoPE and KV-cache store, block-table updates and dense <-> paged KV copies.
#include "stage_kernels.h"

namespace stg {
namespace {

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void store_kv(void *pool, size_t e, float v, int kv_fp32) {
    if (kv_fp32)
        static_cast<float *>(pool)[e] = v;
    else
        static_cast<uint16_t *>(pool)[e] = to_bf16(v);
}

// One workgroup per row: rotate q and k (pairs (i, i + d/2) by p * theta^(-2i/d), from the
// per-position cos/sin tables), write rotated q, and store rotated k and v into the row's
// position of the paged cache in the KV element type.
__global__ __launch_bounds__(256) void rope_kv_kernel(RopeKvArgs a) {
    const int row = blockIdx.x;
    const int sidx = row / a.meta->rows_per_seq;
    const int pos = a.meta->pos0[sidx] + row % a.meta->rows_per_seq;
    const int slot = a.meta->seq_slot[sidx];
    const int d = a.kv.head_dim, half = d / 2;
    const int hq = a.n_q_heads, hkv = a.kv.n_kv_heads;
    const size_t ld = (size_t)(hq + 2 * hkv) * d;
    const float *src = a.qkv + row * ld;
    const float *cs = a.cos_t + (size_t)pos * half;
    const float *sn = a.sin_t + (size_t)pos * half;
    const int block = a.kv.block_table[(size_t)slot * a.kv.max_blocks + pos / kBlockTokens];
    const size_t kbase = (size_t)block * 2 * hkv * kBlockTokens * d + (size_t)(pos % kBlockTokens) * d;
    const size_t head_stride = (size_t)kBlockTokens * d;

    for (int i = threadIdx.x; i < (hq + hkv) * half; i += blockDim.x) {
        const int h = i / half, j = i % half;
        const float x1 = src[h * d + j], x2 = src[h * d + j + half];
        const float c = cs[j], s = sn[j];
        const float r1 = x1 * c - x2 * s;
        const float r2 = x1 * s + x2 * c;
        if (h < hq) {
            float *q = a.q_out + row * (size_t)hq * d + h * d;
            q[j] = r1;
            q[j + half] = r2;
        } else {
            const size_t e = kbase + (size_t)(h - hq) * head_stride;
            store_kv(a.kv.pool, e + j, r1, a.kv_fp32);
            store_kv(a.kv.pool, e + j + half, r2, a.kv_fp32);
        }
    }
    for (int i = threadIdx.x; i < hkv * d; i += blockDim.x) {
        const int g = i / d, c = i % d;
        const size_t e = kbase + (size_t)(hkv + g) * head_stride + c;
        store_kv(a.kv.pool, e, src[(size_t)(hq + hkv) * d + i], a.kv_fp32);
    }
}

__global__ void meta_write_kernel(CallMeta m, CallMeta *dst) {
    const int *src = reinterpret_cast<const int *>(&m);
    int *d = reinterpret_cast<int *>(dst);
    for (int i = threadIdx.x; i < (int)(sizeof(CallMeta) / sizeof(int)); i += blockDim.x) d[i] = src[i];
}

constexpr int kTableChunk = 240;
struct TableChunk {
    int *table;
    int n;
    int idx[kTableChunk];
    int val[kTableChunk];
};

__global__ void table_write_kernel(TableChunk c) {
    const int i = threadIdx.x;
    if (i < c.n) c.table[c.idx[i]] = c.val[i];
}

template <typename T>
__global__ __launch_bounds__(256) void kv_copy_kernel(KvCopyArgs a) {
    const int t = blockIdx.x, layer = blockIdx.y;
    const int pos = a.pos0 + t;
    const int d = a.head_dim, hkv = a.n_kv_heads;
    const int block = a.block_table[(size_t)a.slot * a.max_blocks + pos / kBlockTokens];
    T *pool = reinterpret_cast<T *>(static_cast<char *>(a.pool_base) + (size_t)layer * a.layer_stride);
    const size_t pbase = (size_t)block * 2 * hkv * kBlockTokens * d + (size_t)(pos % kBlockTokens) * d;
    const size_t dbase = ((size_t)layer * a.n + t) * hkv * d;
    T *dk = static_cast<T *>(a.k);
    T *dv = static_cast<T *>(a.v);
    for (int i = threadIdx.x; i < hkv * d; i += blockDim.x) {
        const int g = i / d, c = i % d;
        const size_t pk = pbase + (size_t)g * kBlockTokens * d + c;
        const size_t pv = pbase + (size_t)(hkv + g) * kBlockTokens * d + c;
        if (a.to_pool) {
            pool[pk] = dk[dbase + i];
            pool[pv] = dv[dbase + i];
        } else {
            dk[dbase + i] = pool[pk];
            dv[dbase + i] = pool[pv];
        }
    }
}

// 16-byte chunks, four in flight per lane, on kParkWorkgroups workgroups: the traffic crosses
// the host link at a few tens of GB/s, and a full-grid copy would hold every compute unit's
// memory pipeline behind slow host accesses while decode kernels wait for HBM.
__global__ __launch_bounds__(256) void kv_park_kernel(KvParkArgs a) {
    const int row_chunks = a.head_dim * a.elem_bytes / 16;  // one (token, head) vector
    const size_t per_layer = (size_t)a.n * a.n_kv_heads * row_chunks;
    const size_t total = 2 * (size_t)a.n_layers * per_layer;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const size_t head_bytes = (size_t)kBlockTokens * a.head_dim * a.elem_bytes;
    char *pool = static_cast<char *>(a.pool_base);
    uint4 *host = static_cast<uint4 *>(a.host);
    auto pool_chunk = [&](size_t c) -> uint4 * {
        const int j = (int)(c % row_chunks);
        size_t r = c / row_chunks;
        const int g = (int)(r % a.n_kv_heads);
        r /= a.n_kv_heads;
        const int t = (int)(r % a.n);
        r /= a.n;
        const int layer = (int)(r % a.n_layers);
        const int kv = (int)(r / a.n_layers);
        const int pos = a.pos0 + t;
        const int block = a.block_table[(size_t)a.slot * a.max_blocks + pos / kBlockTokens];
        const size_t off = (size_t)layer * a.layer_stride + (((size_t)block * 2 + kv) * a.n_kv_heads + g) * head_bytes +
                           (size_t)(pos % kBlockTokens) * a.head_dim * a.elem_bytes + (size_t)j * 16;
        return reinterpret_cast<uint4 *>(pool + off);
    };
    for (size_t c0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c0 < total; c0 += 4 * stride) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t c = c0 + u * stride;
            if (c < total) v[u] = a.to_pool ? host[c] : *pool_chunk(c);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t c = c0 + u * stride;
            if (c < total) {
                if (a.to_pool) *pool_chunk(c) = v[u];
                else host[c] = v[u];
            }
        }
    }
}

}  // namespace

hipError_t launch_kv_park(const KvParkArgs &a, hipStream_t st) {
    if (a.n <= 0) return hipSuccess;
    STG_LAUNCH(kv_park_kernel, dim3(kParkWorkgroups), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_rope_kv_store(const RopeKvArgs &a, hipStream_t st) {
    if (a.rows <= 0) return hipSuccess;
    STG_LAUNCH(rope_kv_kernel, dim3(a.rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_meta_write(const CallMeta &m, CallMeta *dst, hipStream_t st) {
    STG_LAUNCH(meta_write_kernel, dim3(1), dim3(256), 0, st, m, dst);
    return hipGetLastError();
}

hipError_t launch_table_write(int *table, const int *idx, const int *val, int n, hipStream_t st) {
    for (int b = 0; b < n; b += kTableChunk) {
        TableChunk c;
        c.table = table;
        c.n = n - b < kTableChunk ? n - b : kTableChunk;
        for (int i = 0; i < c.n; ++i) {
            c.idx[i] = idx[b + i];
            c.val[i] = val[b + i];
        }
        STG_LAUNCH(table_write_kernel, dim3(1), dim3(256), 0, st, c);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_kv_copy(const KvCopyArgs &a, hipStream_t st) {
    if (a.n <= 0) return hipSuccess;
    dim3 grid(a.n, a.n_layers);
    if (a.kv_fp32)
        STG_LAUNCH(kv_copy_kernel<float>, grid, dim3(256), 0, st, a);
    else
        STG_LAUNCH(kv_copy_kernel<uint16_t>, grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace stg
