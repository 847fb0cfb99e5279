// Internal interface between the stage runtime (stage_runtime.cpp) and the HIP kernels.
// Not part of the public ABI (include/stage.h).
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace stg {

// Kernel launches made by this thread through the launch helpers below (the runtime reports the
// count per call in its statistics).
extern thread_local long long tl_launches;
#define STG_LAUNCH(...)                  \
    do {                                 \
        ++::stg::tl_launches;            \
        hipLaunchKernelGGL(__VA_ARGS__);    \
    } while (0)
#define STG_EXT_LAUNCH(...)              \
    do {                                 \
        ++::stg::tl_launches;            \
        hipExtLaunchKernelGGL(__VA_ARGS__); \
    } while (0)

constexpr int kMaxSeqs = 64;     // sequences in one call
constexpr int kBlockTokens = 16; // tokens per paged-KV block

// Rows of a call: sequence k of the call owns rows [k*rows_per_seq, (k+1)*rows_per_seq);
// its row t sits at position pos0[k] + t and its block table is row seq_slot[k].
struct CallMeta {
    int n_seqs;
    int rows_per_seq;
    int seq_slot[kMaxSeqs];
    int pos0[kMaxSeqs];
};

// Paged KV pool of one layer: block b holds K then V, each [n_kv_heads][16][head_dim].
struct KvView {
    void *pool;              // element type: bf16 bits or fp32 (kv_fp32)
    const int *block_table;  // [n_seq_slots][max_blocks]
    int max_blocks;
    int n_kv_heads;
    int head_dim;
};

enum GemvMode {
    GEMV_PLAIN_RESIDUAL = 1, // out = res + W act
    GEMV_NORM_SWIGLU = 2,    // out = silu(Wg y) * (Wu y), y = rmsnorm(act) * gain
    GEMV_NORM_ROPE_KV = 3    // [q | k | v] = Wqkv y; rotate q, k; q -> q_out, k and v -> KV cache
};

struct GemvArgs {
    const uint16_t *w;    // [N, K] bf16
    const uint16_t *w2;   // second [N, K] matrix (SWIGLU: up projection)
    const float *act;     // [rows, K] with row stride act_ld
    const uint16_t *gain; // [K] bf16 (NORM modes)
    const float *res;     // [rows, N] with row stride out_ld (RESIDUAL)
    float *out;           // [rows, N] with row stride out_ld (ROPE_KV: rotated q, [rows, Hq d])
    long act_ld, out_ld;
    int N, K;
    int rows;  // rows in this launch
    int row0;  // index of the launch's first row among the call's rows (ROPE_KV: row metadata)
    float eps;
    // ROPE_KV only
    const float *cos_t, *sin_t;  // [max_context, d/2]
    KvView kv;
    int n_q_heads;
    int kv_fp32;
    const CallMeta *meta;  // device copy of the call's row metadata
    // Matrix-core launches split K across workgroups when given this workspace (and the layer
    // shape calls for it): [8][2][16][units] partial products, [8][16] partial sums of squares.
    float *split_part;
    float *split_ss;
};
constexpr int kGemvMaxSplits = 8;

// Compute units of the current device (256 on a whole MI355X; fewer on a partitioned one), read
// once per device.  Launch shapes that aim at one or two workgroups per compute unit use it.
int device_compute_units();

// y = W x for `rows` activation rows (any number; launched in chunks of up to 8 rows).  K must be a
// multiple of 8.  Non-null events are recorded at the start of the first and the end of the last
// launch (kernel timestamps, no extra stream packets).
hipError_t launch_gemv(int mode, GemvArgs a, hipStream_t st, hipEvent_t ev_start = nullptr,
                       hipEvent_t ev_stop = nullptr);

enum GemmMode { GEMM_STORE = 0, GEMM_RESIDUAL = 1, GEMM_SWIGLU = 2 };

// A prefill GEMM operand is an fp32 matrix X [M, K] held as the exact-sum pair X = hi + lo of two
// bf16 matrices, interleaved by 32-wide k blocks: row m holds, for each block b, the 32 hi values
// of k = 32 b .. 32 b + 31 and then their 32 lo values, so element k of the row has its hi at
// 64 (k / 32) + k % 32 and its lo 32 further.  Row stride pair_ld(K) (K rounded up to a whole
// block; a partial last block's padding is never read).
constexpr long pair_ld(long k) { return 2 * ((k + 31) / 32 * 32); }
__host__ __device__ constexpr long pair_at(long k) { return 2 * (k & ~31L) + (k & 31); }

// Prefill projection on the matrix cores: out[m, out_col + n] (+)= sum_k (hi + lo)[m, k] W[n, k].
// SWIGLU (K a multiple of 32, n_mats = 1): w[0] = Wg, w[1] = Wu, both [N, K]; writes
// h = silu(Wg a) * (Wu a) as a pair [M, N] to out_pair with row stride ldo.
struct GemmArgs {
    const uint16_t *a;            // [M, lda] pair of the fp32 activation (lda >= pair_ld(K))
    long lda;
    const uint16_t *w[2];         // [N, K] bf16; grid z selects the matrix
    float *out;                   // row stride ldo
    const float *res;             // RESIDUAL: added, same indexing as out
    long ldo;
    int out_col[2];               // output column offset of each matrix
    int M, N, K;
    uint16_t *out_pair;           // SWIGLU output pair (row stride ldo >= pair_ld(N))
};
hipError_t launch_gemm(int mode, const GemmArgs &a, int n_mats, hipStream_t st);
// y = rmsnorm(x) * g as a pair [rows, H] (row stride ld).
hipError_t launch_rmsnorm_split(const float *x, const uint16_t *g, float eps, int rows, int H, uint16_t *pair,
                                long ld, hipStream_t st);
// The pair [rows, n] (row stride ld) of an fp32 matrix [rows, n].
hipError_t launch_split(const float *x, int rows, int n, uint16_t *pair, long ld, hipStream_t st);
// silu(gate) * up of gu [rows, 2F] (gate columns first) as a pair [rows, F] (row stride ld).
hipError_t launch_swiglu_split(const float *gu, int F, int rows, uint16_t *pair, long ld, hipStream_t st);

struct RopeKvArgs {
    const float *qkv;  // [rows, (Hq + 2 Hkv) d]: q heads, then k heads, then v heads
    float *q_out;      // [rows, Hq d] rotated queries
    const float *cos_t, *sin_t;  // [max_context, d/2]
    KvView kv;
    int n_q_heads;
    int kv_fp32;
    int rows;
    const CallMeta *meta; // device copy of the call's row metadata
};
hipError_t launch_rope_kv_store(const RopeKvArgs &a, hipStream_t st);

struct AttnArgs {
    const float *q;      // [rows, Hq d] rotated
    float *out;          // [rows, Hq d]
    // prefill with the bf16 cache: when set, the output goes here instead of `out`, as the hi/lo
    // pair the O projection GEMM reads ([rows, out_pair_ld], pair_at layout)
    uint16_t *out_pair;
    long out_pair_ld;
    float *part_o;       // [rows, Hq, max_splits, d] unnormalised partial outputs
    float *part_ml;      // [rows, Hq, max_splits, 2] partial max and sum
    KvView kv;
    int n_q_heads;
    int kv_fp32;
    int rows;
    int split_keys;      // keys per split; 0 = one split per row (final output directly)
    int max_splits;      // stride of the partial buffers
    int grid_splits;     // splits launched: ceil(longest context in the call / split_keys)
    int n_seqs;          // sequences in the call and rows per sequence: host copies of the row
    int rows_per_seq;    // metadata (the prefill launch grid; the decode kernels' row -> sequence map)
    const CallMeta *meta; // device copy of the call's row metadata
};
hipError_t launch_attention(const AttnArgs &a, hipStream_t st);
bool attention_supported(int group, int head_dim);

// Writes the call's row metadata to device memory (one small launch per call; the hot kernels
// read it from there instead of carrying it in their arguments).
hipError_t launch_meta_write(const CallMeta &m, CallMeta *dst, hipStream_t st);

// Slot tags (stage_config.slot_check): tag = {layer, load}, two ints.  The check compares a tag
// with the expected layer and load and counts into rec[8]: [0] checks run, [1] mismatches, [2..7]
// the first mismatch (where, slot, expected layer, expected load, found layer, found load).
hipError_t launch_slot_tag_write(int *tag, int layer, int load, hipStream_t st);
hipError_t launch_slot_tag_check(const int *tag, int slot, int layer, int load, int where, int *rec,
                                 hipStream_t st);

// Writes table[idx[i]] = val[i] for i < n (any n; chunked).
hipError_t launch_table_write(int *table, const int *idx, const int *val, int n, hipStream_t st);

// Moves K/V between a dense buffer [n_layers][n][Hkv][d] and positions pos0..pos0+n-1 of the
// sequence whose block table row is `slot`.  to_pool: dense -> pool, else pool -> dense.
struct KvCopyArgs {
    void *pool_base;        // layer 0 pool; layer l at pool_base + l * layer_stride bytes
    size_t layer_stride;
    const int *block_table;
    int max_blocks;
    int n_kv_heads, head_dim, kv_fp32;
    int n_layers;
    int slot, pos0, n;
    void *k, *v;            // dense device buffers
    int to_pool;
};
hipError_t launch_kv_copy(const KvCopyArgs &a, hipStream_t st);

// One sequence's KV tail between the paged pool and a dense [K|V][layer][token][head][d] buffer
// in pinned host memory, addressed by the device (KV parking).
struct KvParkArgs {
    void *pool_base;        // layer 0 pool; layer l at pool_base + l * layer_stride bytes
    size_t layer_stride;
    const int *block_table;
    int max_blocks;
    int n_kv_heads, head_dim, elem_bytes;
    int n_layers;
    int slot, pos0, n;
    void *host;             // device address of the pinned buffer
    int to_pool;
};
constexpr int kParkWorkgroups = 32;  // few compute units: the host link is the bound
hipError_t launch_kv_park(const KvParkArgs &a, hipStream_t st);

// Bytes of the per-device scratch array of stage_decode_noalloc (noalloc.hip).
constexpr size_t kScratchBytes = size_t(64) << 20;
// Device address of the current device's scratch array, looked up on the first call for
// `device` (which must be current) and kept.
hipError_t scratch_setup(int device, void **out);

}  // namespace stg
