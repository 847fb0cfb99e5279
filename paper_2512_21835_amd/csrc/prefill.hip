// Prefill projections on the matrix cores: C[M, N] = A[M, K] . W[N, K]^T with bf16 weights W and
// an fp32 activation A taken as the exact-sum pair A = hi + lo of two bf16 matrices (hi = bf16(A),
// lo = bf16(A - hi); the pair keeps ~16 bits of A's mantissa, a single bf16 only 8).  Each 16-wide
// k step issues v_mfma_f32_32x32x16_bf16 twice per output block, hi then lo, accumulating in fp32.
// The pair is stored interleaved by 32-wide k blocks (hi block, then lo block, per row), so the
// operand bytes of one k tile of a row are 128 contiguous bytes.
//
// Tiling: a workgroup (4 wavefronts) computes a 128 x 128 tile of C, each wavefront a 64 x 64
// sub-tile as 2 x 2 blocks of 32 x 32; or, when the grid of 256 x 256 tiles still has a workgroup
// for every compute unit, a 256 x 256 tile with 4 x 4 blocks per wavefront.  K advances 32 at a
// time.  gemm_dma_kernel (K a multiple of 32) copies tiles global -> LDS directly into a ring of
// three stages, two tiles ahead; gemm_kernel (any K) stages them through registers into two LDS
// stages, one tile ahead.  Tiles are stored in LDS in MFMA fragment order (lane l of a fragment at
// offset 16 l), so every fragment read is one conflict-free ds_read_b128 per lane.  Workgroups that
// share a weight tile are adjacent in launch order (x over M tiles), so each weight tile is read
// from HBM once and re-served from L2.
//
// The producers of A write the hi/lo pair directly: RMSNorm (before QKV and gate/up), the
// attention output (before O) and the SwiGLU of the gate/up output (before down).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "lanes.h"
#include "pair.h"
#include "stage_kernels.h"

namespace stg {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int kFrag = (BM / 32) * (BK / 16) * 64;  // 16-byte fragment slots per operand tile (512)

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4 &v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// LDS slot of 16-byte chunk `ch` (k offset 8 ch) of tile row `row`.
__device__ __forceinline__ int frag_slot(int row, int ch) {
    return ((row >> 5) * (BK / 16) + (ch >> 1)) * 64 + (row & 31) + 32 * (ch & 1);
}

// Stores one 32 x 32 accumulator block (rows mb .. mb + 31, this lane's column c): register r of
// lane l is row mb + 8 (r / 4) + 4 (l / 32) + r % 4.  RESIDUAL: for a block inside M all 16
// residual values are loaded before any sum is stored, in straight-line code, so their loads are in
// flight together and the stores wait for nothing (out may alias res: each element is read and
// written by this lane only, read first).  A block crossing M stores element by element.
template <int MODE>
__device__ __forceinline__ void store_block(const GemmArgs &a, const f32x16 &acc, int mb, int M, int c, int lane) {
    const size_t o0 = (size_t)(mb + 4 * (lane >> 5)) * a.ldo + c;
    auto off = [&](int r) { return o0 + (size_t)(8 * (r >> 2) + (r & 3)) * a.ldo; };
    if (mb + 32 <= M) {   // the same for the whole wavefront
        float rv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) rv[r] = MODE == GEMM_RESIDUAL ? a.res[off(r)] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) a.out[off(r)] = MODE == GEMM_RESIDUAL ? rv[r] + acc[r] : acc[r];
        return;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int m = mb + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m < M) a.out[off(r)] = MODE == GEMM_RESIDUAL ? a.res[off(r)] + acc[r] : acc[r];
    }
}

template <int MODE>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
    __shared__ uint4 lds[2][3][kFrag];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
    const uint16_t *W = a.w[blockIdx.z];
    const int M = a.M, N = a.N, K = a.K;

    // global -> register tile load: chunk q = tid + 256 i, row q / 4, 16-byte chunk q % 4
    uint4 rh[2], rl[2], rw[2];
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int q = tid + 256 * i, row = q >> 2, ch = q & 3, k = k0 + ch * 8;
            const bool kin = k < K;
            const int m = m0 + row, n = n0 + row;
            rh[i] = rl[i] = rw[i] = make_uint4(0, 0, 0, 0);
            if (kin && m < M) {
                const uint16_t *p = a.a + (size_t)m * a.lda + pair_at(k);
                rh[i] = *reinterpret_cast<const uint4 *>(p);
                rl[i] = *reinterpret_cast<const uint4 *>(p + 32);
            }
            if (kin && n < N) rw[i] = *reinterpret_cast<const uint4 *>(W + (size_t)n * K + k);
        }
    };
    auto store = [&](int st) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int q = tid + 256 * i;
            const int s = frag_slot(q >> 2, q & 3);
            lds[st][0][s] = rh[i];
            lds[st][1][s] = rl[i];
            lds[st][2][s] = rw[i];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    load(0);
    store(0);
    int st = 0;
    for (int k0 = 0; k0 < K; k0 += BK) {
        __syncthreads();
        const bool more = k0 + BK < K;
        if (more) load(k0 + BK);
#pragma unroll
        for (int step = 0; step < BK / 16; ++step) {
            bf16x8 ah[2], al[2], bw[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int sa = ((wm * 2 + b) * (BK / 16) + step) * 64 + lane;
                const int sb = ((wn * 2 + b) * (BK / 16) + step) * 64 + lane;
                ah[b] = as_bf16x8(lds[st][0][sa]);
                al[b] = as_bf16x8(lds[st][1][sa]);
                bw[b] = as_bf16x8(lds[st][2][sb]);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[i], bw[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[i], bw[j], acc[i][j], 0, 0, 0);
                }
        }
        if (more) store(st ^ 1);
        st ^= 1;
    }

    // result register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32 of the block
    const int col_off = a.out_col[blockIdx.z];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn * 64 + j * 32 + (lane & 31);
            if (n >= N) continue;
            store_block<MODE>(a, acc[i][j], m0 + wm * 64 + i * 32, M, col_off + n, lane);
        }
}

// Copies 16 bytes per lane from global memory straight into LDS (global_load_lds_dwordx4): lane l
// of the wavefront writes LDS bytes [lds_addr + 16 l, lds_addr + 16 l + 16).  Issued as inline
// assembly so that the compiler does not wait for every such load before each LDS read (it cannot
// tell which LDS bytes a DMA load writes); the kernel waits for them itself (wait_vm).  m0 holds
// the wavefront-uniform LDS address; nothing else in the kernel uses m0.  An LDS DMA must not
// directly follow a scalar write of m0 (gfx9 asks for one wait state there; the compiler inserts it
// in code it generates, not inside inline assembly), hence the s_nop.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr) : "memory");
}

// s_waitcnt vmcnt(N), other counters untouched.
template <int N>
__device__ __forceinline__ void wait_vm() {
    __builtin_amdgcn_s_waitcnt(0x3F70 | (N & 0xF) | ((N >> 4) << 14));
}

// s_waitcnt lgkmcnt(N), other counters untouched.
template <int N>
__device__ __forceinline__ void wait_lgkm() {
    static_assert(N >= 0 && N < 16, "lgkmcnt is four bits");
    __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
}

// The same product as gemm_kernel (same MFMAs in the same order: bit-identical results) for K a
// multiple of 32, with the operand tiles copied into a ring of three LDS stages by
// global_load_lds: tile t + 2 is in flight while tile t is multiplied, and no registers stage it.
// Each wavefront computes WB x WB blocks of 32 x 32, so a workgroup tile is 64 WB square: WB = 2
// gives the 128 x 128 tile, WB = 4 the 256 x 256 tile (16 accumulator blocks per wavefront, one
// wavefront per SIMD), which reads half as many operand bytes per product from L2 and LDS.
// The weight tile in LDS is row-major, four 16-byte k segments per row (BK = 32), segment s of row
// r stored at slot 4 r + (s ^ ((r >> 2) & 3)): each DMA instruction then copies 16 rows x 64
// contiguous bytes (lane l: row 16 q + l / 4 of instruction q), and the 32 x 32 fragment reads
// (lane l: row l % 32, segment 2 step + l / 32) touch every LDS bank once per 16 lanes.  (Loading
// in fragment order instead, 32 rows x 32 bytes per instruction, took 1.3-1.6x as long.)  The
// activation tile holds a row's whole 128-byte k block (hi segments 0-3, lo segments 4-7),
// segment g of row r at slot 8 r + (g ^ ((r >> 1) & 7)): one DMA instruction copies 8 rows x 128
// contiguous bytes (full cache lines; 16 rows x 64 bytes of hi and of lo took 5-15% longer per
// GEMM), and the fragment reads again meet every bank once per 16 lanes.
//
// With one wavefront per SIMD (WB = 4) nothing else hides the latency of a fragment read or of the
// barrier, so that loop is software-pipelined (K >= 64): the fragments of the next k step are
// read one whole batch of 32 MFMAs before they are used, the tile's barrier sits between its two
// k steps, and the DMA of tile t + 2 is issued between the MFMAs of tile t's first step.  Schedule
// fences keep the compiler from moving the MFMAs across the barrier or the reads to their use.
template <int MODE, int WB>
__global__ __launch_bounds__(256) void gemm_dma_kernel(GemmArgs a) {
    constexpr int S = 3;
    constexpr int TILE = 64 * WB;                 // workgroup tile rows of each operand
    constexpr int SLOTS = TILE * (BK / 8);        // 16-byte slots per operand tile (4 per row)
    constexpr int AI = 2 * WB;                    // activation copies per wavefront per k tile
    constexpr int PER_TILE = AI + WB;             // load instructions per wavefront per k tile
    static_assert(SLOTS == 4 * WB * 64, "each wavefront loads WB instructions of the weight tile");
    static_assert(BK == 32, "the segment swizzles assume 32-wide k tiles");
    __shared__ uint4 lds[S][3][SLOTS];            // per stage: activation tile (2 SLOTS), weight tile
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4 *)&lds[0][0][0];
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.x * TILE, n0 = blockIdx.y * TILE;
    const uint16_t *W = a.w[blockIdx.z];
    const int M = a.M, N = a.N, K = a.K, nk = K / BK;

    // activation copy qa = wave * AI + i: lane l copies segment (l % 8) ^ ((row >> 1) & 7) of the
    // 128-byte k block of row 8 qa + l / 8 into slot 64 qa + l; weight copy q = wave * WB + i: lane
    // l copies row 16 q + l / 4, k segment (l % 4) ^ ((row >> 2) & 3) into slot 64 q + l.  Rows past
    // M or N are clamped (in bounds), their results are never stored.
    // SWIGLU: the weight tile's 32-row blocks alternate between Wg and Wu rows n0 / 2 + 32 (b / 2) ..
    const uint16_t *src_a[AI], *src_w[WB];
#pragma unroll
    for (int i = 0; i < AI; ++i) {
        const int r = 8 * (wave * AI + i) + (lane >> 3), g = (lane & 7) ^ ((r >> 1) & 7);
        src_a[i] = a.a + (size_t)min(m0 + r, M - 1) * a.lda + 8 * g;
    }
#pragma unroll
    for (int i = 0; i < WB; ++i) {
        const int q = wave * WB + i, r = 16 * q + (lane >> 2), seg = (lane & 3) ^ ((r >> 2) & 3);
        if (MODE == GEMM_SWIGLU) {
            const int b = r >> 5, n = min(n0 / 2 + 32 * (b >> 1) + (r & 31), N - 1);
            src_w[i] = a.w[b & 1] + (size_t)n * K + 8 * seg;
        } else {
            src_w[i] = W + (size_t)min(n0 + r, N - 1) * K + 8 * seg;
        }
    }
    // this wavefront's share of tile t, part i: activation copies 2 i and 2 i + 1, weight copy i
    auto issue_part = [&](int t, int i) {
        const int st = t % S, q = wave * WB + i, qa = wave * AI + 2 * i;
        dma16(src_a[2 * i] + 64 * t, lds_base + ((st * 3) * SLOTS + qa * 64) * 16);
        dma16(src_a[2 * i + 1] + 64 * t, lds_base + ((st * 3) * SLOTS + (qa + 1) * 64) * 16);
        dma16(src_w[i] + BK * t, lds_base + ((st * 3 + 2) * SLOTS + q * 64) * 16);
    };
    auto issue = [&](int t) {
#pragma unroll
        for (int i = 0; i < WB; ++i) issue_part(t, i);
    };

    f32x16 acc[WB][WB];
#pragma unroll
    for (int i = 0; i < WB; ++i)
#pragma unroll
        for (int j = 0; j < WB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int fr = lane & 31, fk = lane >> 5;   // fragment row and k half of this lane
    // the fragments of k step `step` (0 or 1) of tile t, which is in stage t % S
    auto read = [&](int t, int step, bf16x8 (&ah)[WB], bf16x8 (&al)[WB], bf16x8 (&bw)[WB]) {
        const uint4 *L = &lds[t % S][0][0];
        const int seg = 2 * step + fk;
#pragma unroll
        for (int b = 0; b < WB; ++b) {
            const int ra = 32 * (wm * WB + b) + fr, rb = 32 * (wn * WB + b) + fr;
            const int sw = (ra >> 1) & 7;
            const int sb = 4 * rb + (seg ^ ((rb >> 2) & 3));
            ah[b] = as_bf16x8(L[8 * ra + (seg ^ sw)]);
            al[b] = as_bf16x8(L[8 * ra + ((4 + seg) ^ sw)]);
            bw[b] = as_bf16x8(L[2 * SLOTS + sb]);
        }
    };
    // one k step of accumulator row i: hi then lo into each block
    auto mma_row = [&](int i, const bf16x8 (&ah)[WB], const bf16x8 (&al)[WB], const bf16x8 (&bw)[WB]) {
#pragma unroll
        for (int j = 0; j < WB; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[i], bw[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[i], bw[j], acc[i][j], 0, 0, 0);
        }
    };

    if constexpr (WB != 4) {
        issue(0);
        if (nk > 1) issue(1);
        for (int t = 0; t < nk; ++t) {
            // tile t has landed when at most the next tile's loads are still in flight
            if (t + 1 < nk) wait_vm<PER_TILE>();
            else wait_vm<0>();
            __syncthreads();  // every wavefront's part of tile t is in LDS; stage (t - 1) % S is free
            if (t + 2 < nk) issue(t + 2);
#pragma unroll
            for (int step = 0; step < BK / 16; ++step) {
                bf16x8 ah[WB], al[WB], bw[WB];
                read(t, step, ah, al, bw);
#pragma unroll
                for (int i = 0; i < WB; ++i) mma_row(i, ah, al, bw);
            }
        }
    } else {
        // nk >= 2 (launch_gemm_mode).  The loop body is straight-line (the last two tiles are
        // peeled), so that no merge of control flow makes the second batch wait for the reads
        // issued after the barrier.
        issue(0);
        issue(1);
        wait_vm<PER_TILE>();
        __syncthreads();
        bf16x8 h0[WB], l0[WB], w0[WB], h1[WB], l1[WB], w1[WB];
        read(0, 0, h0, l0, w0);
        auto tile = [&](int t, auto more_dma, auto more_tiles) {
            read(t, 1, h1, l1, w1);
            __builtin_amdgcn_sched_barrier(0);
            // the DMA of tile t + 2 goes to stage (t + 2) % S, which held tile t - 1: every
            // wavefront finished reading it before the previous tile's barrier
#pragma unroll
            for (int i = 0; i < WB; ++i) {
                mma_row(i, h0, l0, w0);
                if constexpr (decltype(more_dma)::value) issue_part(t + 2, i);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (decltype(more_tiles)::value) {
                if constexpr (decltype(more_dma)::value) wait_vm<PER_TILE>();   // tile t + 1 has landed
                else wait_vm<0>();
                wait_lgkm<0>();   // this wavefront's reads of tile t are done
                __syncthreads();
                read(t + 1, 0, h0, l0, w0);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int i = 0; i < WB; ++i) mma_row(i, h1, l1, w1);
            __builtin_amdgcn_sched_barrier(0);
        };
        int t = 0;
        for (; t + 2 < nk; ++t) tile(t, std::true_type{}, std::true_type{});
        tile(t, std::false_type{}, std::true_type{});
        tile(t + 1, std::false_type{}, std::false_type{});
    }

    if (MODE == GEMM_SWIGLU) {   // blocks j (gate) and j + 1 (up) hold the same rows of h
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
            for (int j = 0; j < WB; j += 2) {
                const int n = n0 / 2 + 32 * ((wn * WB + j) >> 1) + (lane & 31);
                if (n >= N) continue;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = m0 + wm * 32 * WB + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    if (m >= M) continue;
                    const float gt = acc[i][j][r], up = acc[i][j + 1][r];
                    const size_t o = (size_t)m * a.ldo + pair_at(n);
                    split_pair(gt / (1.f + expf(-gt)) * up, a.out_pair[o], a.out_pair[o + 32]);
                }
            }
        return;
    }
    const int col_off = a.out_col[blockIdx.z];
#pragma unroll
    for (int i = 0; i < WB; ++i)
#pragma unroll
        for (int j = 0; j < WB; ++j) {
            const int n = n0 + wn * 32 * WB + j * 32 + (lane & 31);
            if (n >= N) continue;
            store_block<MODE>(a, acc[i][j], m0 + wm * 32 * WB + i * 32, M, col_off + n, lane);
        }
}

// y = x / sqrt(mean(x^2) + eps) * g, written as a pair (row stride ld).  One workgroup per row.
__global__ __launch_bounds__(256) void rmsnorm_split_kernel(const float *x, const uint16_t *g, float eps, int H,
                                                             uint16_t *pair, long ld) {
    const int row = blockIdx.x;
    const float *xr = x + (size_t)row * H;
    // sum of squares: four elements per thread and step (H % 4 == 0), the loads of four steps
    // issued before their products
    float ss = 0.f;
#pragma unroll 4
    for (int i = 4 * threadIdx.x; i < H; i += 1024) {
        const float4 v = *reinterpret_cast<const float4 *>(xr + i);
        ss = fmaf(v.x, v.x, ss);
        ss = fmaf(v.y, v.y, ss);
        ss = fmaf(v.z, v.z, ss);
        ss = fmaf(v.w, v.w, ss);
    }
    __shared__ float red[4];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += lane_xor(ss, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = ((red[0] + red[1]) + red[2]) + red[3];
    const float scale = 1.f / sqrtf(tot / (float)H + eps);
    // four elements per thread (H % 4 == 0): one 16-byte load, 8-byte stores of their hi and lo
    for (int i = 4 * threadIdx.x; i < H; i += 1024) {
        const float4 v = *reinterpret_cast<const float4 *>(xr + i);
        const uint2 gg = *reinterpret_cast<const uint2 *>(g + i);
        store_pair4(pair + (size_t)row * ld + pair_at(i),
                    make_float4(v.x * scale * __uint_as_float(gg.x << 16), v.y * scale * __uint_as_float(gg.x & 0xFFFF0000u),
                                v.z * scale * __uint_as_float(gg.y << 16), v.w * scale * __uint_as_float(gg.y & 0xFFFF0000u)));
    }
}

// The same for H = 1024 NV (NV <= 8): a thread's NV float4 of the row stay in registers between
// the sum of squares and the output, so the row is read once (same arithmetic in the same order:
// identical results).
template <int NV>
__global__ __launch_bounds__(256) void rmsnorm_split_rows_kernel(const float *x, const uint16_t *g, float eps,
                                                                 uint16_t *pair, long ld) {
    constexpr int H = 1024 * NV;
    const int row = blockIdx.x;
    const float *xr = x + (size_t)row * H + 4 * threadIdx.x;
    float4 v[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) v[j] = *reinterpret_cast<const float4 *>(xr + 1024 * j);
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        ss = fmaf(v[j].x, v[j].x, ss);
        ss = fmaf(v[j].y, v[j].y, ss);
        ss = fmaf(v[j].z, v[j].z, ss);
        ss = fmaf(v[j].w, v[j].w, ss);
    }
    __shared__ float red[4];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += lane_xor(ss, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = ((red[0] + red[1]) + red[2]) + red[3];
    const float scale = 1.f / sqrtf(tot / (float)H + eps);
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = 4 * threadIdx.x + 1024 * j;
        const uint2 gg = *reinterpret_cast<const uint2 *>(g + i);
        store_pair4(pair + (size_t)row * ld + pair_at(i),
                    make_float4(v[j].x * scale * __uint_as_float(gg.x << 16), v[j].y * scale * __uint_as_float(gg.x & 0xFFFF0000u),
                                v[j].z * scale * __uint_as_float(gg.y << 16), v[j].w * scale * __uint_as_float(gg.y & 0xFFFF0000u)));
    }
}

// The pair (row stride ld) of an fp32 matrix [rows, n] (row stride n, n % 4 == 0), four elements
// per thread.
__global__ __launch_bounds__(256) void split_kernel(const float *x, int rows, int n, uint16_t *pair, long ld) {
    const size_t quads = (size_t)rows * n / 4;
    for (size_t q = blockIdx.x * 256ull + threadIdx.x; q < quads; q += (size_t)gridDim.x * 256) {
        const size_t r = 4 * q / n;
        const int c = (int)(4 * q % n);
        store_pair4(pair + r * ld + pair_at(c), *reinterpret_cast<const float4 *>(x + 4 * q));
    }
}

// h = silu(gate) * up from gu [rows, 2F] (gate columns first), written as a pair [rows, F] (row
// stride ld; F % 4 == 0), four elements per thread.
__global__ __launch_bounds__(256) void swiglu_split_kernel(const float *gu, int F, int rows, uint16_t *pair,
                                                            long ld) {
    const size_t quads = (size_t)rows * F / 4;
    for (size_t q = blockIdx.x * 256ull + threadIdx.x; q < quads; q += (size_t)gridDim.x * 256) {
        const size_t r = 4 * q / F;
        const int f = (int)(4 * q % F);
        const float4 g4 = *reinterpret_cast<const float4 *>(gu + r * 2 * F + f);
        const float4 u4 = *reinterpret_cast<const float4 *>(gu + r * 2 * F + F + f);
        auto sw = [](float gt, float up) { return gt / (1.f + expf(-gt)) * up; };
        store_pair4(pair + r * ld + pair_at(f), make_float4(sw(g4.x, u4.x), sw(g4.y, u4.y), sw(g4.z, u4.z), sw(g4.w, u4.w)));
    }
}

int grid_for(size_t count) {
    const size_t g = (count + 255) / 256;
    return (int)(g < 8192 ? g : 8192);
}

template <int MODE>
void launch_gemm_mode(const GemmArgs &a, int n_mats, hipStream_t st) {
    // SWIGLU tiles span the rows of both matrices: 2N virtual rows, one grid layer
    const int nv = MODE == GEMM_SWIGLU ? 2 * a.N : a.N;
    dim3 grid((a.M + BM - 1) / BM, (nv + BN - 1) / BN, n_mats);
    dim3 wide((a.M + 255) / 256, (nv + 255) / 256, n_mats);
    if constexpr (MODE != GEMM_SWIGLU) {
        if (a.K % BK != 0) {
            STG_LAUNCH(gemm_kernel<MODE>, grid, dim3(256), 0, st, a);
            return;
        }
    }
    // the wide tiles when they still fill every compute unit (their pipelined loop takes K >= 64)
    if ((long)wide.x * wide.y * wide.z >= device_compute_units() && a.K >= 2 * BK)
        STG_LAUNCH((gemm_dma_kernel<MODE, 4>), wide, dim3(256), 0, st, a);
    else
        STG_LAUNCH((gemm_dma_kernel<MODE, 2>), grid, dim3(256), 0, st, a);
}

}  // namespace

hipError_t launch_gemm(int mode, const GemmArgs &a, int n_mats, hipStream_t st) {
    if (a.M <= 0) return hipSuccess;
    // every variant runs the same MFMAs in the same order: the choice never changes a bit
    if (a.lda < pair_ld(a.K)) return hipErrorInvalidValue;
    if (mode == GEMM_SWIGLU) {
        if (a.K % BK != 0 || n_mats != 1 || !a.out_pair || a.ldo < pair_ld(a.N)) return hipErrorInvalidValue;
        launch_gemm_mode<GEMM_SWIGLU>(a, 1, st);
    } else if (mode == GEMM_RESIDUAL) {
        launch_gemm_mode<GEMM_RESIDUAL>(a, n_mats, st);
    } else {
        launch_gemm_mode<GEMM_STORE>(a, n_mats, st);
    }
    return hipGetLastError();
}

hipError_t launch_rmsnorm_split(const float *x, const uint16_t *g, float eps, int rows, int H, uint16_t *pair,
                                long ld, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (ld < pair_ld(H) || H % 4 != 0) return hipErrorInvalidValue;
    switch (H) {
        case 4096: STG_LAUNCH(rmsnorm_split_rows_kernel<4>, dim3(rows), dim3(256), 0, st, x, g, eps, pair, ld); break;
        case 8192: STG_LAUNCH(rmsnorm_split_rows_kernel<8>, dim3(rows), dim3(256), 0, st, x, g, eps, pair, ld); break;
        default: STG_LAUNCH(rmsnorm_split_kernel, dim3(rows), dim3(256), 0, st, x, g, eps, H, pair, ld);
    }
    return hipGetLastError();
}

hipError_t launch_split(const float *x, int rows, int n, uint16_t *pair, long ld, hipStream_t st) {
    if (rows <= 0 || n <= 0) return hipSuccess;
    if (ld < pair_ld(n)) return hipErrorInvalidValue;
    if (n % 4 != 0) return hipErrorInvalidValue;
    STG_LAUNCH(split_kernel, dim3(grid_for((size_t)rows * n / 4)), dim3(256), 0, st, x, rows, n, pair, ld);
    return hipGetLastError();
}

hipError_t launch_swiglu_split(const float *gu, int F, int rows, uint16_t *pair, long ld, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (ld < pair_ld(F)) return hipErrorInvalidValue;
    if (F % 4 != 0) return hipErrorInvalidValue;
    STG_LAUNCH(swiglu_split_kernel, dim3(grid_for((size_t)rows * F / 4)), dim3(256), 0, st, gu, F, rows, pair, ld);
    return hipGetLastError();
}

}  // namespace stg
