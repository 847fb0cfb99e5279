// Memory-bound projections for decode: y = W x with bf16 weights W [N, K] (row-major) and fp32
// activations, fp32 accumulation.  One pass over the weights serves up to 8 activation rows.
//
// Work split: a workgroup is 4 wavefronts of 64 lanes.  Each wavefront owns R output rows (or R
// gate/up row pairs) over the whole K range; lane l reads 16 bytes (8 bf16) of every owned row at
// k = l*8 + 512*i, so one load instruction covers 1 KiB of contiguous weights per row.  Lane
// partial sums are combined with a butterfly of cross-lane shuffles.
//
// Fused steps: the RMSNorm in front of the QKV and gate/up projections (the sum of squares of
// x is accumulated from the same loads, and the 1/rms scale applied to the dot product), the
// SwiGLU of the gate/up pair, and the residual add after the O and down projections.
//
// Every output element is produced by one fixed sequence of fused multiply-adds and one fixed
// butterfly, whatever the number of activation rows or the row tiling: results do not depend on
// how many micro-batches share a call.
#include "stage_kernels.h"

namespace stg {
namespace {

constexpr int kWaves = 4;
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

template <int M, int R, int MODE>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
    constexpr bool kNorm = (MODE == GEMV_NORM_STORE || MODE == GEMV_NORM_SWIGLU);
    constexpr int NW = (MODE == GEMV_NORM_SWIGLU) ? 2 : 1;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int unit0 = (blockIdx.x * kWaves + wave) * R;
    if (unit0 >= a.N) return;

    const uint16_t *wbase[NW];
    wbase[0] = a.w;
    if (NW == 2) wbase[NW - 1] = a.w2;

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

    for (int k = lane * 8; k < a.K; k += 512) {
        uint4 wv[NW][R];
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int row = min(unit0 + r, a.N - 1);
                wv[w][r] = load_stream16(wbase[w] + (size_t)row * a.K + k);
            }
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
                    unpack8(wv[w][r], f);
#pragma unroll
                    for (int j = 0; j < 8; ++j) acc[w][r][m] = fmaf(f[j], x[j], acc[w][r][m]);
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

    // Epilogue: lane (r * M + m) writes output row unit0 + r of activation row m.
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int m = 0; m < M; ++m) {
            if (lane != r * M + m) continue;
            const int row = unit0 + r;
            if (row >= a.N || m >= a.rows) continue;
            float scale = 1.f;
            if (kNorm) scale = 1.f / sqrtf(ss[m] / (float)a.K + a.eps);
            float *o = a.out + m * a.out_ld + row;
            if (MODE == GEMV_NORM_STORE) {
                *o = acc[0][r][m] * scale;
            } else if (MODE == GEMV_PLAIN_RESIDUAL) {
                *o = a.res[m * a.out_ld + row] + acc[0][r][m];
            } else {
                const float gt = acc[0][r][m] * scale;
                const float up = acc[NW - 1][r][m] * scale;
                *o = gt / (1.f + expf(-gt)) * up;
            }
        }
    }
}

template <int MODE, int R>
hipError_t launch_mode(GemvArgs a, hipStream_t st) {
    const int grid = (a.N + kWaves * R - 1) / (kWaves * R);
    const int total = a.rows;
    for (int r0 = 0; r0 < total; r0 += kMaxRowsPerLaunch) {
        GemvArgs c = a;
        c.rows = min(kMaxRowsPerLaunch, total - r0);
        c.act = a.act + (size_t)r0 * a.act_ld;
        c.out = a.out + (size_t)r0 * a.out_ld;
        if (a.res) c.res = a.res + (size_t)r0 * a.out_ld;
        if (c.rows == 1)
            hipLaunchKernelGGL((gemv_kernel<1, R, MODE>), dim3(grid), dim3(256), 0, st, c);
        else if (c.rows == 2)
            hipLaunchKernelGGL((gemv_kernel<2, R, MODE>), dim3(grid), dim3(256), 0, st, c);
        else if (c.rows <= 4)
            hipLaunchKernelGGL((gemv_kernel<4, R, MODE>), dim3(grid), dim3(256), 0, st, c);
        else
            hipLaunchKernelGGL((gemv_kernel<8, R, MODE>), dim3(grid), dim3(256), 0, st, c);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_gemv(int mode, GemvArgs a, hipStream_t st) {
    if (a.rows <= 0) return hipSuccess;
    switch (mode) {
        case GEMV_NORM_STORE: return launch_mode<GEMV_NORM_STORE, 2>(a, st);
        case GEMV_PLAIN_RESIDUAL: return launch_mode<GEMV_PLAIN_RESIDUAL, 2>(a, st);
        case GEMV_NORM_SWIGLU: return launch_mode<GEMV_NORM_SWIGLU, 1>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace stg
