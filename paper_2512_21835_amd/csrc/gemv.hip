// Per-projection decode kernels (one launch per projection); the device code is in gemv_device.h.
#include <hip/hip_ext.h>

#include "gemv_device.h"

namespace stg {
namespace {

using namespace gemv_dev;
constexpr int kMaxRowsPerLaunch = 8;

template <int M, int R, int MODE>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
    const Prefetch<MODE, R, 1> none{};
    gemv_wave<M, R, MODE, 1>(a, (blockIdx.x * kWaves + (threadIdx.x >> 6)) * R, false, none);
}

template <int M, int R, int MODE>
void launch_one(const GemvArgs &c, int grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    if (e0 || e1)
        hipExtLaunchKernelGGL((gemv_kernel<M, R, MODE>), dim3(grid), dim3(256), 0, st, e0, e1, 0, c);
    else
        hipLaunchKernelGGL((gemv_kernel<M, R, MODE>), dim3(grid), dim3(256), 0, st, c);
}

template <int MODE, int R>
hipError_t launch_mode(GemvArgs a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    const int units = MODE == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N;
    const int grid = (units + kWaves * R - 1) / (kWaves * R);
    const int total = a.rows;
    for (int r0 = 0; r0 < total; r0 += kMaxRowsPerLaunch) {
        GemvArgs c = a;
        c.rows = min(kMaxRowsPerLaunch, total - r0);
        c.row0 = a.row0 + r0;
        c.act = a.act + (size_t)r0 * a.act_ld;
        c.out = a.out + (size_t)r0 * a.out_ld;
        if (a.res) c.res = a.res + (size_t)r0 * a.out_ld;
        hipEvent_t e0 = r0 == 0 ? ev_start : nullptr;
        hipEvent_t e1 = r0 + kMaxRowsPerLaunch >= total ? ev_stop : nullptr;
        if (c.rows == 1)
            launch_one<1, R, MODE>(c, grid, st, e0, e1);
        else if (c.rows == 2)
            launch_one<2, R, MODE>(c, grid, st, e0, e1);
        else if (c.rows <= 4)
            launch_one<4, R, MODE>(c, grid, st, e0, e1);
        else
            launch_one<8, R, MODE>(c, grid, st, e0, e1);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_gemv(int mode, GemvArgs a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    if (a.rows <= 0) return hipSuccess;
    // Two units per wavefront pay off once a matrix is large (measured on the 70B-shaped layer:
    // one unit per wavefront leaves the long rows of the down projection short of loads in
    // flight); one unit per wavefront keeps more wavefronts busy on the smaller ones.
    const long units = mode == GEMV_NORM_ROPE_KV ? a.N / 2 : a.N;
    const bool big = units * (long)a.K >= 200L * 1000 * 1000;
    switch (mode) {
        case GEMV_NORM_STORE:
            return big ? launch_mode<GEMV_NORM_STORE, 2>(a, st, ev_start, ev_stop)
                       : launch_mode<GEMV_NORM_STORE, 1>(a, st, ev_start, ev_stop);
        case GEMV_PLAIN_RESIDUAL:
            return big ? launch_mode<GEMV_PLAIN_RESIDUAL, 2>(a, st, ev_start, ev_stop)
                       : launch_mode<GEMV_PLAIN_RESIDUAL, 1>(a, st, ev_start, ev_stop);
        case GEMV_NORM_SWIGLU:
            return big ? launch_mode<GEMV_NORM_SWIGLU, 2>(a, st, ev_start, ev_stop)
                       : launch_mode<GEMV_NORM_SWIGLU, 1>(a, st, ev_start, ev_stop);
        case GEMV_NORM_ROPE_KV:
            return big ? launch_mode<GEMV_NORM_ROPE_KV, 2>(a, st, ev_start, ev_stop)
                       : launch_mode<GEMV_NORM_ROPE_KV, 1>(a, st, ev_start, ev_stop);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace stg
