// Persistent decode kernel of one layer: the layer's five phases in one launch.
//
//   phase 0  QKV projection + RoPE + KV store     (needs x: the previous launch)
//   phase 1  decode attention (splits + merge)    (needs phase 0 everywhere: q and the new K/V)
//   phase 2  O projection + residual              (needs phase 1: every head's output)
//   phase 3  gate/up projection + SwiGLU          (needs phase 2: the updated x)
//   phase 4  down projection + residual           (needs phase 3: all of h)
//
// A fixed grid of workgroups, all resident at once (sized with the occupancy API), walks the
// phases in order; phase p's tasks go to workgroups round-robin.  A workgroup signals phase p once,
// after all its phase-p tasks, with a release fence and an atomic increment of the phase counter;
// before its first task of phase p+1 it issues that task's weight loads and only then waits,
// polling the phase-p counter with acquire loads, for every workgroup that had phase-p tasks.
// The weight stream thus continues across phase boundaries and under the latency-bound attention
// phase, where separate kernels would drain and refill the machine five times per layer.
//
// Every wait is bounded: past the spin limit the workgroup raises the abort flag and every
// workgroup stops at its next wait, so a launch always ends; the host turns the flag into an
// error.  The last workgroup to finish phase 4 resets the counters for the next launch.
//
// The projections and the attention are the device code of the per-projection kernels
// (gemv_device.h, attention_device.h) with the same per-output arithmetic, so this kernel and the
// per-projection path give bit-identical results.
#include <hip/hip_runtime.h>

#include "attention_device.h"
#include "gemv_device.h"

namespace stg {
namespace {

using gemv_dev::Prefetch;
using gemv_dev::gemv_prefetch;
using gemv_dev::gemv_wave;

constexpr int kU = 4;       // k steps loaded ahead per wavefront
constexpr int kR = 1;       // units per wavefront
constexpr int kUnitsPerTile = 4 * kR;

__device__ __forceinline__ int tiles_of(int units) { return (units + kUnitsPerTile - 1) / kUnitsPerTile; }

// Waits until `*cnt` reaches `target` (thread 0 polls; the workgroup then proceeds together).
// Returns false if the launch is aborting.
__device__ __forceinline__ bool wait_phase(const DecodeLayerArgs &L, const int *cnt, int target, int *s_flag) {
    if (threadIdx.x == 0) {
        int ok = 1;
        long spins = 0;
        while (true) {
            if (__hip_atomic_load(L.abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) { ok = 0; break; }
            if (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) break;
            __builtin_amdgcn_s_sleep(1);
            if (++spins > L.spin_limit) {
                __hip_atomic_store(L.abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ok = 0;
                break;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        *s_flag = ok;
    }
    __syncthreads();
    return *s_flag != 0;
}

// Publishes this workgroup's phase results.
__device__ __forceinline__ void signal_phase(int *cnt) {
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

template <int M, int MODE>
__device__ __forceinline__ void gemv_phase(const DecodeLayerArgs &L, const GemvArgs &g, int phase, int units,
                                           int *s_flag, bool &alive) {
    const int W = gridDim.x, wg = blockIdx.x, wave = threadIdx.x >> 6;
    const int tiles = tiles_of(units);
    if (wg >= tiles || !alive) return;
    Prefetch<MODE, kR, kU> pre;
    gemv_prefetch<MODE, kR, kU>(g, (wg * 4 + wave) * kR, pre);
    if (phase > 0) {
        const int prev_tasks = L.phase_tasks[phase - 1];
        if (!wait_phase(L, &L.phase[phase - 1], prev_tasks < W ? prev_tasks : W, s_flag)) {
            alive = false;
            return;
        }
    }
    for (int t = wg; t < tiles; t += W) gemv_wave<M, kR, MODE, kU>(g, (t * 4 + wave) * kR, t == wg, pre);
    signal_phase(&L.phase[phase]);
}

template <int M, int G, int D, bool F32KV>
__global__ __launch_bounds__(256) void decode_layer_kernel(DecodeLayerArgs L) {
    __shared__ attn_dev::DecodeSmem<G, D> sm;
    __shared__ int s_flag;
    const int W = gridDim.x, wg = blockIdx.x;
    bool alive = true;

    gemv_phase<M, GEMV_NORM_ROPE_KV>(L, L.qkv, 0, L.qkv.N / 2, &s_flag, alive);

    const int n_attn = L.phase_tasks[1];
    if (wg < n_attn && alive) {
        const int prev = L.phase_tasks[0];
        if (!wait_phase(L, &L.phase[0], prev < W ? prev : W, &s_flag)) {
            alive = false;
        } else {
            const int splits = L.at.grid_splits, hkv = L.at.kv.n_kv_heads;
            for (int t = wg; t < n_attn; t += W) {
                const int split = t % splits, g = (t / splits) % hkv, row = t / (splits * hkv);
                attn_dev::attn_decode_task<G, D, F32KV>(L.at, split, g, row, sm);
                __syncthreads();
            }
            signal_phase(&L.phase[1]);
        }
    }

    gemv_phase<M, GEMV_PLAIN_RESIDUAL>(L, L.o, 2, L.o.N, &s_flag, alive);
    gemv_phase<M, GEMV_NORM_SWIGLU>(L, L.gu, 3, L.gu.N, &s_flag, alive);
    gemv_phase<M, GEMV_PLAIN_RESIDUAL>(L, L.dn, 4, L.dn.N, &s_flag, alive);

    // The last workgroup to finish phase 4 resets the counters for the next launch.  Every
    // workgroup that waits at all has passed its last wait before it could signal phase 4.
    const int last_tasks = L.phase_tasks[4] < W ? L.phase_tasks[4] : W;
    if (alive && wg < L.phase_tasks[4] && threadIdx.x == 0) {
        if (__hip_atomic_load(&L.phase[4], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == last_tasks &&
            __hip_atomic_fetch_add(&L.phase[5], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) == 0) {
            for (int p = 0; p < 6; ++p) __hip_atomic_store(&L.phase[p], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <int M, int G, int D, bool F32KV>
void *kernel_ptr() {
    return reinterpret_cast<void *>(&decode_layer_kernel<M, G, D, F32KV>);
}

template <int M, int G, int D>
void *pick_kv(bool f32) {
    return f32 ? kernel_ptr<M, G, D, true>() : kernel_ptr<M, G, D, false>();
}

template <int M, int D>
void *pick_g(int G, bool f32) {
    switch (G) {
        case 1: return pick_kv<M, 1, D>(f32);
        case 2: return pick_kv<M, 2, D>(f32);
        case 4: return pick_kv<M, 4, D>(f32);
        case 8: return pick_kv<M, 8, D>(f32);
        default: return nullptr;
    }
}

void *pick(int M, int G, int D, bool f32) {
    if (M == 1) return D == 128 ? pick_g<1, 128>(G, f32) : D == 64 ? pick_g<1, 64>(G, f32) : nullptr;
    if (M == 2) return D == 128 ? pick_g<2, 128>(G, f32) : D == 64 ? pick_g<2, 64>(G, f32) : nullptr;
    return nullptr;
}

}  // namespace

void fill_decode_layer_tasks(DecodeLayerArgs &L) {
    const int hkv = L.at.kv.n_kv_heads;
    L.phase_tasks[0] = (L.qkv.N / 2 + kUnitsPerTile - 1) / kUnitsPerTile;
    L.phase_tasks[1] = L.at.grid_splits * hkv * L.at.rows;
    L.phase_tasks[2] = (L.o.N + kUnitsPerTile - 1) / kUnitsPerTile;
    L.phase_tasks[3] = (L.gu.N + kUnitsPerTile - 1) / kUnitsPerTile;
    L.phase_tasks[4] = (L.dn.N + kUnitsPerTile - 1) / kUnitsPerTile;
}

bool decode_layer_supported(int rows, int group, int head_dim) {
    return pick(rows, group, head_dim, false) != nullptr;
}

hipError_t decode_layer_grid(int rows, int group, int head_dim, bool kv_fp32, int *grid) {
    void *k = pick(rows, group, head_dim, kv_fp32);
    if (!k) return hipErrorInvalidValue;
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, 256, 0);
    if (e != hipSuccess) return e;
    if (per_cu < 1) return hipErrorInvalidConfiguration;
    *grid = cus * (per_cu < 2 ? per_cu : 2);
    return hipSuccess;
}

hipError_t launch_decode_layer(const DecodeLayerArgs &L, int grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    void *k = pick(L.qkv.rows, L.at.n_q_heads / L.at.kv.n_kv_heads, L.at.kv.head_dim, L.at.kv_fp32 != 0);
    if (!k) return hipErrorInvalidValue;
    DecodeLayerArgs a = L;
    void *args[] = {&a};
    return hipExtLaunchKernel(k, dim3(grid), dim3(256), args, 0, st, e0, e1, 0);
}

}  // namespace stg
