// Slot tags (include/stage.h, stage_config.slot_check): a reusable HBM slot is refilled only after
// the kernels reading its previous layer have finished, and read only after its copy completed
// (Section III-C's ready signal and buffer reuse).  With the check on, every block of a slot
// carries a tag {layer, load number}; the copy stream invalidates it before refilling the block
// and writes the new tag after the copy, and the compute stream compares it with what the call
// expects before the block's first kernel and after the layer's last one.
//
// Tags and the check record are written and read with system-scope atomics (coherent across the
// XCDs' L2 caches without relying on kernel-boundary cache maintenance).  No kernel here stops or
// traps: a mismatch is counted, and the first one recorded, for the host to report.
#include "stage_kernels.h"

namespace stg {
namespace {

__global__ void slot_tag_write_kernel(int *tag, int layer, int load) {
    if (threadIdx.x != 0) return;
    __hip_atomic_store(tag, layer, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(tag + 1, load, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// rec: [0] checks run, [1] mismatches, then the first mismatch: [2] where, [3] slot, [4] expected
// layer, [5] expected load, [6] found layer, [7] found load
__global__ void slot_tag_check_kernel(const int *tag, int slot, int layer, int load, int where, int *rec) {
    if (threadIdx.x != 0) return;
    const int got_layer = __hip_atomic_load(tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const int got_load = __hip_atomic_load(tag + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_fetch_add(rec, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    if (got_layer == layer && got_load == load) return;
    if (__hip_atomic_fetch_add(rec + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0) return;
    const int first[6] = {where, slot, layer, load, got_layer, got_load};
    for (int i = 0; i < 6; ++i) __hip_atomic_store(rec + 2 + i, first[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace

hipError_t launch_slot_tag_write(int *tag, int layer, int load, hipStream_t st) {
    STG_LAUNCH(slot_tag_write_kernel, dim3(1), dim3(64), 0, st, tag, layer, load);
    return hipGetLastError();
}

hipError_t launch_slot_tag_check(const int *tag, int slot, int layer, int load, int where, int *rec,
                                 hipStream_t st) {
    STG_LAUNCH(slot_tag_check_kernel, dim3(1), dim3(64), 0, st, tag, slot, layer, load, where, rec);
    return hipGetLastError();
}

}  // namespace stg
