// Cross-lane exchange inside a 64-lane wavefront without the LDS crossbar.  lane_xor(v, o) returns
// the v of lane (lane ^ o), o in {1, 2, 4, 8, 16, 32} -- the value __shfl_xor(v, o, 64) returns,
// which the compiler issues as ds_bpermute_b32 through LDS.  Here: DPP moves within rows of 16
// lanes (quad permutations for 1 and 2, row shifts for 4, a row rotation for 8) and gfx950's
// v_permlane16_swap / v_permlane32_swap across rows.  Every lane of the wavefront must be active.
#pragma once
#include <hip/hip_runtime.h>

namespace stg {

__device__ __forceinline__ int lane_xor_bits(int x, int o) {
    const int lane = __lane_id();
    switch (o) {
        case 1: return __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
        case 2: return __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
        case 4: {
            const int up = __builtin_amdgcn_update_dpp(x, x, 0x104, 0xF, 0xF, false);  // row_shl 4: lane + 4
            const int dn = __builtin_amdgcn_update_dpp(x, x, 0x114, 0xF, 0xF, false);  // row_shr 4: lane - 4
            return (lane & 4) ? dn : up;
        }
        case 8: return __builtin_amdgcn_update_dpp(x, x, 0x128, 0xF, 0xF, false);  // row_ror 8
        case 16: {
            // element 1 holds lane + 16 on the even rows, element 0 lane - 16 on the odd rows
            const auto s = __builtin_amdgcn_permlane16_swap(x, x, false, false);
            return (lane & 16) ? (int)s[0] : (int)s[1];
        }
        default: {
            const auto s = __builtin_amdgcn_permlane32_swap(x, x, false, false);
            return (lane & 32) ? (int)s[0] : (int)s[1];
        }
    }
}

__device__ __forceinline__ float lane_xor(float v, int o) {
    return __int_as_float(lane_xor_bits(__float_as_int(v), o));
}

}  // namespace stg
