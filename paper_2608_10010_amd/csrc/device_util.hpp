// Small device helpers shared by the libcurvefp kernels.
#pragma once

#include <cstdint>
#include <hip/hip_runtime.h>

namespace curvefp {

// DPP quad permutes: lane i of each group of four reads lane perm[i].
// quad_perm control = p0 | p1 << 2 | p2 << 4 | p3 << 6.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)0, (int)v, CTRL, 0xF, 0xF, false);
}
constexpr int QP_XOR1 = 1 | (0 << 2) | (3 << 4) | (2 << 6);   // [1,0,3,2]
constexpr int QP_XOR2 = 2 | (3 << 2) | (0 << 4) | (1 << 6);   // [2,3,0,1]
constexpr int QP_NEXT = 1 | (2 << 2) | (3 << 4) | (3 << 6);   // [1,2,3,3]

__device__ __forceinline__ uint32_t quad_max_u32(uint32_t v) {
    v = max(v, dpp_u32<QP_XOR1>(v));
    v = max(v, dpp_u32<QP_XOR2>(v));
    return v;
}

}  // namespace curvefp
