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
// lane i of each row of 16 reads lane 15 - i; of each half-row of 8, lane 7 - i
constexpr int DPP_ROW_MIRROR = 0x140;
constexpr int DPP_ROW_HALF_MIRROR = 0x141;

__device__ __forceinline__ uint32_t quad_max_u32(uint32_t v) {
    v = max(v, dpp_u32<QP_XOR1>(v));
    v = max(v, dpp_u32<QP_XOR2>(v));
    return v;
}

// quotient by an invariant divisor d >= 1 (Granlund and Montgomery, "Division by invariant
// integers using multiplication", 1994): l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1,
// n / d = (mulhi(n, m) + n) >> l for every 32-bit n
struct Div32 {
    uint32_t m;
    int l;
};

__device__ __forceinline__ uint32_t div32(uint32_t n, Div32 d) {
    return (uint32_t)(((uint64_t)__umulhi(n, d.m) + n) >> d.l);
}

inline Div32 make_div32(uint32_t d) {
    int l = 0;
    while ((1ull << l) < d) l++;
    Div32 r;
    r.m = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
    r.l = l;
    return r;
}

// streaming (non-temporal) global loads and stores: data touched once
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <bool NT>
__device__ __forceinline__ uint4 ld16(const uint4* p) {
    if (!NT) return *p;
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

template <bool NT>
__device__ __forceinline__ void st4(uint32_t* p, uint32_t x) {
    if (!NT) *p = x;
    else __builtin_nontemporal_store(x, p);
}

template <bool NT>
__device__ __forceinline__ void st8(uint8_t* p, uint32_t x, uint32_t y) {
    if (!NT) {
        *reinterpret_cast<uint2*>(p) = make_uint2(x, y);
    } else {
        u32x2 v;
        v.x = x;
        v.y = y;
        __builtin_nontemporal_store(v, reinterpret_cast<u32x2*>(p));
    }
}

template <bool NT>
__device__ __forceinline__ void st16(void* p, uint32_t x, uint32_t y, uint32_t z, uint32_t w) {
    if (!NT) {
        *reinterpret_cast<uint4*>(p) = make_uint4(x, y, z, w);
    } else {
        u32x4 v;
        v.x = x;
        v.y = y;
        v.z = z;
        v.w = w;
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
    }
}

}  // namespace curvefp
