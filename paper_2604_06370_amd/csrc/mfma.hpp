// gfx950 MFMA fragments and small device helpers shared by the attention kernels.
//
// Lane layouts used throughout (64-lane wavefront, lane = 16*grp + col):
//   v_mfma_f32_16x16x32_bf16  A[16 x 32]: lane holds A[col][8*grp .. 8*grp+7]
//                             B[32 x 16]: lane holds B[8*grp .. 8*grp+7][col]
//   v_mfma_f32_16x16x16_bf16  A[16 x 16]: lane holds A[col][4*grp .. 4*grp+3]
//                             B[16 x 16]: lane holds B[4*grp .. 4*grp+3][col]
//   accumulator D[16 x 16]:   lane holds D[4*grp + i][col], i = 0..3
// Because D's per-lane shape equals the A/B shape of the 16x16x16 form (four
// consecutive k for one column), a D tile can feed the next 16x16x16 product
// without any data movement.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fkvk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 mfma32(const u32x4 &a, const u32x4 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(const u32x2 &a, const u32x2 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a), __builtin_bit_cast(s16x4, b), c,
                                                     0, 0, 0);
}

// Two fp32 -> packed bf16 pair (round to nearest even; v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ u32x2 pack4(const f32x4 &x) {
    u32x2 r;
    r.x = pack_bf16(x.x, x.y);
    r.y = pack_bf16(x.z, x.w);
    return r;
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ u32x4 ldg128(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }
__device__ __forceinline__ u32x2 ldg64(const void *p) { return *reinterpret_cast<const u32x2 *>(p); }
// Loads through an address held as an integer (a device-memory pointer read from LDS):
// the global address space keeps them off the LDS counter that generic loads also use.
typedef const u32x4 __attribute__((address_space(1))) *gptr128;
__device__ __forceinline__ u32x4 ldg128_at(uint64_t addr) { return *reinterpret_cast<gptr128>(addr); }

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Zero tokens 4grp+i >= vis of a [.][token] fragment (bf16 pairs).
__device__ __forceinline__ u32x2 mask4(u32x2 v, int vis, int grp) {
    if (4 * grp + 0 >= vis) v.x &= 0xffff0000u;
    if (4 * grp + 1 >= vis) v.x &= 0x0000ffffu;
    if (4 * grp + 2 >= vis) v.y &= 0xffff0000u;
    if (4 * grp + 3 >= vis) v.y &= 0x0000ffffu;
    return v;
}

// Maximum over the four lane groups (lanes l, l^16, l^32, l^48) with the gfx950 lane
// swaps (plain VALU, no LDS round trip).
__device__ __forceinline__ float max_over_groups(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = fmaxf(x, __uint_as_float((threadIdx.x & 32) ? a[0] : a[1]));
    const uint32_t v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return fmaxf(y, __uint_as_float((threadIdx.x & 16) ? b[0] : b[1]));
}

}  // namespace fkvk
