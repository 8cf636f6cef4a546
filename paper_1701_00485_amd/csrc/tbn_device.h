// tbn_device.h -- device-side building blocks shared by the gfx950 kernels:
// bf16 conversion, the two-bit decode, MFMA fragment types and the launch geometry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tbn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// fp32 -> bf16 bits, round to nearest even (the gfx950 conversion instruction).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Two bf16 values packed low/high into one 32-bit word (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v;
    v.x = (__bf16)lo;
    v.y = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// Decode four bf16 pairs (8 consecutive elements) from one packed word.
//   `w` is the packed word already shifted right by 4*half (half = which 8 of its 16
//   elements), `base` the bf16 pair every code multiplies: 0x3F803F80 (= 1.0, 1.0) for
//   the plain codes, or (bf16(a_lo), bf16(a_hi)) for codes scaled by a positive a.
//   Bit 7/23 of the pair gets the magnitude bit (exponent + 1 = times 2) and bit 15/31
//   the sign bit (times -1); adding them to the base multiplies it by the code exactly.
__device__ __forceinline__ u32x4 decode8(uint32_t w, u32x4 base) {
    u32x4 r;
    r.x = ((w & 0x01010101u) << 7) + base.x;
    r.y = ((w & 0x02020202u) << 6) + base.y;
    r.z = ((w & 0x04040404u) << 5) + base.z;
    r.w = ((w & 0x08080808u) << 4) + base.w;
    return r;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).  This
// maps dispatch index b of nblocks to a work index such that every XCD receives one
// contiguous range of work indices, keeping neighbouring tiles in one L2.
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nblocks) {
    constexpr int64_t kXcd = 8;
    const int64_t per = nblocks / kXcd, rem = nblocks % kXcd;
    const int64_t xcd = b % kXcd, local = b / kXcd;
    return xcd * per + (xcd < rem ? xcd : rem) + local;
}

}  // namespace tbn
