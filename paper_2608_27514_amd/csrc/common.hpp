// Shared device helpers for the gfx950 kernels of libtrajspec.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace trajspec {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

// Per-device status word (TRAJ_DEV_* bits); kernels OR into it with vector atomics.
__device__ int32_t g_device_status;

__device__ __forceinline__ void flag_device_status(int32_t bits) {
    atomicOr(&g_device_status, bits);
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits16) {
    return __builtin_bit_cast(float, bits16 << 16);
}

// Low / high bf16 of a packed dword as fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }

__device__ __forceinline__ uint64_t ballot64(bool p) { return __ballot(p); }
__device__ __forceinline__ bool ballot64_all(bool p) { return __ballot(!p) == 0ull; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// XCD-aware workgroup order: the dispatcher hands workgroup i to XCD (i % 8).  Returning
// a logical id such that the workgroups that land on one XCD get consecutive logical ids
// keeps the tiles that share K/V (consecutive logical ids) in one XCD's L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    constexpr int kXcd = 8;
    const int per = nblocks / kXcd;          // full rounds
    const int rem = nblocks - per * kXcd;    // XCDs that get one extra block
    const int xcd = bid % kXcd;
    const int slot = bid / kXcd;
    // XCDs [0, rem) own per+1 logical ids, the others own per.
    const int base = xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per;
    return base + slot;
}

}  // namespace trajspec
