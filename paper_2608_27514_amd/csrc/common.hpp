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

// Wave reductions run on the lane-exchange network rather than through the LDS crossbar
// (ds_bpermute).  At step t every lane receives two values a, b to combine, its own and a
// partner's in some order: t = 0, 1 pair lanes 1 and 2 apart inside quads (DPP quad
// permutations); t = 2, 3 take the lane 4 and 8 below in the row of 16, cyclically (DPP row
// rotations: once the lanes of each quad agree they combine whole quads); t = 4 pairs rows 0 with
// 1 and 2 with 3, t = 5 the two halves of the wave (gfx950 permlane swaps, which hand each lane
// both values).  Combining with a commutative, associative operation at steps 0 .. 5 leaves the
// wave's result in every lane; steps 0 .. 3 alone reduce each row of 16 lanes.
__device__ __forceinline__ void lane_pair(int step, uint32_t v, uint32_t& a, uint32_t& b) {
    const int iv = (int)v;
    switch (step) {  // a compile-time constant wherever this is inlined into an unrolled loop
    case 0: a = v; b = (uint32_t)__builtin_amdgcn_update_dpp(iv, iv, 0xB1, 0xF, 0xF, false); break;  // quad [1,0,3,2]
    case 1: a = v; b = (uint32_t)__builtin_amdgcn_update_dpp(iv, iv, 0x4E, 0xF, 0xF, false); break;  // quad [2,3,0,1]
    case 2: a = v; b = (uint32_t)__builtin_amdgcn_update_dpp(iv, iv, 0x124, 0xF, 0xF, false); break;  // row_ror:4
    case 3: a = v; b = (uint32_t)__builtin_amdgcn_update_dpp(iv, iv, 0x128, 0xF, 0xF, false); break;  // row_ror:8
    case 4: {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        a = r[0];
        b = r[1];
        break;
    }
    default: {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        a = r[0];
        b = r[1];
        break;
    }
    }
}

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
