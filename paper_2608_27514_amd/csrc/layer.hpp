// One verification layer around the trajectory-masked attention (a pre-norm decoder layer of
// the 8B-shaped diffusion LMs the method runs on): the elementwise kernels between the
// library GEMMs.  All activations are bf16 in HBM, arithmetic in fp32.
//   rmsnorm_kernel     out = x / sqrt(mean(x^2) + eps) * w            (one workgroup per token)
//   rope_split_kernel  [q | k | v] rows of the QKV projection -> q, k_draft, v_draft in the
//                      attention's layouts, rotary position embedding on q and k (pairs d and
//                      d + D/2, angle = pos * theta^(-2d/D)); token p of every draft of a block
//                      sits at position pos0[b] + p (the drafts are alternative states of the
//                      same block)
//   swiglu_kernel      act = silu(gate) * up from the [gate | up] rows of the gate/up projection
//   cache_gather_kernel  the dual-cache refresh's copy of the rotated K / V rows outside the
//                      current block into the prefix | suffix cache
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kLayerThreads = 256;
constexpr int kLayerMaxHalf = 64;  // D / 2 for the head sizes the attention supports (64, 128)

__device__ __forceinline__ uint16_t f2bf(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);  // round to nearest even
}

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = 0.f;
    for (int w = 0; w < kLayerThreads / 64; ++w) t += red[w];
    __syncthreads();
    return t;
}

// x, out: [T, hidden] bf16 (rows contiguous); w: [hidden].  hidden % 8 == 0.
__global__ __launch_bounds__(kLayerThreads) void rmsnorm_kernel(const uint16_t* __restrict__ x,
                                                                const uint16_t* __restrict__ w,
                                                                uint16_t* __restrict__ out, int hidden, float eps) {
    __shared__ float red[kLayerThreads / 64];
    const uint16_t* xr = x + (int64_t)blockIdx.x * hidden;
    uint16_t* orow = out + (int64_t)blockIdx.x * hidden;
    const int nv = hidden / 8;
    float ss = 0.f;
    for (int i = threadIdx.x; i < nv; i += kLayerThreads) {
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(xr + 8 * i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = bf16_lo(v[e]), b = bf16_hi(v[e]);
            ss += a * a + b * b;
        }
    }
    const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)hidden + eps);
    for (int i = threadIdx.x; i < nv; i += kLayerThreads) {
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(xr + 8 * i);
        const u32x4_t g = *reinterpret_cast<const u32x4_t*>(w + 8 * i);
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = bf16_lo(v[e]) * inv * bf16_lo(g[e]);
            const float b = bf16_hi(v[e]) * inv * bf16_hi(g[e]);
            o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
        }
        *reinterpret_cast<u32x4_t*>(orow + 8 * i) = o;
    }
}

// qkv: [T, (Hq + 2 Hkv) D] rows [q heads | k heads | v heads]; token t = (b N + n) L + p.
// q: [T, Hq, D], kd / vd: [T, Hkv, D].  One workgroup per token: the D / 2 rotation angles
// depend on the position only, so they are computed once per token (into LDS) for all heads;
// every head then moves 16-byte chunks (8 elements of the first half and the matching 8 of the
// second).  D % 16 == 0.
__global__ __launch_bounds__(kLayerThreads) void rope_split_kernel(const uint16_t* __restrict__ qkv,
                                                                   const int32_t* __restrict__ pos0,
                                                                   uint16_t* __restrict__ q, uint16_t* __restrict__ kd,
                                                                   uint16_t* __restrict__ vd, int NL, int L, int Hq,
                                                                   int Hkv, int D, float log2_theta) {
    __shared__ float cs[kLayerMaxHalf], sn[kLayerMaxHalf];
    const int t = blockIdx.x;
    const int b = t / NL;
    const int p = t % L;
    const float pos = (float)(pos0 != nullptr ? pos0[b] + p : p);
    const int half = D / 2;
    for (int d = threadIdx.x; d < half; d += kLayerThreads) {
        const float inv_freq = exp2f(-(2.0f * d / (float)D) * log2_theta);
        sincosf(pos * inv_freq, &sn[d], &cs[d]);
    }
    __syncthreads();
    const int width = (Hq + 2 * Hkv) * D;
    const uint16_t* row = qkv + (int64_t)t * width;
    // rotated pairs of the q and k heads: task = (head, chunk of 8 in the first half)
    const int cpr = half / 8;  // chunks per half
    for (int i = threadIdx.x; i < (Hq + Hkv) * cpr; i += kLayerThreads) {
        const int head = i / cpr, d0 = 8 * (i - head * cpr);
        const uint16_t* src = row + head * D;
        const u32x4_t a = *reinterpret_cast<const u32x4_t*>(src + d0);
        const u32x4_t c = *reinterpret_cast<const u32x4_t*>(src + d0 + half);
        u32x4_t lo, hi;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int d = d0 + 2 * e;
            const float x1a = bf16_lo(a[e]), x1b = bf16_hi(a[e]);
            const float x2a = bf16_lo(c[e]), x2b = bf16_hi(c[e]);
            lo[e] = (uint32_t)f2bf(x1a * cs[d] - x2a * sn[d]) | ((uint32_t)f2bf(x1b * cs[d + 1] - x2b * sn[d + 1]) << 16);
            hi[e] = (uint32_t)f2bf(x2a * cs[d] + x1a * sn[d]) | ((uint32_t)f2bf(x2b * cs[d + 1] + x1b * sn[d + 1]) << 16);
        }
        uint16_t* dst = head < Hq ? q + ((int64_t)t * Hq + head) * D : kd + ((int64_t)t * Hkv + (head - Hq)) * D;
        *reinterpret_cast<u32x4_t*>(dst + d0) = lo;
        *reinterpret_cast<u32x4_t*>(dst + d0 + half) = hi;
    }
    // v heads: copied in 16-byte chunks
    const uint16_t* vsrc = row + (Hq + Hkv) * D;
    uint16_t* vdst = vd + (int64_t)t * Hkv * D;
    for (int i = threadIdx.x; i < Hkv * D / 8; i += kLayerThreads)
        *reinterpret_cast<u32x4_t*>(vdst + 8 * i) = *reinterpret_cast<const u32x4_t*>(vsrc + 8 * i);
}

// gu: [T, 2 I] rows [gate | up]; act: [T, I].  Grid-stride over the T * I / 8 chunks of
// 8 elements (I % 8 == 0).
__global__ __launch_bounds__(kLayerThreads) void swiglu_kernel(const uint16_t* __restrict__ gu,
                                                               uint16_t* __restrict__ act, int64_t T, int I) {
    const int cpr = I / 8;  // chunks per row
    const int64_t total = T * cpr;
    for (int64_t q = (int64_t)blockIdx.x * kLayerThreads + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * kLayerThreads) {
        const int64_t t = q / cpr;
        const int i = (int)(q - t * cpr);
        const u32x4_t g = *reinterpret_cast<const u32x4_t*>(gu + t * 2 * I + 8 * i);
        const u32x4_t u = *reinterpret_cast<const u32x4_t*>(gu + t * 2 * I + I + 8 * i);
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float g0 = bf16_lo(g[e]), g1 = bf16_hi(g[e]);
            const float a = g0 / (1.0f + __expf(-g0)) * bf16_lo(u[e]);
            const float c = g1 / (1.0f + __expf(-g1)) * bf16_hi(u[e]);
            o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(c) << 16);
        }
        *reinterpret_cast<u32x4_t*>(act + t * I + 8 * i) = o;
    }
}

// Dual-cache refresh: the rotated K and V rows of every position outside the current block go
// to the cache, prefix rows then suffix rows.  kd / vd: [B, T, Hkv D] (T = S + L positions);
// caches: [B, S, Hkv D]; block_start[b] in [0, S] (a value outside is reported and clamped).
// Grid-stride over the B * S * Hkv D / 8 chunks of 8 elements.
__global__ __launch_bounds__(kLayerThreads) void cache_gather_kernel(const uint16_t* __restrict__ kd,
                                                                     const uint16_t* __restrict__ vd,
                                                                     const int32_t* __restrict__ block_start,
                                                                     uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                                     int B, int S, int L, int width) {
    const int cpr = width / 8;  // chunks per key row
    const int64_t total = (int64_t)B * S * cpr;
    const int T = S + L;
    for (int64_t q = (int64_t)blockIdx.x * kLayerThreads + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * kLayerThreads) {
        const int64_t row = q / cpr;  // b S + s
        const int c = (int)(q - row * cpr);
        const int b = (int)(row / S);
        const int sp = (int)(row - (int64_t)b * S);
        int bs = block_start[b];
        if (bs < 0 || bs > S) {
            if (sp == 0 && c == 0) flag_device_status(4);
            bs = bs < 0 ? 0 : S;
        }
        const int t = sp < bs ? sp : sp + L;  // position in the sequence
        const int64_t src = ((int64_t)b * T + t) * width + 8 * c;
        const int64_t dst = row * width + 8 * c;
        *reinterpret_cast<u32x4_t*>(kc + dst) = *reinterpret_cast<const u32x4_t*>(kd + src);
        *reinterpret_cast<u32x4_t*>(vc + dst) = *reinterpret_cast<const u32x4_t*>(vd + src);
    }
}

}  // namespace trajspec
