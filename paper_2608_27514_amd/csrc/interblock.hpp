// Inter-block speculation trigger (Sec. 3.4 "Trigger condition"): per sequence, the top-1
// confidences of the current block B_t and of the next block B_{t+1} (largest c(x) over each
// block's still-masked positions, 0 when none) and the decision c_{t+1} > c_t or
// c_{t+1} > tau, taken only while B_{t+1} has a masked position.  One wave per sequence:
// lane i holds position i of B_t and position L + i of B_{t+1}.
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kTriggerMaxBlock = 64;

struct TriggerParams {
    const int32_t* state;  // [B, 2L]
    const float* conf;     // [B, 2L, k]
    uint8_t* trigger;      // [B]
    float* c_cur;          // [B] or null
    float* c_next;         // [B] or null
    int B, L, k;
    float tau;
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
    return x;
}

__global__ __launch_bounds__(64) void interblock_trigger_kernel(TriggerParams P) {
    const int b = blockIdx.x;
    const int i = threadIdx.x;
    const bool in = i < P.L;
    const int32_t* st = P.state + (int64_t)b * 2 * P.L;
    const float* cf = P.conf + (int64_t)b * 2 * P.L * P.k;
    const bool m_cur = in && st[i] == -1;
    const bool m_next = in && st[P.L + i] == -1;
    const float c_cur = wave_max(m_cur ? cf[(int64_t)i * P.k] : 0.f);
    const float c_next = wave_max(m_next ? cf[(int64_t)(P.L + i) * P.k] : 0.f);
    const bool open = ballot64(m_next) != 0ull;
    if (i == 0) {
        P.trigger[b] = (open && (c_next > c_cur || c_next > P.tau)) ? 1 : 0;
        if (P.c_cur != nullptr) P.c_cur[b] = c_cur;
        if (P.c_next != nullptr) P.c_next[b] = c_next;
    }
}

}  // namespace trajspec
