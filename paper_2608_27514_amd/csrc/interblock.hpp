// Inter-block speculation (Sec. 3.4, App. D).
//
// Trigger ("Trigger condition"): per sequence, the top-1 confidences of the current block B_t
// and of the next block B_{t+1} (largest c(x) over each block's still-masked positions, 0 when
// none) and the decision c_{t+1} > c_t or c_{t+1} > tau, taken only while B_{t+1} has a masked
// position.  One wave per sequence: lane i holds position i of B_t and position L + i of B_{t+1}.
//
// Joint packing ("Joint tree construction"): the trees of B_t (drafts 0 .. n_cur-1) and B_{t+1}
// (drafts n_cur .. n_cur+n_next-1) are verified in one attention pass, and each draft of one tree
// additionally sees the root draft of the other tree.  joint_peers_kernel writes those extra
// visible drafts as the per-draft bit masks the attention kernel ORs into its ancestor masks.
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

constexpr int32_t kDevBadRoot = 0x8;  // a root index outside its tree (taken as 0)

struct JointPeersParams {
    const int32_t* root_cur;   // [B] root draft of B_t's tree, in [0, n_cur), or null (= 0)
    const int32_t* root_next;  // [B] root draft of B_{t+1}'s tree, in [0, n_next), or null (= 0)
    uint64_t* peers;           // [B, n_cur + n_next]
    int B, n_cur, n_next;
};

// One thread per (sequence, draft).
__global__ __launch_bounds__(256) void joint_peers_kernel(JointPeersParams P) {
    const int N = P.n_cur + P.n_next;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)P.B * N) return;
    const int b = (int)(t / N);
    const int n = (int)(t - (int64_t)b * N);
    int rc = P.root_cur != nullptr ? P.root_cur[b] : 0;
    int rn = P.root_next != nullptr ? P.root_next[b] : 0;
    if (rc < 0 || rc >= P.n_cur || rn < 0 || rn >= P.n_next) {
        if (n == 0) flag_device_status(kDevBadRoot);
        if (rc < 0 || rc >= P.n_cur) rc = 0;
        if (rn < 0 || rn >= P.n_next) rn = 0;
    }
    // drafts of B_t see B_{t+1}'s root, drafts of B_{t+1} see B_t's root
    const int other_root = n < P.n_cur ? P.n_cur + rn : rc;
    P.peers[t] = 1ull << other_root;
}

}  // namespace trajspec
