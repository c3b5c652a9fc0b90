// Draft tree construction (Alg. 1): confidence stratification of the accepted block state,
// top-k expansion at the first level, top-1 expansion deeper, each level pruned to its width
// by path confidence.  One wave per sequence, lane = block position (L <= 64).
//
// Every node of a level fills the same position: nodes differ only in the candidate chosen at
// the first level's position, and all nodes of a level have the same masked set.  So the
// positions visited are the low-confidence positions in rank order (q_1, q_2, ...), level 1
// holds candidates 0 .. c_1-1 at q_1 (their scores fall with the candidate index, so pruning
// keeps a prefix), and level l extends the first c_l nodes of level l-1 by the top-1 token at
// q_l (equal increments keep the parents' order).  Node (l, i) is the root with q_1 set to
// candidate i and q_2 .. q_l set to their top-1 tokens; its parent is node (l-1, i).
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kTreeThreads = 64;
constexpr int kTreeMaxBlock = 64;
constexpr int kTreeMaxK = 8;

struct TreeParams {
    const int32_t* state;  // [B,L]
    const int32_t* leaf;   // [B] or null
    const float* conf;     // [B,n_prev,L,k]
    const int32_t* idx;    // [B,n_prev,L,k]
    const float* conf0;    // [B,L,k]
    const int32_t* idx0;   // [B,L,k]
    int32_t* tokens;       // [B,n_max,L]
    int32_t* parent;       // [B,n_max]
    int32_t* n_nodes;      // [B]
    float* score;          // [B,n_max] or null
    float* conf_next;      // [B,L,k] or null
    int32_t* idx_next;     // [B,L,k] or null
    int B, L, k, n_prev, width, depth, branch, full, n_max;
    float tau;
};

// Kept width of level l (1-based).
__device__ __forceinline__ int tree_level_width(const TreeParams& P, int l) {
    return P.full ? P.width : max(P.width - l + 1, 1);
}

__global__ __launch_bounds__(kTreeThreads) void build_tree_kernel(TreeParams P) {
    __shared__ int pos[kTreeMaxBlock];  // low-confidence positions by rank
    const int b = blockIdx.x;
    const int p = threadIdx.x;
    const int L = P.L, k = P.k;
    const bool in = p < L;

    int lf = P.leaf != nullptr ? P.leaf[b] : -1;
    if (lf < -1 || lf >= P.n_prev) {
        if (p == 0) flag_device_status(2);
        lf = -1;
    }
    const float* C = lf >= 0 ? P.conf + (((int64_t)b * P.n_prev + lf) * L) * k : P.conf0 + (int64_t)b * L * k;
    const int32_t* I = lf >= 0 ? P.idx + (((int64_t)b * P.n_prev + lf) * L) * k : P.idx0 + (int64_t)b * L * k;

    const int s = in ? P.state[(int64_t)b * L + p] : 0;
    const float c0 = in ? C[p * k] : 0.f;
    const int top1 = in ? I[p * k] : 0;
    const bool masked = in && s == -1;
    const bool hi = masked && c0 > P.tau;
    const bool low = masked && !hi;
    const uint64_t hmask = ballot64(hi);
    const uint64_t lmask = ballot64(low);
    if (in && P.conf_next != nullptr) {
        for (int j = 0; j < k; ++j) {
            P.conf_next[((int64_t)b * L + p) * k + j] = C[p * k + j];
            P.idx_next[((int64_t)b * L + p) * k + j] = I[p * k + j];
        }
    }

    // rank of this low position: low positions of larger confidence, or equal confidence
    // and smaller index, come first
    int rank = 0;
    for (int q = 0; q < L; ++q) {
        const float cq = __shfl(c0, q);
        const bool lq = ((lmask >> q) & 1ull) != 0ull;
        rank += (lq && (cq > c0 || (cq == c0 && q < p))) ? 1 : 0;
    }
    if (low) pos[rank] = p;
    __syncthreads();
    const int nlow = __popcll(lmask);

    const int root_tok = hi ? top1 : s;
    int32_t* tok_b = P.tokens + (int64_t)b * P.n_max * L;
    int32_t* par_b = P.parent + (int64_t)b * P.n_max;
    float* sc_b = P.score != nullptr ? P.score + (int64_t)b * P.n_max : nullptr;

    int n = 0;
    const bool has_root = hmask != 0ull;
    if (has_root) {
        if (in) tok_b[p] = root_tok;
        if (p == 0) {
            par_b[0] = -1;
            if (sc_b != nullptr) sc_b[0] = 0.f;
        }
        n = 1;
    }
    const int base = has_root ? 0 : -1;
    float sc[kTreeMaxK];  // scores of the previous level's nodes (uniform)
    int prev_first = 0, cnt = 0;
    const int q1 = nlow > 0 ? pos[0] : -1;
    for (int l = 1; l <= P.depth && l <= nlow; ++l) {
        const int ql = pos[l - 1];
        const int w = tree_level_width(P, l);
        const int c = l == 1 ? min(P.branch, w) : min(w, cnt);
        const float inc = l == 1 ? 0.f : logf(C[ql * k]);
#pragma unroll
        for (int i = 0; i < kTreeMaxK; ++i) {
            if (i >= c) break;
            const int node = n + i;
            int t = root_tok;
            if (p == q1) {
                t = I[p * k + i];
            } else if (low && rank >= 1 && rank < l) {
                t = top1;
            }
            if (in) tok_b[(int64_t)node * L + p] = t;
            const float s_node = l == 1 ? logf(C[q1 * k + i]) : sc[i] + inc;
            sc[i] = s_node;
            if (p == 0) {
                par_b[node] = l == 1 ? base : prev_first + i;
                if (sc_b != nullptr) sc_b[node] = s_node;
            }
        }
        prev_first = n;
        n += c;
        cnt = c;
    }
    for (int node = n; node < P.n_max; ++node) {
        if (in) tok_b[(int64_t)node * L + p] = s;
        if (p == 0) {
            par_b[node] = -1;
            if (sc_b != nullptr) sc_b[node] = -__builtin_huge_valf();
        }
    }
    if (p == 0) P.n_nodes[b] = n;
}

}  // namespace trajspec
