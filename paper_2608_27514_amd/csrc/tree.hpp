// Draft tree construction (Alg. 1): confidence stratification of the accepted block state,
// top-k expansion at the first level, deeper levels expanded with the top `branch_deep`
// candidates (1 = the hybrid top-1 policy), each level pruned to its width by path confidence.
// One wave per sequence, lane = block position (L <= 64).
//
// All nodes of a level share their masked set (every level fills one position, the same for
// all of its nodes), so level l fills q_l, the l-th low-confidence position in rank order.
// Level l's candidates are (kept node i of level l-1, candidate j of q_l) in generation order
// (i major); each is ranked by score (sum of logf of the chosen confidences, fp32) with
// generation order breaking ties, and the first w_l ranks become the level's nodes.  Node
// states are built in LDS (a node's row = its parent's row plus one position) and written out
// at the end.
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kTreeThreads = 64;
constexpr int kTreeMaxBlock = 64;
constexpr int kTreeMaxNodes = 64;
constexpr int kTreeMaxK = 8;
constexpr int kTreeMaxCand = kTreeMaxNodes * kTreeMaxK;  // candidates of one level

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
    int B, L, k, n_prev, width, depth, branch, branch_deep, full, n_max;
    float tau;
};

// Kept width of level l (1-based).
__device__ __forceinline__ int tree_level_width(const TreeParams& P, int l) {
    return P.full ? P.width : max(P.width - l + 1, 1);
}

__global__ __launch_bounds__(kTreeThreads) void build_tree_kernel(TreeParams P) {
    __shared__ int pos[kTreeMaxBlock];                 // low-confidence positions by rank
    __shared__ int tok[kTreeMaxNodes][kTreeMaxBlock];  // node states
    __shared__ int par[kTreeMaxNodes];
    __shared__ float nsc[kTreeMaxNodes];               // node scores
    __shared__ float csc[kTreeMaxCand];                // candidate scores of the current level
    __shared__ int cnode[kTreeMaxCand];                // candidate -> new node slot, -1 if pruned
    __shared__ float cs[kTreeMaxBlock][kTreeMaxK];     // the state's candidates, staged once
    __shared__ int is[kTreeMaxBlock][kTreeMaxK];
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
    const bool masked = in && s == -1;
    const bool hi = masked && c0 > P.tau;
    const bool low = masked && !hi;
    const uint64_t hmask = ballot64(hi);
    const uint64_t lmask = ballot64(low);
    if (in) {
        for (int j = 0; j < k; ++j) {
            cs[p][j] = C[p * k + j];
            is[p][j] = I[p * k + j];
        }
        if (P.conf_next != nullptr) {
            for (int j = 0; j < k; ++j) {
                P.conf_next[((int64_t)b * L + p) * k + j] = cs[p][j];
                P.idx_next[((int64_t)b * L + p) * k + j] = is[p][j];
            }
        }
    }

    // rank of this low position: larger confidence first, then smaller index
    int rank = 0;
    for (int q = 0; q < L; ++q) {
        const float cq = __shfl(c0, q);
        const bool lq = ((lmask >> q) & 1ull) != 0ull;
        rank += (lq && (cq > c0 || (cq == c0 && q < p))) ? 1 : 0;
    }
    if (low) pos[rank] = p;
    const int nlow = __popcll(lmask);
    const int root_tok = hi ? is[p][0] : s;

    int n = 0;
    const bool has_root = hmask != 0ull;
    if (has_root) {
        if (in) tok[0][p] = root_tok;
        if (p == 0) {
            par[0] = -1;
            nsc[0] = 0.f;
        }
        n = 1;
    }
    __syncthreads();
    int prev_first = 0, prev_cnt = 1;  // level 0: the root (node 0, or the state itself)
    for (int l = 1; l <= P.depth && l <= nlow; ++l) {
        const int q = pos[l - 1];
        const int bl = l == 1 ? P.branch : P.branch_deep;
        const int M = prev_cnt * bl;
        const int w = tree_level_width(P, l);
        for (int m = p; m < M; m += kTreeThreads) {
            const int i = m / bl, j = m - i * bl;
            const float base = (l == 1) ? 0.f : nsc[prev_first + i];
            csc[m] = base + logf(cs[q][j]);
        }
        __syncthreads();
        for (int m = p; m < M; m += kTreeThreads) {
            const float sm = csc[m];
            int r = 0;
            for (int m2 = 0; m2 < M; ++m2) {
                const float s2 = csc[m2];
                r += (s2 > sm || (s2 == sm && m2 < m)) ? 1 : 0;
            }
            const int slot = r < w ? n + r : -1;
            cnode[m] = slot;
            if (slot >= 0) {
                const int i = m / bl;
                par[slot] = (l == 1) ? (has_root ? 0 : -1) : prev_first + i;
                nsc[slot] = sm;
            }
        }
        __syncthreads();
        // node states: the parent's row with q set to the chosen candidate
        for (int m = 0; m < M; ++m) {
            const int slot = cnode[m];
            if (slot < 0) continue;
            const int i = m / bl, j = m - i * bl;
            const int src = (l == 1) ? -1 : prev_first + i;
            int t = src < 0 ? root_tok : tok[src][in ? p : 0];
            if (p == q) t = is[q][j];
            if (in) tok[slot][p] = t;
        }
        __syncthreads();
        const int c = min(w, M);
        prev_first = n;
        prev_cnt = c;
        n += c;
    }

    int32_t* tok_b = P.tokens + (int64_t)b * P.n_max * L;
    for (int node = 0; node < P.n_max; ++node) {
        if (in) tok_b[(int64_t)node * L + p] = node < n ? tok[node][p] : s;
    }
    for (int node = p; node < P.n_max; node += kTreeThreads) {
        P.parent[(int64_t)b * P.n_max + node] = node < n ? par[node] : -1;
        if (P.score != nullptr) P.score[(int64_t)b * P.n_max + node] = node < n ? nsc[node] : -__builtin_huge_valf();
    }
    if (p == 0) P.n_nodes[b] = n;
}

}  // namespace trajspec
