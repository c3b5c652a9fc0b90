// Acceptance of the longest consistent trajectory (Sec. 3.3 "Verification procedure"),
// with the threshold-decoding step of Sec. 2.1 and the high-confidence set of Alg. 1
// phase 1.  One 256-thread workgroup per sequence; every per-state / per-draft test is a
// 64-lane wave operation (lane = block position, L <= 64), the walk is a loop of wave
// ballots (lane = draft, N <= 64).
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kAcceptThreads = 256;
constexpr int kMaxDrafts = 64;
constexpr int kMaxBlock = 64;

struct AcceptParams {
    const float* conf;       // [B,N,L,k]
    const int32_t* idx;      // [B,N,L,k]
    const int32_t* tokens;   // [B,N,L]
    const int32_t* parent;   // [B,N]
    const int32_t* committed;// [B,L]
    const float* conf0;      // [B,L,k]
    const int32_t* idx0;     // [B,L,k]
    int32_t* leaf;           // [B]
    uint8_t* on_path;        // [B,N]
    int32_t* n_accepted;     // [B]
    int32_t* out_tokens;     // [B,L]
    uint8_t* hi;             // [B,N,L]
    int B, N, L, k, mode, traversal;
    float tau;
};

__global__ __launch_bounds__(kAcceptThreads) void accept_kernel(AcceptParams P) {
    __shared__ int par[kMaxDrafts];
    __shared__ int expected[kMaxDrafts + 1][kMaxBlock];
    __shared__ int has_step[kMaxDrafts + 1];
    __shared__ int consistent[kMaxDrafts];
    __shared__ int gain[kMaxDrafts];

    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    constexpr int NW = kAcceptThreads / 64;
    const int N = P.N, L = P.L, k = P.k;
    const int32_t MASK = -1;

    // Parents: anything outside [-1, n) is reported and treated as -1.
    for (int n = tid; n < N; n += kAcceptThreads) {
        int q = P.parent[(int64_t)b * N + n];
        if (q < -1 || q >= n) {
            flag_device_status(1);
            q = -1;
        }
        par[n] = q;
    }

    // Threshold step of every state q in [-1, N): one wave per state, one lane per position.
    const bool lane_in = lane < L;
    for (int q = wave - 1; q < N; q += NW) {
        int s = MASK, t1 = 0;
        float c = 0.f;
        if (lane_in) {
            if (q < 0) {
                const int64_t o = (int64_t)b * L + lane;
                s = P.committed[o];
                c = P.conf0[o * k];
                t1 = P.idx0[o * k];
            } else {
                const int64_t o = ((int64_t)b * N + q) * L + lane;
                s = P.tokens[o];
                c = P.conf[o * k];
                t1 = P.idx[o * k];
            }
        }
        const bool masked = lane_in && s == MASK;
        const bool over = masked && c > P.tau;
        const uint64_t mmask = ballot64(masked);
        const uint64_t hmask = ballot64(over);
        if (q >= 0 && lane_in) P.hi[((int64_t)b * N + q) * L + lane] = over ? 1 : 0;
        bool chosen = over;
        if (hmask == 0 && mmask != 0) {
            // fallback: most confident masked position, smallest position on ties
            float bc = masked ? c : -1.0f;
            int bp = masked ? lane : 0x7fffffff;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                const float oc = __shfl_xor(bc, off);
                const int op = __shfl_xor(bp, off);
                if (oc > bc || (oc == bc && op < bp)) {
                    bc = oc;
                    bp = op;
                }
            }
            chosen = lane == bp;
        }
        if (lane_in) expected[q + 1][lane] = chosen ? t1 : s;
        if (lane == 0) has_step[q + 1] = mmask != 0;
    }
    __syncthreads();

    // Consistency of every draft with its parent state; gain w.r.t. the committed state.
    for (int cnode = wave; cnode < N; cnode += NW) {
        const int q = par[cnode];
        int t = MASK, sp = MASK, s0 = MASK;
        if (lane_in) {
            t = P.tokens[((int64_t)b * N + cnode) * L + lane];
            s0 = P.committed[(int64_t)b * L + lane];
            sp = q < 0 ? s0 : P.tokens[((int64_t)b * N + q) * L + lane];
        }
        bool ok;
        bool ok_all;
        if (P.mode == 0) {
            ok = !lane_in || t == expected[q + 1][lane];
            ok_all = has_step[q + 1] && ballot64(!ok) == 0;
        } else {
            const int kk = P.mode == 1 ? 1 : k;
            bool isnew = false;
            if (!lane_in) {
                ok = true;
            } else if (sp != MASK) {
                ok = t == sp;
            } else if (t == MASK) {
                ok = true;
            } else {
                isnew = true;
                ok = false;
                const int32_t* cand = q < 0 ? P.idx0 + ((int64_t)b * L + lane) * k
                                            : P.idx + (((int64_t)b * N + q) * L + lane) * k;
                for (int j = 0; j < kk; ++j) ok = ok || cand[j] == t;
            }
            ok_all = ballot64(!ok) == 0 && ballot64(isnew) != 0;
        }
        const uint64_t gm = ballot64(lane_in && s0 == MASK && t != MASK);
        if (lane == 0) {
            consistent[cnode] = ok_all ? 1 : 0;
            gain[cnode] = __popcll(gm);
        }
    }
    __syncthreads();
    if (wave != 0) return;

    // Walk (lane = draft).
    const bool node_in = lane < N;
    const int my_par = node_in ? par[lane] : -2;
    const bool my_cons = node_in && consistent[lane];
    int leaf = -1;
    if (P.traversal == 0) {
        int cur = -1;
        for (int step = 0; step <= N; ++step) {
            const uint64_t cand = ballot64(my_cons && my_par == cur);
            if (cand == 0) break;
            cur = __ffsll((unsigned long long)cand) - 1;
            leaf = cur;
        }
    } else {
        uint64_t valid = ballot64(my_cons && my_par == -1);
        for (int it = 0; it < N; ++it) {
            const bool v = my_cons && (my_par == -1 || (my_par >= 0 && ((valid >> my_par) & 1ull)));
            const uint64_t nv = ballot64(v);
            if (nv == valid) break;
            valid = nv;
        }
        const bool v = node_in && ((valid >> lane) & 1ull);
        int bg = v ? gain[lane] : -1;
        int bn = v ? lane : 0x7fffffff;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const int og = __shfl_xor(bg, off);
            const int on = __shfl_xor(bn, off);
            if (og > bg || (og == bg && on < bn)) {
                bg = og;
                bn = on;
            }
        }
        leaf = bg >= 0 ? bn : -1;
    }
    uint64_t path = 0;
    for (int j = leaf, hops = 0; j >= 0 && hops <= N; j = par[j], ++hops) path |= 1ull << j;
    if (node_in) P.on_path[(int64_t)b * N + lane] = (path >> lane) & 1ull ? 1 : 0;
    if (lane_in) {
        P.out_tokens[(int64_t)b * L + lane] =
            leaf >= 0 ? P.tokens[((int64_t)b * N + leaf) * L + lane] : P.committed[(int64_t)b * L + lane];
    }
    if (lane == 0) {
        P.leaf[b] = leaf;
        P.n_accepted[b] = leaf >= 0 ? gain[leaf] : 0;
    }
}

}  // namespace trajspec
