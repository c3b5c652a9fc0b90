// Acceptance of the longest consistent trajectory (Sec. 3.3 "Verification procedure"),
// with the threshold-decoding step of Sec. 2.1 and the high-confidence set of Alg. 1
// phase 1.  One 1024-thread workgroup per sequence.  The kernel is latency-bound: every input
// it reads (draft tokens, their top-1 confidences and tokens, the committed state, the parents)
// is first staged into LDS in one round of independent loads, so the sequence pays one memory
// latency instead of one per state and per draft; every per-state / per-draft test is then a
// 64-lane wave operation on LDS (lane = block position, L <= 64, 16 waves in parallel), and the
// walk is a loop of wave ballots (lane = draft, N <= 64).
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kAcceptThreads = 1024;
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

// The wave's best (value, position) pair in every lane: the larger value, then the smaller
// position (T = float or int; positions are non-negative).
template <typename T>
__device__ __forceinline__ void wave_argmax(T& v, int& pos) {
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        uint32_t av, bv, ap, bp;
        lane_pair(t, __builtin_bit_cast(uint32_t, v), av, bv);
        lane_pair(t, (uint32_t)pos, ap, bp);
        const T va = __builtin_bit_cast(T, av), vb = __builtin_bit_cast(T, bv);
        const bool take_b = vb > va || (vb == va && (int)bp < (int)ap);
        v = take_b ? vb : va;
        pos = take_b ? (int)bp : (int)ap;
    }
}

__global__ __launch_bounds__(kAcceptThreads) void accept_kernel(AcceptParams P) {
    // staged inputs, [n * L + p] for draft n (the committed state separately)
    __shared__ int tok[kMaxDrafts * kMaxBlock];
    __shared__ float top_c[kMaxDrafts * kMaxBlock];
    __shared__ int top_t[kMaxDrafts * kMaxBlock];
    __shared__ int s0[kMaxBlock];
    __shared__ float c0[kMaxBlock];
    __shared__ int t0[kMaxBlock];
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
    const int NL = N * L;
    const int32_t MASK = -1;

    // Stage: at most kMaxDrafts * kMaxBlock / kAcceptThreads = 4 elements of each draft array
    // per thread, all loads issued before any is used.
    {
        constexpr int R = kMaxDrafts * kMaxBlock / kAcceptThreads;
        const int64_t base = (int64_t)b * NL;
        int vt[R], vi[R];
        float vc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int e = tid + r * kAcceptThreads;
            if (e < NL) {
                vt[r] = P.tokens[base + e];
                vc[r] = P.conf[(base + e) * k];
                vi[r] = P.idx[(base + e) * k];
            }
        }
        int q = -1, cs = 0, ct = 0;
        float cc = 0.f;
        if (tid < N) q = P.parent[(int64_t)b * N + tid];
        if (tid < L) {
            const int64_t o = (int64_t)b * L + tid;
            cs = P.committed[o];
            cc = P.conf0[o * k];
            ct = P.idx0[o * k];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int e = tid + r * kAcceptThreads;
            if (e < NL) {
                tok[e] = vt[r];
                top_c[e] = vc[r];
                top_t[e] = vi[r];
            }
        }
        // Parents: anything outside [-1, n) is reported and treated as -1.
        if (tid < N) {
            if (q < -1 || q >= tid) {
                flag_device_status(1);
                q = -1;
            }
            par[tid] = q;
        }
        if (tid < L) {
            s0[tid] = cs;
            c0[tid] = cc;
            t0[tid] = ct;
        }
    }
    __syncthreads();

    // Threshold step of every state q in [-1, N): one wave per state, one lane per position.
    const bool lane_in = lane < L;
    for (int q = wave - 1; q < N; q += NW) {
        int s = MASK, t1 = 0;
        float c = 0.f;
        if (lane_in) {
            if (q < 0) {
                s = s0[lane];
                c = c0[lane];
                t1 = t0[lane];
            } else {
                s = tok[q * L + lane];
                c = top_c[q * L + lane];
                t1 = top_t[q * L + lane];
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
            wave_argmax(bc, bp);
            chosen = lane == bp;
        }
        if (lane_in) expected[q + 1][lane] = chosen ? t1 : s;
        if (lane == 0) has_step[q + 1] = mmask != 0;
    }
    __syncthreads();

    // Consistency of every draft with its parent state; gain w.r.t. the committed state.
    for (int cnode = wave; cnode < N; cnode += NW) {
        const int q = par[cnode];
        int t = MASK, sp = MASK, sc = MASK;
        if (lane_in) {
            t = tok[cnode * L + lane];
            sc = s0[lane];
            sp = q < 0 ? sc : tok[q * L + lane];
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
        const uint64_t gm = ballot64(lane_in && sc == MASK && t != MASK);
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
        wave_argmax(bg, bn);
        leaf = bg >= 0 ? bn : -1;
    }
    uint64_t path = 0;
    for (int j = leaf, hops = 0; j >= 0 && hops <= N; j = par[j], ++hops) path |= 1ull << j;
    if (node_in) P.on_path[(int64_t)b * N + lane] = (path >> lane) & 1ull ? 1 : 0;
    if (lane_in) {
        P.out_tokens[(int64_t)b * L + lane] = leaf >= 0 ? tok[leaf * L + lane] : s0[lane];
    }
    if (lane == 0) {
        P.leaf[b] = leaf;
        P.n_accepted[b] = leaf >= 0 ? gain[leaf] : 0;
    }
}

}  // namespace trajspec
