// Trajectory-masked verification attention (Sec. 3.3) for grids of at most one 4-wave workgroup
// of 32-row waves per CU (one sequence's drafts: 8-32 drafts x 32 heads).
//
// With 32 query rows per wave such a grid holds one wave per SIMD, and that wave alternates on
// its own between the vector ALU (softmax) and the matrix core: about half of each SIMD's cycles
// issue neither.  Here a wave owns 16 query rows and multiplies with v_mfma_f32_16x16x32_bf16,
// so the same rows make twice the waves, two per SIMD on the larger one-sequence grids, whose
// softmax and matrix phases overlap as the two workgroups per CU of the batched grids do.  A
// workgroup of 4 waves owns 64 rows; it stages every cache tile in LDS once for its 4 waves (the
// same stages and loads as the 32-row kernel), and each wave reads whole K / V fragments for 16
// queries instead of 32, i.e. twice the LDS fragment traffic per MFMA, which these grids have to
// spare.
//
// Math layout (v_mfma_f32_16x16x32_bf16, wave64; lane l, lane group q = l / 16)
//   S^T = K Q^T per 16-key block: A = 16 K rows (lane l: key l % 16, head dims 32 ks + 8 q ..
//   + 7), B = Q^T (lane l: query l % 16, the same dims).  The result holds, in lane l, the
//   scores of keys 4 q .. 4 q + 3 of the block for query l % 16: a query's row maximum and sum
//   combine the lanes l, l ^ 16, l ^ 32, l ^ 48 (two lane swaps).
//   O^T += V^T P^T per 32 keys (blocks 2 j, 2 j + 1): the contraction index of the B operand in
//   lane l runs over the keys 4 q .. 4 q + 3 of block 2 j, then of block 2 j + 1, which is
//   exactly what the score layout leaves in the lane (no data movement); the A operand V^T
//   takes the same keys through two transposing LDS reads (rows 4 q .. + 3 and 16 + 4 q .. + 3).
//   O^T in lane l: head dims 16 db + 4 q .. + 3 of query l % 16 (one 8-byte store per block db).
//
// Phases, stage layout, lazy online softmax, ancestor masks and the draft tile walk are those of
// the 32-row kernel (verify_attn.hpp).
#pragma once

#include "verify_attn.hpp"

namespace trajspec {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Per-lane constants of the 16-row kernel.
template <int D>
struct AttnLane16 {
    int kq[D / 32];  // K fragment offset of k-step ks within a 16-key block (block-relative, elements)
    int vq[D / 16];  // V transposing-read offset of head-dim block db within a 32-key group
    int ri;          // row of this lane's chunk within a wave-wide direct load
    int pc;          // LDS chunk slot of this lane within that row
};

__device__ __forceinline__ float swap16_max(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                    false, false);
    const uint32_t a = r[0], b = r[1];
    return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
__device__ __forceinline__ float swap16_sum(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                    false, false);
    const uint32_t a = r[0], b = r[1];
    return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}
// x combined over the four lanes l, l^16, l^32, l^48 that hold one query.
__device__ __forceinline__ float quad_max(float x) { return pair_max(swap16_max(x)); }
__device__ __forceinline__ float quad_sum(float x) { return pair_sum(swap16_sum(x)); }

// Folds a joint maximum mx (already combined over the query's four lanes) into the reference,
// rescaling O and the running sum when it passes the lazy trigger (as fold_max).
template <int D>
__device__ __forceinline__ void fold_max16(float mx, float c, float thr, SoftState& st, f32x4_t (&o)[D / 16]) {
    const bool need = mx > st.mthr;
    if (ballot64(need) != 0ull) {
        const float m_new = need ? mx : st.m;
        const float alpha = need ? fast_exp2((st.m - m_new) * c) : 1.0f;
        st.lsum *= alpha;
#pragma unroll
        for (int db = 0; db < D / 16; ++db) o[db] *= alpha;
        st.m = m_new;
        st.neg_mc = m_new == kNegInf ? 0.f : -m_new * c;
        st.mthr = m_new + thr;
    }
}

// Scores of keys key0 .. key0+15 (one 16-key block) at or beyond S are masked.
__device__ __forceinline__ void mask_tail16(f32x4_t& s, int key0, int S, int q) {
#pragma unroll
    for (int r = 0; r < 4; ++r) s[r] = key0 + 4 * q + r < S ? s[r] : kNegInf;
}

// Softmax phase of a 64-key step (four 16-key blocks): weights against the query's reference,
// with the lazy trigger tested on the lane's weight sum (softmax_phase).  pf[j] receives the bf16
// weights of blocks 2 j, 2 j + 1 in the B-operand order of the PV multiply.
template <int D>
__device__ __forceinline__ void softmax16(const f32x4_t (&s)[4], float c, float thr, SoftState& st,
                                          f32x4_t (&o)[D / 16], bf16x8_t (&pf)[2]) {
    float neg_mc = st.neg_mc;
    float sum = 0.f;
    float p[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        p[v] = fast_exp2(__builtin_fmaf(s[v >> 2][v & 3], c, neg_mc));
        sum += p[v];
    }
    const bool big = !(sum <= (float)(1 << (int)kLazyLog2)) || st.m == kNegInf;
    if (ballot64(big) != 0ull) {
        float mx = kNegInf;
#pragma unroll
        for (int v = 0; v < 16; v += 2)
            mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mx, s[v >> 2][v & 3]), s[v >> 2][(v & 3) + 1]);
        fold_max16<D>(quad_max(mx), c, thr, st, o);
        neg_mc = st.neg_mc;
        sum = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            p[v] = fast_exp2(__builtin_fmaf(s[v >> 2][v & 3], c, neg_mc));
            sum += p[v];
        }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) pf[v >> 3][v & 7] = (__bf16)p[v];
    st.lsum += sum;
}

// Scores of the four 16-key blocks whose K rows start at kbase: four independent MFMA chains,
// each fragment read issued after an MFMA, two MFMAs ahead (see qk_pair).
template <int D>
__device__ __forceinline__ void qk16x4(const uint16_t* kbase, const AttnLane16<D>& ln, const bf16x8_t (&qf)[D / 32],
                                       f32x4_t (&sn)[4]) {
    constexpr int KS = D / 32;
    constexpr int NM = 4 * KS;
    bf16x8_t kf[NM];
    kf[0] = lds16(kbase + ln.kq[0]);
    kf[1] = lds16(kbase + 16 * D + ln.kq[0]);
    f32x4_t a[4] = {{}, {}, {}, {}};
#pragma unroll
    for (int n = 0; n < NM; ++n) {
        a[n & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[n], qf[n >> 2], a[n & 3], 0, 0, 0);
        if (n + 2 < NM) kf[n + 2] = lds16(kbase + ((n + 2) & 3) * 16 * D + ln.kq[(n + 2) >> 2]);
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) sn[j] = a[j];
}

// V^T fragment of head-dim block db for the 32 keys whose V rows start at vbase.
template <int D>
__device__ __forceinline__ bf16x8_t v_frag16(const uint16_t* vbase, const AttnLane16<D>& ln, int db) {
    const bf16x4_t a0 = lds_read_tr(vbase + ln.vq[db]);
    const bf16x4_t a1 = lds_read_tr(vbase + ln.vq[db] + 16 * D);
    return __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
}

// O^T += V^T P^T for the 64 keys whose V rows start at vbase (two groups of 32 keys); each
// fragment is read two MFMAs ahead.
template <int D>
__device__ __forceinline__ void pv16x2(const uint16_t* vbase, const AttnLane16<D>& ln, const bf16x8_t (&pf)[2],
                                       f32x4_t (&o)[D / 16]) {
    constexpr int NDB = D / 16;
    constexpr int NM = 2 * NDB;
    bf16x8_t va[NM];
    va[0] = v_frag16<D>(vbase, ln, 0);
    va[1] = v_frag16<D>(vbase, ln, 1);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
        o[m % NDB] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[m], pf[m / NDB], o[m % NDB], 0, 0, 0);
        if (m + 2 < NM) va[m + 2] = v_frag16<D>(vbase + ((m + 2) / NDB) * 32 * D, ln, (m + 2) % NDB);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Matrix phase of a full step: scores of the next four blocks (K rows at kbase) and O += V P of
// the current 64 keys (V rows at vbase); the first two V fragments ride on the last score MFMAs.
template <int D>
__device__ __forceinline__ void matrix16(const uint16_t* kbase, const uint16_t* vbase, const AttnLane16<D>& ln,
                                         const bf16x8_t (&qf)[D / 32], f32x4_t (&sn)[4], const bf16x8_t (&pf)[2],
                                         f32x4_t (&o)[D / 16]) {
    constexpr int KS = D / 32;
    constexpr int NK = 4 * KS;
    constexpr int NDB = D / 16;
    constexpr int NV = 2 * NDB;
    bf16x8_t kf[NK];
    bf16x8_t va[NV];
    kf[0] = lds16(kbase + ln.kq[0]);
    kf[1] = lds16(kbase + 16 * D + ln.kq[0]);
    f32x4_t a[4] = {{}, {}, {}, {}};
#pragma unroll
    for (int n = 0; n < NK; ++n) {
        a[n & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[n], qf[n >> 2], a[n & 3], 0, 0, 0);
        if (n + 2 < NK) {
            kf[n + 2] = lds16(kbase + ((n + 2) & 3) * 16 * D + ln.kq[(n + 2) >> 2]);
        } else {
            const int m = n + 2 - NK;  // 0, 1
            va[m] = v_frag16<D>(vbase, ln, m);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) sn[j] = a[j];
#pragma unroll
    for (int m = 0; m < NV; ++m) {
        o[m % NDB] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[m], pf[m / NDB], o[m % NDB], 0, 0, 0);
        if (m + 2 < NV) va[m + 2] = v_frag16<D>(vbase + ((m + 2) / NDB) * 32 * D, ln, (m + 2) % NDB);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// One full 64-key step (next stage full): the 16-row counterpart of full_step.
template <int D>
__device__ __forceinline__ void full_step16(int t, const CacheArgs& a, const AttnLane16<D>& ln, const uint16_t* cur,
                                            uint16_t* nxt, const bf16x8_t (&qf)[D / 32], f32x4_t (&s)[4],
                                            SoftState& st, f32x4_t (&o)[D / 16]) {
    using G = AttnGeom<D, 16>;
    stage_dma<D, false, 16>(a.krs, a.vrs, a.kv_stride, t + 1, a.S, a.wave, ln, nxt);
    bf16x8_t pf[2];
    softmax16<D>(s, a.c, a.thr, st, o, pf);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(1);
    matrix16<D>(cur, cur + G::kTileElems, ln, qf, s, pf, o);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
}

// Scores, weights and O += V P of the draft tile k0 .. k0+31 held in the wave's regions kw, vw.
template <int D>
__device__ __forceinline__ void draft_tile16(const DraftArgs& a, int k0, int q, const uint16_t* kw, const uint16_t* vw,
                                             const AttnLane16<D>& ln, const bf16x8_t (&qf)[D / 32], SoftState& st,
                                             f32x4_t (&o)[D / 16], float c, float thr) {
    constexpr int KS = D / 32;
    constexpr int NDB = D / 16;
    const int jlo = k0 / a.L;
    const int jhi = min(a.N - 1, (k0 + 31) / a.L);
    const uint64_t T = (jhi - jlo == 63) ? ~0ull : (((1ull << (jhi - jlo + 1)) - 1) << jlo);
    const bool lane_full = !a.row_valid || ((a.anc & T) == T);
    const bool all_full = ballot64_all(lane_full);
    const bool full = (k0 + 32 <= a.NL) & all_full;
    f32x4_t s[2] = {{}, {}};
#pragma unroll
    for (int n = 0; n < 2 * KS; ++n)
        s[n & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds16(kw + (n & 1) * 16 * D + ln.kq[n >> 1]), qf[n >> 1],
                                                           s[n & 1], 0, 0, 0);
    if (!full) {
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            const int key = k0 + 16 * (v >> 2) + 4 * q + (v & 3);
            const int blk = min(key, a.NL - 1) / a.L;
            const bool vis = (key < a.NL) & (((a.anc >> blk) & 1ull) != 0ull);
            s[v >> 2][v & 3] = vis ? s[v >> 2][v & 3] : kNegInf;
        }
    }
    float mx = kNegInf;
#pragma unroll
    for (int v = 0; v < 8; ++v) mx = __builtin_elementwise_maximum(mx, s[v >> 2][v & 3]);
    fold_max16<D>(quad_max(mx), c, thr, st, o);
    bf16x8_t pf;
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < 8; ++v) {
        const float p = fast_exp2(__builtin_fmaf(s[v >> 2][v & 3], c, st.neg_mc));
        sum += p;
        pf[v] = (__bf16)p;
    }
    st.lsum += sum;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v_frag16<D>(vw, ln, db), pf, o[db], 0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 2) void verify_attn16_kernel(AttnParams P) {
    using G = AttnGeom<D, 16>;
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[G::kStageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[G::kStageElems];
    __shared__ uint64_t anc[64];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4;  // lane group: keys 4 q .. 4 q + 3 of each 16-key block

    const int lid = xcd_logical_id(blockIdx.x, P.num_wg);
    const int wg_in_group = lid % P.wg_per_group;
    const int bg = lid / P.wg_per_group;
    const int g = bg % P.Hkv;
    const int b = bg / P.Hkv;
    const int N = P.N, L = P.L, S = P.S;
    const float c = P.scale_log2;
    const float thr = kLazyLog2 / c;

    const int pj = (P.parent != nullptr && wave == 0 && lane < N) ? P.parent[(int64_t)b * N + lane] : -1;
    const uint64_t peer_bits = (P.peers != nullptr && wave == 0 && lane < N) ? P.peers[(int64_t)b * N + lane] : 0ull;

    // This lane's query row (lanes l, l^16, l^32, l^48 share a row).
    const int row = (wg_in_group * kAttnWaves + wave) * 16 + (lane & 15);
    const bool row_valid = row < P.rows_per_group;
    const int NL = N * L;
    auto row_offset = [&](int& nd_out) -> int64_t {
        const int hg = row / NL;
        const int rem = row - hg * NL;
        nd_out = rem / L;
        const int p = rem - nd_out * L;
        return ((((int64_t)b * N + nd_out) * L + p) * P.Hq + (g * P.group + hg)) * D;
    };
    int nd_q = 0;
    const int64_t row_off_q = row_valid ? row_offset(nd_q) : 0;
    bf16x8_t qf[D / 32];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
        if (row_valid) {
            qf[ks] = __builtin_bit_cast(bf16x8_t, ldg16(P.q + row_off_q + ks * 32 + q * 8));
        } else {
            qf[ks] = bf16x8_t{};
        }
    }

    const int kv_stride = P.Hkv * D;
    AttnLane16<D> ln;
    {
        const int r = lane & 15;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) ln.kq[ks] = r * D + (((4 * ks + q) ^ G::k_swz(r)) << 3);
        const int i = lane & 15;
        const int vr = 4 * q + (i >> 2);
#pragma unroll
        for (int db = 0; db < D / 16; ++db) {
            const int chunk = 2 * db + ((i & 3) >> 1);
            ln.vq[db] = vr * D + ((chunk ^ G::v_rot(vr)) << 3) + (i & 1) * 4;
        }
        ln.ri = lane / G::kChunks;
        ln.pc = lane % G::kChunks;
    }

    f32x4_t o[D / 16];
#pragma unroll
    for (int db = 0; db < D / 16; ++db) o[db] = f32x4_t{};
    SoftState st = {kNegInf, 0.f, kNegInf, 0.f};

    // ---------------- phase 1: cache keys ----------------
    CacheArgs ca;
    {
        const uint16_t* kc_base = P.kc + ((int64_t)b * S * P.Hkv + g) * D;
        const uint16_t* vc_base = P.vc + ((int64_t)b * S * P.Hkv + g) * D;
        const int64_t total = (int64_t)P.B * S * P.Hkv * D * 2;
        const int64_t start = ((int64_t)b * S * P.Hkv + g) * D * 2;
        const int64_t rem = total - start;
        const int nrec = rem > 0x7FFFFFFF ? 0x7FFFFFFF : (int)rem;
        ca.krs = __builtin_amdgcn_make_buffer_rsrc((void*)kc_base, (short)0, nrec, kBufferFlags);
        ca.vrs = __builtin_amdgcn_make_buffer_rsrc((void*)vc_base, (short)0, nrec, kBufferFlags);
    }
    ca.kv_stride = kv_stride;
    ca.S = S;
    ca.wave = wave;
    ca.h = q;
    ca.c = c;
    ca.thr = thr;

    const int nb = (S + 31) / 32;   // 32-key blocks
    const int nst = (nb + 1) / 2;   // 64-key steps, one stage each
    f32x4_t s[4] = {{}, {}, {}, {}};  // scores of the step's four 16-key blocks
    if (nb > 0) {
        if (64 <= S) {
            cache_rows_dma<D, false, false, 16>(ca.krs, kv_stride, 0, S, wave, ln, buf1);
        } else {
            cache_rows_dma<D, true, false, 16>(ca.krs, kv_stride, 0, S, wave, ln, buf1);
        }
        if (128 <= S) {
            stage_dma<D, false, 16>(ca.krs, ca.vrs, kv_stride, 0, S, wave, ln, buf0);
        } else {
            stage_dma<D, true, 16>(ca.krs, ca.vrs, kv_stride, 0, S, wave, ln, buf0);
        }
    }
    if (wave == 0) {
        uint64_t msk = 1ull << lane;
        int j = pj, prev = lane;
        bool live = lane < N;
        while (true) {  // every step moves prev strictly down, so at most N steps
            const bool step = live && j != -1;
            const bool bad = step && (j < -1 || j >= prev);
            if (bad) flag_device_status(1);
            const bool go = step && !bad;
            if (ballot64(go) == 0ull) break;
            if (go) {
                msk |= 1ull << j;
                prev = j;
            }
            const int nj = __shfl(pj, go ? j : 0);
            j = go ? nj : -1;
            live = go;
        }
        const uint64_t in_range = N == 64 ? ~0ull : ((1ull << N) - 1ull);
        if (lane < N) anc[lane] = P.drafts_visible ? (msk | (peer_bits & in_range)) : 0ull;
    }
    if (nb > 0) {
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        qk16x4<D>(buf1, ln, qf, s);
        if (S < 64) {
#pragma unroll
            for (int j = 0; j < 4; ++j) mask_tail16(s[j], 16 * j, S, q);
        }
    }
    __syncthreads();
    int t = 0;
    for (; 64 * t + 256 <= S; t += 2) {
        full_step16<D>(t, ca, ln, buf0, buf1, qf, s, st, o);
        full_step16<D>(t + 1, ca, ln, buf1, buf0, qf, s, st, o);
    }
    for (; t < nst; ++t) {
        uint16_t* cur = (t & 1) ? buf1 : buf0;
        uint16_t* nxt = (t & 1) ? buf0 : buf1;
        if (t + 1 < nst) {
            if (64 * t + 192 <= S) {
                stage_dma<D, false, 16>(ca.krs, ca.vrs, kv_stride, t + 1, S, wave, ln, nxt);
            } else {
                stage_dma<D, true, 16>(ca.krs, ca.vrs, kv_stride, t + 1, S, wave, ln, nxt);
            }
        }
        bf16x8_t pf[2];
        softmax16<D>(s, c, thr, st, o, pf);
        __builtin_amdgcn_sched_barrier(0);
        if (2 * t + 2 < nb) {
            qk16x4<D>(cur, ln, qf, s);
            if (64 * t + 128 > S) {
#pragma unroll
                for (int j = 0; j < 4; ++j) mask_tail16(s[j], 64 * t + 64 + 16 * j, S, q);
            }
        }
        pv16x2<D>(cur + G::kTileElems, ln, pf, o);
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
    }

    // ---------------- phase 2: draft blocks on the root path ----------------
    int nd = 0;
    if (row_valid) (void)row_offset(nd);
    const uint64_t my_anc = row_valid ? anc[nd] : 0ull;
    const DraftArgs da = draft_args<D>(P, b, g, lane, my_anc, row_valid, q);
    uint16_t* kw = (wave < 2 ? buf0 : buf1) + (wave & 1) * G::kWaveRegionElems;
    TileWalk walk{uniform64(wave_or64(my_anc)), 0, -1};
    for (int tt = walk.next(L); tt >= 0; tt = walk.next(L)) {
        wave_lds_sync();
        draft_tile_dma<D, 16>(da, tt * 32, kw, kw + 32 * D);
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        wave_lds_sync();
        draft_tile16<D>(da, tt * 32, q, kw, kw + 32 * D, ln, qf, st, o, c, thr);
    }

    // ---------------- epilogue ----------------
    const float l = quad_sum(st.lsum);
    const float inv = l > 0.f ? 1.0f / l : 0.f;
    if (row_valid) {
        int nd_o = 0;
        const int64_t row_off = row_offset(nd_o);
#pragma unroll
        for (int db = 0; db < D / 16; ++db) {
            const int d = db * 16 + 4 * q;
            u32x2_t w;
            const __bf16 e0 = (__bf16)(o[db][0] * inv);
            const __bf16 e1 = (__bf16)(o[db][1] * inv);
            const __bf16 e2 = (__bf16)(o[db][2] * inv);
            const __bf16 e3 = (__bf16)(o[db][3] * inv);
            w[0] = (uint32_t)__builtin_bit_cast(uint16_t, e0) | ((uint32_t)__builtin_bit_cast(uint16_t, e1) << 16);
            w[1] = (uint32_t)__builtin_bit_cast(uint16_t, e2) | ((uint32_t)__builtin_bit_cast(uint16_t, e3) << 16);
            *reinterpret_cast<u32x2_t*>(P.out + row_off + d) = w;
        }
    }
}

}  // namespace trajspec
