// Trajectory-masked verification attention (Sec. 3.3) on gfx950 bf16 MFMA.
//
// Work decomposition
//   Queries of one (sequence b, K/V head g) are flattened as rows r = (hg, n, p): query head
//   g*G + hg, draft n, block position p.  A wave owns 32 consecutive rows; a workgroup of
//   4 waves owns 128 rows that all read the same K/V head, so every cache tile is staged in
//   LDS once and consumed by all four waves (cache K/V is shared by every draft).
//
// Math layout (v_mfma_f32_32x32x16_bf16, wave64)
//   Scores are computed transposed, S^T = K Q^T (32 keys x 32 queries per MFMA block): the
//   accumulator then holds one query per lane column, so the row max / row sum of the
//   online softmax is a per-lane reduction plus one exchange with lane^32 (a VALU lane
//   swap), and the output O^T = V^T P^T rescales with a per-lane scalar.  Q stays in
//   registers as the B operand.  V^T fragments come straight from a row-major V tile with
//   ds_read_b64_tr_b16.
//
// LDS layouts (both conflict-free for their readers and writers)
//   K tile: rows padded to D+8 elements, so the 32 rows read by one fragment load start in
//           different banks and every per-lane address is a base plus an immediate.
//   V tile: rows of D elements; the 16-byte chunk index of row r is XOR-ed with a
//           per-row multiple of 4 so the 4 rows x 64 bytes that half a wave reads with one
//           transposing load cover all 64 banks once.
//
// Phases per workgroup
//   1. cache: tiles of 64 keys, double-buffered in LDS with a register prefetch of the next
//      tile; one barrier per tile.  The loop is unrolled over the two buffers so that every
//      LDS address is a per-lane base plus an immediate, and the (at most one) ragged tail
//      tile is a separate instantiation so full tiles carry no masking code.
//   2. drafts: each wave walks the 32-key tiles of the packed draft keys and processes
//      only tiles holding its own block or an ancestor block (a 64-bit ancestor mask per
//      draft, built from the parent array).  Tiles that hold only fully visible blocks need
//      no per-element mask (always the case when L is a multiple of 32).
#pragma once

#include "common.hpp"

namespace trajspec {

struct AttnParams {
    const uint16_t* q;
    const uint16_t* kc;
    const uint16_t* vc;
    const uint16_t* kd;
    const uint16_t* vd;
    const int32_t* parent;
    uint16_t* out;
    int B, N, L, Hq, Hkv, S;
    int group;           // Hq / Hkv
    int rows_per_group;  // group * N * L
    int wg_per_group;    // workgroups per (b, g)
    int num_wg;
    float scale_log2;    // softmax scale * log2(e)
};

constexpr int kAttnWaves = 4;
// s_waitcnt immediate (gfx9 encoding) waiting for vector-memory loads only: vmcnt = 0,
// expcnt and lgkmcnt left at their maxima.
constexpr int kWaitVmcnt0 = 0x0F70;
constexpr int kAttnThreads = kAttnWaves * 64;
constexpr int kAttnTile = 64;  // cache keys per LDS tile
// Online softmax: the reference maximum of a query only moves when a new score exceeds it
// by more than this many powers of two, so weights stay below 2^kLazyLog2.
constexpr float kLazyLog2 = 8.0f;

typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

template <int D>
struct AttnGeom {
    static constexpr int kChunks = D / 8;                     // 16-byte chunks per key row
    static constexpr int kKStride = D + 8;                    // padded K row (elements)
    static constexpr int kKTile = kAttnTile * kKStride;       // one K tile (elements)
    static constexpr int kVTile = kAttnTile * D;              // one V tile (elements)
    static constexpr int kStage = kKTile + kVTile;
    static constexpr int kLdsElems = 2 * kStage;              // double buffer
    static constexpr int kWaveRegion = 32 * kKStride + 32 * D;  // per-wave draft tile
    static_assert(kAttnWaves * kWaveRegion <= kLdsElems, "draft regions must fit the tile buffers");
    static constexpr int kFillRowsPerPass = kAttnThreads / kChunks;
    static constexpr int kFillPasses = kAttnTile / kFillRowsPerPass;
    static constexpr int kWaveRowsPerPass = 64 / kChunks;     // per-wave fill of 32 draft keys
    static constexpr int kWavePasses = 32 / kWaveRowsPerPass;

    static __device__ __forceinline__ int k_off(int r, int c) { return r * kKStride + c * 8; }
    static __device__ __forceinline__ int v_rot(int r) {
        return kChunks == 16 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
    }
    static __device__ __forceinline__ int v_off(int r, int c) { return r * D + ((c ^ v_rot(r)) << 3); }
};

__device__ __forceinline__ bf16x4_t lds_read_tr(const uint16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p));
}

__device__ __forceinline__ u32x4_t ldg16(const uint16_t* p) { return *reinterpret_cast<const u32x4_t*>(p); }

__device__ __forceinline__ void sts16(uint16_t* p, const u32x4_t& v) { *reinterpret_cast<u32x4_t*>(p) = v; }

__device__ __forceinline__ bf16x8_t lds16(const uint16_t* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

__device__ __forceinline__ uint64_t wave_or64(uint64_t x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)x, off);
        const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), off);
        x |= ((uint64_t)hi << 32) | lo;
    }
    return x;
}

// x combined with the value of lane l^32 (v_permlane32_swap: pure VALU, no LDS round trip).
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                    false, false);
    const uint32_t a = r[0], b = r[1];  // copy out: bit_cast of a vector element reads element 0
    return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                    false, false);
    const uint32_t a = r[0], b = r[1];
    return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// Online-softmax update with NB 32-key blocks of raw scores (masked keys = -inf); the lane
// holds 16 scores per block for its query column, lane^32 the other 16.  `m` is the
// query's reference maximum in raw score units and `c` = scale * log2(e), so a weight is
// exp2(c * (score - m)): one FMA and one exp2 per score.  The reference only moves (and O
// and the running sum are only rescaled) when a block maximum exceeds it by more than
// kLazyLog2 in the log2 domain: weights then stay below 2^kLazyLog2, which fp32
// accumulators and bf16 weights hold at full relative precision, and most tiles skip the
// rescale.  The decision is per query, the branch wave-uniform.  pf[2*kb + half] receives
// the bf16 weights of keys 16*(2*kb + half) .. +15 in MFMA B-operand order.
template <int D, int NB>
__device__ __forceinline__ void softmax_update(const f32x16_t (&s)[NB], float c, float& m, float& lsum,
                                               f32x16_t (&o)[D / 32], bf16x8_t (&pf)[2 * NB]) {
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; v += 2) mx = fmaxf(fmaxf(mx, s[kb][v]), s[kb][v + 1]);
    }
    mx = pair_max(mx);
    const bool need = (mx - m) * c > kLazyLog2;  // false for an all-masked block (NaN or -inf)
    if (ballot64(need) != 0ull) {
        const float m_new = need ? mx : m;
        const float alpha = need ? fast_exp2((m - m_new) * c) : 1.0f;  // 0 when m was -inf
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) o[db] *= alpha;
        m = m_new;
    }
    const float neg_mc = m == kNegInf ? 0.f : -m * c;
    float sum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const float p = fast_exp2(__builtin_fmaf(s[kb][v], c, neg_mc));
            sum += p;
            pf[2 * kb + (v >> 3)][v & 7] = (__bf16)p;
        }
    }
    lsum += sum;
}

// S^T for NB 32-key blocks of a K region; kq = region base + this lane's fragment base.
template <int D, int NB>
__device__ __forceinline__ void qk_blocks(const uint16_t* kq, const bf16x8_t (&qf)[D / 16], f32x16_t (&s)[NB]) {
    using G = AttnGeom<D>;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) s[kb] = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            const bf16x8_t a = lds16(kq + kb * 32 * G::kKStride + ks * 16);
            s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[kb], 0, 0, 0);
        }
    }
}

// O^T += V^T P^T for NB 32-key blocks of a V region; vq[db] = region base + this lane's
// transposing-read base for output block db.
template <int D, int NB>
__device__ __forceinline__ void pv_blocks(const uint16_t* const (&vq)[D / 32], const bf16x8_t (&pf)[2 * NB],
                                          f32x16_t (&o)[D / 32]) {
#pragma unroll
    for (int kk = 0; kk < 2 * NB; ++kk) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            const bf16x4_t a0 = lds_read_tr(vq[db] + (16 * kk) * D);
            const bf16x4_t a1 = lds_read_tr(vq[db] + (16 * kk + 8) * D);
            const bf16x8_t a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kk], o[db], 0, 0, 0);
        }
    }
}

template <int D>
struct CacheStager {
    using G = AttnGeom<D>;
    u32x4_t pk[G::kFillPasses], pv[G::kFillPasses];
    const uint16_t* kc_base;
    const uint16_t* vc_base;
    int64_t kv_stride;
    int S, fc, fr0;

    // FULL: every key of the tile is < S (all tiles but the last), so no bounds test.
    template <bool FULL>
    __device__ __forceinline__ void gload(int tile) {
#pragma unroll
        for (int j = 0; j < G::kFillPasses; ++j) {
            const int key = tile * kAttnTile + fr0 + j * G::kFillRowsPerPass;
            if (FULL || key < S) {
                pk[j] = ldg16(kc_base + key * kv_stride + fc * 8);
                pv[j] = ldg16(vc_base + key * kv_stride + fc * 8);
            } else {
                pk[j] = u32x4_t{0, 0, 0, 0};
                pv[j] = u32x4_t{0, 0, 0, 0};
            }
        }
    }
    __device__ __forceinline__ void lstore(uint16_t* stage) {
#pragma unroll
        for (int j = 0; j < G::kFillPasses; ++j) {
            const int r = fr0 + j * G::kFillRowsPerPass;
            sts16(stage + G::k_off(r, fc), pk[j]);
            sts16(stage + G::kKTile + G::v_off(r, fc), pv[j]);
        }
    }
};

// One 64-key cache tile from LDS buffer STAGE, one 32-key block at a time.  RAGGED masks
// keys >= S.
template <int D, int STAGE, bool RAGGED>
__device__ __forceinline__ void cache_tile(const uint16_t* lds, int kq_off, const int (&vq_off)[D / 32],
                                           const bf16x8_t (&qf)[D / 16], float c, int key0, int S, int h,
                                           float& m, float& lsum, f32x16_t (&o)[D / 32]) {
    using G = AttnGeom<D>;
    const uint16_t* stage = lds + STAGE * G::kStage;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        f32x16_t s[1];
        qk_blocks<D, 1>(stage + kq_off + kb * 32 * G::kKStride, qf, s);
        if (RAGGED) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = key0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                s[0][v] = key < S ? s[0][v] : kNegInf;
            }
        }
        bf16x8_t pf[2];
        softmax_update<D, 1>(s, c, m, lsum, o, pf);
        const uint16_t* vq[D / 32];
#pragma unroll
        for (int db = 0; db < D / 32; ++db) vq[db] = stage + G::kKTile + kb * 32 * D + vq_off[db];
        pv_blocks<D, 1>(vq, pf, o);
    }
}

// Tile t of the cache loop from buffer STAGE.  With MORE, tile t+1 (full iff NEXT_FULL)
// is prefetched into registers during the compute and staged into the other buffer
// afterwards; a barrier closes the step.
template <int D, int STAGE, bool RAGGED, bool MORE, bool NEXT_FULL>
__device__ __forceinline__ void cache_step(int t, CacheStager<D>& st, uint16_t* lds, int kq_off,
                                           const int (&vq_off)[D / 32], const bf16x8_t (&qf)[D / 16], float c,
                                           int S, int h, float& m, float& lsum, f32x16_t (&o)[D / 32]) {
    using G = AttnGeom<D>;
    if (MORE) st.template gload<NEXT_FULL>(t + 1);
    cache_tile<D, STAGE, RAGGED>(lds, kq_off, vq_off, qf, c, t * kAttnTile, S, h, m, lsum, o);
    if (MORE) st.lstore(lds + (STAGE ^ 1) * G::kStage);
    __syncthreads();
}

// The last cache tile (index t, buffer STAGE): no prefetch; masked when S is not a
// multiple of the tile.
template <int D, int STAGE>
__device__ __forceinline__ void cache_last(int t, bool ragged, CacheStager<D>& st, uint16_t* lds, int kq_off,
                                           const int (&vq_off)[D / 32], const bf16x8_t (&qf)[D / 16], float c,
                                           int S, int h, float& m, float& lsum, f32x16_t (&o)[D / 32]) {
    if (ragged) {
        cache_step<D, STAGE, true, false, false>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
    } else {
        cache_step<D, STAGE, false, false, false>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
    }
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 2) void verify_attn_kernel(AttnParams P) {
    using G = AttnGeom<D>;
    __shared__ __attribute__((aligned(16))) uint16_t lds[G::kLdsElems];
    __shared__ uint64_t anc[64];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;

    const int lid = xcd_logical_id(blockIdx.x, P.num_wg);
    const int wg_in_group = lid % P.wg_per_group;
    const int bg = lid / P.wg_per_group;
    const int g = bg % P.Hkv;
    const int b = bg / P.Hkv;
    const int N = P.N, L = P.L, S = P.S;
    const float c = P.scale_log2;

    // Ancestor masks (bit j of anc[n] set when draft j is n itself or on n's root path).
    if (tid < N) {
        uint64_t msk = 1ull << tid;
        int j = P.parent[(int64_t)b * N + tid];
        int prev = tid;
        for (int hops = 0; j != -1 && hops < N; ++hops) {
            if (j < -1 || j >= prev) {  // not topological: report, stop the walk here
                flag_device_status(1);
                break;
            }
            msk |= 1ull << j;
            prev = j;
            j = P.parent[(int64_t)b * N + j];
        }
        anc[tid] = msk;
    }

    // This lane's query row (lanes l and l^32 share a row).
    const int row = (wg_in_group * kAttnWaves + wave) * 32 + (lane & 31);
    const bool row_valid = row < P.rows_per_group;
    const int NL = N * L;
    int nd = 0;
    int64_t row_off = 0;
    if (row_valid) {
        const int hg = row / NL;
        const int rem = row - hg * NL;
        nd = rem / L;
        const int p = rem - nd * L;
        row_off = ((((int64_t)b * N + nd) * L + p) * P.Hq + (g * P.group + hg)) * D;
    }
    bf16x8_t qf[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
        if (row_valid) {
            qf[ks] = __builtin_bit_cast(bf16x8_t, ldg16(P.q + row_off + ks * 16 + h * 8));
        } else {
            qf[ks] = bf16x8_t{};
        }
    }
    // Retire the Q loads here.  Otherwise the loop below starts with Q loads and the
    // previous iteration's K/V prefetch both outstanding at its header, and the first use
    // of Q waits for every outstanding load (the prefetch included) on each tile.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

    // Per-lane LDS fragment bases (region-relative).
    const int kq_off = (lane & 31) * G::kKStride + h * 8;
    int vq_off[D / 32];
    {
        const int i = lane & 15;
        const int dsub = (lane >> 4) & 1;
        const int vr = 4 * h + (i >> 2);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            const int chunk = db * 4 + 2 * dsub + ((i & 3) >> 1);
            vq_off[db] = G::v_off(vr, chunk) + (i & 1) * 4;
        }
    }

    f32x16_t o[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] = f32x16_t{};
    float m = kNegInf, lsum = 0.f;

    // ---------------- phase 1: cache keys ----------------
    const int64_t kv_stride = (int64_t)P.Hkv * D;  // elements between consecutive keys
    CacheStager<D> st;
    st.kc_base = P.kc + ((int64_t)b * S * P.Hkv + g) * D;
    st.vc_base = P.vc + ((int64_t)b * S * P.Hkv + g) * D;
    st.kv_stride = kv_stride;
    st.S = S;
    st.fc = tid % G::kChunks;
    st.fr0 = tid / G::kChunks;

    const int ntiles = (S + kAttnTile - 1) / kAttnTile;
    const bool ragged_last = ntiles * kAttnTile != S;
    if (ntiles > 0) {
        if (ntiles == 1 && ragged_last) {
            st.template gload<false>(0);
        } else {
            st.template gload<true>(0);
        }
        st.lstore(lds);
    }
    __syncthreads();
    if (ntiles > 0) {
        // Tiles 0 .. ntiles-2 are full and each prefetches its successor.  The main loop runs
        // them in pairs (buffers 0 and 1) while both prefetches target full tiles, so its
        // body has no conditional code; the 0-2 remaining full tiles follow, and only the step
        // that prefetches the last tile needs to know whether that tile is ragged.
        const bool last_full = !ragged_last;
        int t = 0;
        for (; t + 2 < ntiles - 1; t += 2) {
            cache_step<D, 0, false, true, true>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            cache_step<D, 1, false, true, true>(t + 1, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
        }
        const int rest = ntiles - 1 - t;  // 0, 1 or 2 full tiles before the last one
        if (rest == 2) {
            cache_step<D, 0, false, true, true>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            if (last_full) {
                cache_step<D, 1, false, true, true>(t + 1, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            } else {
                cache_step<D, 1, false, true, false>(t + 1, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            }
            t += 2;
        } else if (rest == 1) {
            if (last_full) {
                cache_step<D, 0, false, true, true>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            } else {
                cache_step<D, 0, false, true, false>(t, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
            }
            t += 1;
        }
        if (t & 1) {
            cache_last<D, 1>(t, ragged_last, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
        } else {
            cache_last<D, 0>(t, ragged_last, st, lds, kq_off, vq_off, qf, c, S, h, m, lsum, o);
        }
    }

    // ---------------- phase 2: draft blocks on the root path ----------------
    const uint64_t my_anc = row_valid ? anc[nd] : 0ull;
    const uint64_t U = wave_or64(my_anc);
    uint16_t* kw = lds + wave * G::kWaveRegion;
    uint16_t* vw = kw + 32 * G::kKStride;
    const uint16_t* vqw[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) vqw[db] = vw + vq_off[db];
    const uint16_t* kd_base = P.kd + (int64_t)g * D;
    const uint16_t* vd_base = P.vd + (int64_t)g * D;
    const int wc = lane % G::kChunks;
    const int wr0 = lane / G::kChunks;
    const int dtiles = (NL + 31) / 32;
    for (int tt = 0; tt < dtiles; ++tt) {
        const int k0 = tt * 32;
        const int jlo = k0 / L;
        const int jhi = min(N - 1, (k0 + 31) / L);
        const uint64_t T = (jhi - jlo == 63) ? ~0ull : (((1ull << (jhi - jlo + 1)) - 1) << jlo);
        if ((U & T) == 0) continue;  // wave-uniform
        const bool lane_full = !row_valid || ((my_anc & T) == T);
        const bool all_full = ballot64_all(lane_full);
        const bool full = (k0 + 32 <= NL) & all_full;
        // stage the 32 draft keys of this tile in the wave's own LDS region
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int j = 0; j < G::kWavePasses; ++j) {
            const int r = wr0 + j * G::kWaveRowsPerPass;
            const int key = k0 + r;
            u32x4_t kv = u32x4_t{0, 0, 0, 0}, vv = u32x4_t{0, 0, 0, 0};
            if (key < NL) {
                const int64_t tok = (int64_t)b * NL + key;  // (b, n, p) flattened
                kv = ldg16(kd_base + tok * kv_stride + wc * 8);
                vv = ldg16(vd_base + tok * kv_stride + wc * 8);
            }
            sts16(kw + G::k_off(r, wc), kv);
            sts16(vw + G::v_off(r, wc), vv);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        f32x16_t s[1];
        qk_blocks<D, 1>(kw + kq_off, qf, s);
        if (!full) {
            // branch-free per-element visibility (key beyond the packed drafts, or a block
            // that is not on this row's root path)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = k0 + 8 * (v >> 2) + 4 * h + (v & 3);
                const int blk = min(key, NL - 1) / L;
                const bool vis = (key < NL) & (((my_anc >> blk) & 1ull) != 0ull);
                s[0][v] = vis ? s[0][v] : kNegInf;
            }
        }
        bf16x8_t pf[2];
        softmax_update<D, 1>(s, c, m, lsum, o, pf);
        pv_blocks<D, 1>(vqw, pf, o);
    }

    // ---------------- epilogue ----------------
    const float l = pair_sum(lsum);
    const float inv = l > 0.f ? 1.0f / l : 0.f;
    if (row_valid) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
#pragma unroll
            for (int vg = 0; vg < 4; ++vg) {
                const int d = db * 32 + 8 * vg + 4 * h;
                u32x2_t w;
                const __bf16 e0 = (__bf16)(o[db][4 * vg + 0] * inv);
                const __bf16 e1 = (__bf16)(o[db][4 * vg + 1] * inv);
                const __bf16 e2 = (__bf16)(o[db][4 * vg + 2] * inv);
                const __bf16 e3 = (__bf16)(o[db][4 * vg + 3] * inv);
                w[0] = (uint32_t)__builtin_bit_cast(uint16_t, e0) | ((uint32_t)__builtin_bit_cast(uint16_t, e1) << 16);
                w[1] = (uint32_t)__builtin_bit_cast(uint16_t, e2) | ((uint32_t)__builtin_bit_cast(uint16_t, e3) << 16);
                *reinterpret_cast<u32x2_t*>(P.out + row_off + d) = w;
            }
        }
    }
}

}  // namespace trajspec
