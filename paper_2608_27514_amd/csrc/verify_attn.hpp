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
//   online softmax is a per-lane reduction plus one exchange with lane^32, and the output
//   O^T = V^T P^T rescales with a per-lane scalar.  Q stays in registers as the B operand.
//   V^T fragments come straight from a row-major V tile with ds_read_b64_tr_b16.
//
// Phases per workgroup
//   1. cache: tiles of 64 cache keys, double-buffered in LDS with a register prefetch of
//      the next tile; one barrier per tile.
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
constexpr int kAttnThreads = kAttnWaves * 64;
constexpr int kAttnTile = 64;  // cache keys per LDS tile

typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

template <int D>
struct AttnGeom {
    static constexpr int kChunks = D / 8;                   // 16-byte chunks per key row
    static constexpr int kKs = D / 16;                      // MFMA k-steps of Q K^T
    static constexpr int kDb = D / 32;                      // 32-wide output blocks
    static constexpr int kTileElems = kAttnTile * D;        // one K or V tile
    static constexpr int kLdsElems = 2 * 2 * kTileElems;    // 2 stages x (K, V)
    static constexpr int kFillRowsPerPass = kAttnThreads / kChunks;
    static constexpr int kFillPasses = kAttnTile / kFillRowsPerPass;
    static constexpr int kWaveRowsPerPass = 64 / kChunks;   // per-wave fill of 32 draft keys
    static constexpr int kWavePasses = 32 / kWaveRowsPerPass;
    // K rows: 16-byte chunk c of row r lives at c ^ (r mod kChunks) -> the 32 rows read by
    // one Q K^T fragment load spread over all banks.
    static __device__ __forceinline__ int k_off(int r, int c) { return r * D + ((c ^ (r & (kChunks - 1))) << 3); }
    // V rows: chunk pairs are rotated by (r mod kChunks/2) so the 4 rows x 32 bytes that one
    // 16-lane group of a transposing read touches sit in distinct banks.
    static __device__ __forceinline__ int v_off(int r, int c) {
        return r * D + ((c ^ ((r & (kChunks / 2 - 1)) << 1)) << 3);
    }
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

// Online-softmax update of one 32-key block already scaled to the log2 domain; lane holds
// 16 scores of its query column.  Returns nothing; updates m, lsum, o and writes P (bf16)
// into pf (8 values per 16-key half).
template <int D>
__device__ __forceinline__ void softmax_block(f32x16_t& s, float& m, float& lsum, f32x16_t (&o)[D / 32],
                                              bf16x8_t (&pf)[2]) {
    float mx = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const float p = fast_exp2(s[v] - m_use);
        sum += p;
        pf[v >> 3][v & 7] = (__bf16)p;
    }
    lsum = lsum * alpha + sum;
    m = m_new;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] *= alpha;
}

// O^T += V^T P^T for one 32-key block staged at vbase (rows 0..31 of a V region).
template <int D>
__device__ __forceinline__ void pv_block(const uint16_t* vbase, int row0, const bf16x8_t (&pf)[2],
                                         f32x16_t (&o)[D / 32], int lane) {
    using G = AttnGeom<D>;
    const int i = lane & 15;
    const int h = lane >> 5;
    const int dsub = (lane >> 4) & 1;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            const int d = db * 32 + dsub * 16 + (i & 3) * 4;
            const int r0 = row0 + half * 16 + 4 * h + (i >> 2);
            const int r1 = r0 + 8;
            const bf16x4_t a0 = lds_read_tr(vbase + G::v_off(r0, d >> 3) + (d & 7));
            const bf16x4_t a1 = lds_read_tr(vbase + G::v_off(r1, d >> 3) + (d & 7));
            const bf16x8_t a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[half], o[db], 0, 0, 0);
        }
    }
}

// S^T for one 32-key block staged at kbase rows row0..row0+31.
template <int D>
__device__ __forceinline__ f32x16_t qk_block(const uint16_t* kbase, int row0, const bf16x8_t (&qf)[D / 16],
                                             int lane) {
    using G = AttnGeom<D>;
    f32x16_t s = {};
    const int r = row0 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8_t a = lds16(kbase + G::k_off(r, 2 * ks + (lane >> 5)));
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s, 0, 0, 0);
    }
    return s;
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

    f32x16_t o[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] = f32x16_t{};
    float m = kNegInf, lsum = 0.f;

    // ---------------- phase 1: cache keys ----------------
    const int64_t kv_stride = (int64_t)P.Hkv * D;  // elements between consecutive keys
    const uint16_t* kc_base = P.kc + ((int64_t)b * S * P.Hkv + g) * D;
    const uint16_t* vc_base = P.vc + ((int64_t)b * S * P.Hkv + g) * D;
    const int fc = tid % G::kChunks;
    const int fr0 = tid / G::kChunks;
    u32x4_t pk[G::kFillPasses], pv[G::kFillPasses];
    auto gload = [&](int tile) {
#pragma unroll
        for (int j = 0; j < G::kFillPasses; ++j) {
            const int key = tile * kAttnTile + fr0 + j * G::kFillRowsPerPass;
            if (key < S) {
                pk[j] = ldg16(kc_base + key * kv_stride + fc * 8);
                pv[j] = ldg16(vc_base + key * kv_stride + fc * 8);
            } else {
                pk[j] = u32x4_t{0, 0, 0, 0};
                pv[j] = u32x4_t{0, 0, 0, 0};
            }
        }
    };
    auto lstore = [&](int stage) {
        uint16_t* ks_ = lds + stage * 2 * G::kTileElems;
        uint16_t* vs_ = ks_ + G::kTileElems;
#pragma unroll
        for (int j = 0; j < G::kFillPasses; ++j) {
            const int r = fr0 + j * G::kFillRowsPerPass;
            sts16(ks_ + G::k_off(r, fc), pk[j]);
            sts16(vs_ + G::v_off(r, fc), pv[j]);
        }
    };

    const int ntiles = (S + kAttnTile - 1) / kAttnTile;
    if (ntiles > 0) {
        gload(0);
        lstore(0);
    }
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
        const int stage = t & 1;
        if (t + 1 < ntiles) gload(t + 1);
        const uint16_t* ks_ = lds + stage * 2 * G::kTileElems;
        const uint16_t* vs_ = ks_ + G::kTileElems;
        const bool ragged = (t + 1) * kAttnTile > S;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            f32x16_t s = qk_block<D>(ks_, kb * 32, qf, lane);
#pragma unroll
            for (int v = 0; v < 16; ++v) s[v] *= P.scale_log2;
            if (ragged) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = t * kAttnTile + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                    s[v] = key < S ? s[v] : kNegInf;
                }
            }
            bf16x8_t pf[2];
            softmax_block<D>(s, m, lsum, o, pf);
            pv_block<D>(vs_, kb * 32, pf, o, lane);
        }
        if (t + 1 < ntiles) lstore(stage ^ 1);
        __syncthreads();
    }

    // ---------------- phase 2: draft blocks on the root path ----------------
    const uint64_t my_anc = row_valid ? anc[nd] : 0ull;
    const uint64_t U = wave_or64(my_anc);
    uint16_t* kw = lds + wave * (2 * 32 * D);
    uint16_t* vw = kw + 32 * D;
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

        f32x16_t s = qk_block<D>(kw, 0, qf, lane);
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] *= P.scale_log2;
        if (!full) {
            // branch-free per-element visibility (key beyond the packed drafts, or a block
            // that is not on this row's root path)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = k0 + 8 * (v >> 2) + 4 * h + (v & 3);
                const int blk = min(key, NL - 1) / L;
                const bool vis = (key < NL) & (((my_anc >> blk) & 1ull) != 0ull);
                s[v] = vis ? s[v] : kNegInf;
            }
        }
        bf16x8_t pf[2];
        softmax_block<D>(s, m, lsum, o, pf);
        pv_block<D>(vw, 0, pf, o, lane);
    }

    // ---------------- epilogue ----------------
    const float l = lsum + __shfl_xor(lsum, 32);
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
