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
// LDS layouts (contiguous rows of D elements, conflict-free for their readers)
//   K tile: the 16-byte chunk c of row r is stored at c ^ k_swz(r), so the 16 rows that
//           one fragment load reads per bank cycle hit 16 different 16-byte bank groups.
//   V tile: chunk c of row r is stored at c ^ v_rot(r) (a per-row multiple of 4), so the
//           4 rows x 64 bytes that half a wave reads with one transposing load cover all
//           64 banks once.
//   Tiles are filled with global_load_lds_dwordx4 (16 bytes per lane straight into LDS, no
//   VGPR staging): each wave-wide load fills one contiguous kilobyte, i.e. whole rows, and
//   each lane fetches the global chunk that the swizzle puts in its slot.
//
// Phases per workgroup
//   1. cache: tiles of 64 keys in two LDS buffers (separate arrays, so the compiler can see
//      that the direct loads into one never alias reads of the other); the next tile's
//      loads are issued before the current tile is computed, one barrier per tile.  The
//      loop runs full tiles in pairs with no conditional code and peels the ragged tail.
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
    static constexpr int kChunks = D / 8;                         // 16-byte chunks per row
    static constexpr int kTileElems = kAttnTile * D;              // one K or V tile
    static constexpr int kStageElems = 2 * kTileElems;            // K tile then V tile
    static constexpr int kRowsPerDma = 512 / D;                   // rows per wave-wide 1 KB load
    static constexpr int kDmaPerWave = (kAttnTile / kAttnWaves) / kRowsPerDma;
    static constexpr int kWaveRegionElems = 2 * 32 * D;           // per-wave draft tile (K, V)
    static constexpr int kDraftDma = 32 / kRowsPerDma;
    static_assert(2 * kWaveRegionElems <= kStageElems, "two draft regions per buffer");

    static __device__ __forceinline__ int k_swz(int r) { return kChunks == 16 ? (r & 15) : ((r >> 1) & 7); }
    static __device__ __forceinline__ int v_rot(int r) {
        return kChunks == 16 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
    }
};

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ bf16x4_t lds_read_tr(const uint16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p));
}

__device__ __forceinline__ u32x4_t ldg16(const uint16_t* p) { return *reinterpret_cast<const u32x4_t*>(p); }

__device__ __forceinline__ bf16x8_t lds16(const uint16_t* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

// 16 bytes per lane from global memory straight into LDS; the wave writes the contiguous
// kilobyte starting at lds_row0 (lane i -> bytes 16 i .. 16 i + 15).
__device__ __forceinline__ void dma16(const uint16_t* g, uint16_t* lds_row0) {
    __builtin_amdgcn_global_load_lds((const void*)g, (lds_void_t*)lds_row0, 16, 0, 0);
}

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

// Online-softmax update with one 32-key block of raw scores (masked keys = -inf); the lane
// holds 16 scores for its query column, lane^32 the other 16.  `m` is the query's reference
// maximum in raw score units and `c` = scale * log2(e), so a weight is exp2(c * (score - m)):
// one FMA and one exp2 per score.  The reference only moves (and O and the running sum are
// only rescaled) when a block maximum exceeds it by more than kLazyLog2 in the log2 domain:
// weights then stay below 2^kLazyLog2, which fp32 accumulators and bf16 weights hold at full
// relative precision, and most blocks skip the rescale.  The decision is per query, the
// branch wave-uniform.  pf[half] receives the bf16 weights of keys 16*half .. +15 of the
// block in MFMA B-operand order.
template <int D>
__device__ __forceinline__ void softmax_update(const f32x16_t& s, float c, float& m, float& lsum,
                                               f32x16_t (&o)[D / 32], bf16x8_t (&pf)[2]) {
    float mx = fmaxf(s[0], s[1]);
#pragma unroll
    for (int v = 2; v < 16; v += 2) mx = fmaxf(fmaxf(mx, s[v]), s[v + 1]);
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
    for (int v = 0; v < 16; ++v) {
        const float p = fast_exp2(__builtin_fmaf(s[v], c, neg_mc));
        sum += p;
        pf[v >> 3][v & 7] = (__bf16)p;
    }
    lsum += sum;
}

// S^T of one 32-key block: kbase = K region + block row offset; kq[ks] = this lane's
// fragment offset for k-step ks.
template <int D>
__device__ __forceinline__ f32x16_t qk_block(const uint16_t* kbase, const int (&kq)[D / 16],
                                             const bf16x8_t (&qf)[D / 16]) {
    f32x16_t s = {};
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8_t a = lds16(kbase + kq[ks]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s, 0, 0, 0);
    }
    return s;
}

// O^T += V^T P^T for one 32-key block: vbase = V region + block row offset; vq[db] = this
// lane's transposing-read offset for output block db.
template <int D>
__device__ __forceinline__ void pv_block(const uint16_t* vbase, const int (&vq)[D / 32], const bf16x8_t (&pf)[2],
                                         f32x16_t (&o)[D / 32]) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            const bf16x4_t a0 = lds_read_tr(vbase + vq[db] + (16 * half) * D);
            const bf16x4_t a1 = lds_read_tr(vbase + vq[db] + (16 * half + 8) * D);
            const bf16x8_t a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[half], o[db], 0, 0, 0);
        }
    }
}

// Per-lane constants of the cache phase.
template <int D>
struct AttnLane {
    int kq[D / 16];   // K fragment offsets (region-relative, elements)
    int vq[D / 32];   // V transposing-read offsets (region-relative, elements)
    int ri;           // row of this lane's chunk within a wave-wide direct load
    int pc;           // LDS chunk slot of this lane within that row
};

// Issue the direct loads of cache tile `tile` into `stage`: wave `wave` (uniform) fills
// rows [16 wave, 16 wave + 16) of the K and V tiles, kRowsPerDma rows per load.  The
// global row of each load is uniform, so addresses are a scalar base plus this lane's
// 32-bit offset.  RAGGED clamps rows >= S to row S-1 (their scores are masked; the
// clamped values stay finite).
template <int D, bool RAGGED>
__device__ __forceinline__ void cache_dma(const uint16_t* kc_base, const uint16_t* vc_base, int kv_stride,
                                          int tile, int S, int wave, const AttnLane<D>& ln, uint16_t* stage) {
    using G = AttnGeom<D>;
#pragma unroll
    for (int j = 0; j < G::kDmaPerWave; ++j) {
        const int row0 = wave * (kAttnTile / kAttnWaves) + j * G::kRowsPerDma;  // uniform
        const int r = row0 + ln.ri;                                               // tile row
        // first global row of this load (uniform) and this lane's row relative to it; in a
        // ragged tile both are clamped to the last key, so the offset is never negative
        int base_row = tile * kAttnTile + row0;
        int grow = ln.ri;
        if (RAGGED) {
            base_row = min(base_row, S - 1);
            grow = min(tile * kAttnTile + r, S - 1) - base_row;
        }
        const int64_t rowbase = (int64_t)base_row * kv_stride;  // uniform
        const unsigned ok = (unsigned)(grow * kv_stride + ((ln.pc ^ G::k_swz(r)) << 3));
        const unsigned ov = (unsigned)(grow * kv_stride + ((ln.pc ^ G::v_rot(r)) << 3));
        dma16(kc_base + rowbase + ok, stage + row0 * D);
        dma16(vc_base + rowbase + ov, stage + G::kTileElems + row0 * D);
    }
}

// One 64-key cache tile from `stage`, one 32-key block at a time.
template <int D, bool RAGGED>
__device__ __forceinline__ void cache_tile(const uint16_t* stage, const AttnLane<D>& ln,
                                           const bf16x8_t (&qf)[D / 16], float c, int key0, int S, int h,
                                           float& m, float& lsum, f32x16_t (&o)[D / 32]) {
    using G = AttnGeom<D>;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        f32x16_t s = qk_block<D>(stage + kb * 32 * D, ln.kq, qf);
        if (RAGGED) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = key0 + kb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                s[v] = key < S ? s[v] : kNegInf;
            }
        }
        bf16x8_t pf[2];
        softmax_update<D>(s, c, m, lsum, o, pf);
        pv_block<D>(stage + G::kTileElems + kb * 32 * D, ln.vq, pf, o);
    }
}

struct CacheArgs {
    const uint16_t* kc_base;
    const uint16_t* vc_base;
    int kv_stride;
    int S, wave, h;
    float c;
};

// Tile t from `cur`; with MORE, tile t+1 (ragged iff NEXT_RAGGED) is loaded into `nxt`
// meanwhile.  Ends with every load retired and a barrier.
template <int D, bool RAGGED, bool MORE, bool NEXT_RAGGED>
__device__ __forceinline__ void cache_step(int t, const CacheArgs& a, const AttnLane<D>& ln, const uint16_t* cur,
                                           uint16_t* nxt, const bf16x8_t (&qf)[D / 16], float& m, float& lsum,
                                           f32x16_t (&o)[D / 32]) {
    if (MORE) cache_dma<D, NEXT_RAGGED>(a.kc_base, a.vc_base, a.kv_stride, t + 1, a.S, a.wave, ln, nxt);
    cache_tile<D, RAGGED>(cur, ln, qf, a.c, t * kAttnTile, a.S, a.h, m, lsum, o);
    if (MORE) __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 2) void verify_attn_kernel(AttnParams P) {
    using G = AttnGeom<D>;
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[G::kStageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[G::kStageElems];
    __shared__ uint64_t anc[64];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
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
    // Retire the Q loads here, so that no use of Q inside the tile loop has to wait for the
    // next tile's loads as well.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

    const int kv_stride = P.Hkv * D;  // elements between consecutive keys
    AttnLane<D> ln;
    {
        const int r = lane & 31;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) ln.kq[ks] = r * D + (((2 * ks + h) ^ G::k_swz(r)) << 3);
        const int i = lane & 15;
        const int dsub = (lane >> 4) & 1;
        const int vr = 4 * h + (i >> 2);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            const int chunk = db * 4 + 2 * dsub + ((i & 3) >> 1);
            ln.vq[db] = vr * D + ((chunk ^ G::v_rot(vr)) << 3) + (i & 1) * 4;
        }
        ln.ri = lane / G::kChunks;
        ln.pc = lane % G::kChunks;
    }

    f32x16_t o[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] = f32x16_t{};
    float m = kNegInf, lsum = 0.f;

    // ---------------- phase 1: cache keys ----------------
    CacheArgs ca;
    ca.kc_base = P.kc + ((int64_t)b * S * P.Hkv + g) * D;
    ca.vc_base = P.vc + ((int64_t)b * S * P.Hkv + g) * D;
    ca.kv_stride = kv_stride;
    ca.S = S;
    ca.wave = wave;
    ca.h = h;
    ca.c = c;

    const int ntiles = (S + kAttnTile - 1) / kAttnTile;
    const bool ragged_last = ntiles * kAttnTile != S;
    if (ntiles > 0) {
        if (ntiles == 1 && ragged_last) {
            cache_dma<D, true>(ca.kc_base, ca.vc_base, kv_stride, 0, S, wave, ln, buf0);
        } else {
            cache_dma<D, false>(ca.kc_base, ca.vc_base, kv_stride, 0, S, wave, ln, buf0);
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    }
    __syncthreads();
    if (ntiles > 0) {
        // Tiles 0 .. ntiles-2 are full and each loads its successor.  The main loop runs them
        // in pairs (buffers 0 and 1) while both successors are full, so its body has no
        // conditional code; the 0-2 remaining full tiles follow, and only the step that loads
        // the last tile needs to know whether that tile is ragged.
        int t = 0;
        for (; t + 2 < ntiles - 1; t += 2) {
            cache_step<D, false, true, false>(t, ca, ln, buf0, buf1, qf, m, lsum, o);
            cache_step<D, false, true, false>(t + 1, ca, ln, buf1, buf0, qf, m, lsum, o);
        }
        const int rest = ntiles - 1 - t;  // 0, 1 or 2 full tiles before the last one
        if (rest == 2) {
            cache_step<D, false, true, false>(t, ca, ln, buf0, buf1, qf, m, lsum, o);
            if (ragged_last) {
                cache_step<D, false, true, true>(t + 1, ca, ln, buf1, buf0, qf, m, lsum, o);
            } else {
                cache_step<D, false, true, false>(t + 1, ca, ln, buf1, buf0, qf, m, lsum, o);
            }
            t += 2;
        } else if (rest == 1) {
            if (ragged_last) {
                cache_step<D, false, true, true>(t, ca, ln, buf0, buf1, qf, m, lsum, o);
            } else {
                cache_step<D, false, true, false>(t, ca, ln, buf0, buf1, qf, m, lsum, o);
            }
            t += 1;
        }
        const uint16_t* last = (t & 1) ? buf1 : buf0;
        if (ragged_last) {
            cache_step<D, true, false, false>(t, ca, ln, last, nullptr, qf, m, lsum, o);
        } else {
            cache_step<D, false, false, false>(t, ca, ln, last, nullptr, qf, m, lsum, o);
        }
    }

    // ---------------- phase 2: draft blocks on the root path ----------------
    const uint64_t my_anc = row_valid ? anc[nd] : 0ull;
    const uint64_t U = wave_or64(my_anc);
    uint16_t* kw = (wave < 2 ? buf0 : buf1) + (wave & 1) * G::kWaveRegionElems;
    uint16_t* vw = kw + 32 * D;
    const uint16_t* kd_base = P.kd + (int64_t)g * D;
    const uint16_t* vd_base = P.vd + (int64_t)g * D;
    const int wri = lane / G::kChunks;
    const int wpc = lane % G::kChunks;
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
        // load the 32 draft keys of this tile into the wave's own LDS region (rows past the
        // packed drafts read the last draft key; they are masked)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int j = 0; j < G::kDraftDma; ++j) {
            const int row0 = j * G::kRowsPerDma;
            const int r = row0 + wri;
            // rows past the packed drafts read the last draft key; base and lane row are both
            // clamped so the lane offset is never negative
            const int base_row = min(k0 + row0, NL - 1);
            const int grow = min(k0 + r, NL - 1) - base_row;
            const int64_t rowbase = ((int64_t)b * NL + base_row) * kv_stride;  // uniform
            const unsigned ok = (unsigned)(grow * kv_stride + ((wpc ^ G::k_swz(r)) << 3));
            const unsigned ov = (unsigned)(grow * kv_stride + ((wpc ^ G::v_rot(r)) << 3));
            dma16(kd_base + rowbase + ok, kw + row0 * D);
            dma16(vd_base + rowbase + ov, vw + row0 * D);
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        f32x16_t s = qk_block<D>(kw, ln.kq, qf);
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
        softmax_update<D>(s, c, m, lsum, o, pf);
        pv_block<D>(vw, ln.vq, pf, o);
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
