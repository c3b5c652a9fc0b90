// Confidence / top-k pass over vocabulary logits (Sec. 3.2, Eq. 2 and candidate
// collection): per row, m = max, s = sum exp(l - m), the k largest entries (lower index
// first on equal values) and conf_j = exp(l_j - m) / s.
//
// HBM-bound streaming design for gfx950:
//   * one workgroup streams one row (or one slice of a row when there are very few rows) with
//     16-byte non-temporal loads held in a register ring: DEPTH sweeps of U vectors per lane,
//     DEPTH - 1 of them in flight while one is absorbed.  The loop runs whole groups of DEPTH
//     sweeps with unconditional loads (vector indices past the row are clamped to its last
//     vector and discarded), so the compiler's load waits count exactly the older loads; the
//     row's last, partial sweep goes through the same ring, in flight behind the last full one;
//   * the workgroup size follows the row count: one wave per row for large batches (many
//     resident workgroups per CU), 4 or 8 waves per row for short batches;
//   * per lane a lazily moved reference value r (an element of the lane, raised only when a
//     vector maximum exceeds it by 2^8 in the exp2 domain: a wave-uniform branch that is rare
//     after the first vectors) with the running sum of exp2((x - r) log2e); a vector costs its
//     unpack, a 3-input maximum tree, one FMA + one exp2 + one add per value and two compares;
//   * the top-k candidates live in a per-lane sorted list of 64-bit keys (order-preserving value
//     bits, ~index) whose merges are unsigned max/min; a vector takes the insertion path only
//     when its maximum reaches max(wave floor, the lane's k-th key), kept as one float.  The wave
//     floor is a lower bound on the row's k-th largest value (the k-th largest lane maximum),
//     first taken from sweep 0 before anything is absorbed, then after sweeps 1, 3, 7, ...;
//   * lanes merge (reference, sum) and take the wave's keys by k rounds of a wave-wide maximum,
//     both over the DPP / permlane exchange network (no LDS round trips), waves through LDS; row
//     slices write (reference, sum, top-K) partial records that a second one-wave-per-row kernel
//     merges with the same associative rule.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace trajspec {

constexpr int kTopkRecord = 2 + 2 * 8;  // floats per partial record: reference, sum, 8 64-bit keys
// The lazy reference moves when a value exceeds it by this much in the exp2 domain, so every
// term of a lane's sum stays below 2^kTopkLazyLog2 relative to its reference.
constexpr float kTopkLazyLog2 = 8.0f;

// A candidate is packed into one 64-bit key whose unsigned order is the selection order:
// high word = order-preserving image of the fp32 value (-0 folded onto +0), low word =
// ~index, so equal values rank the lower vocabulary index first.  Key 0 is "empty".
__device__ __forceinline__ uint32_t order_bits(float x) {
    const uint32_t u = __builtin_bit_cast(uint32_t, x + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float value_of_bits(uint32_t o) {
    const uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __builtin_bit_cast(float, u);
}
__device__ __forceinline__ uint64_t make_key(float x, int id) {
    return ((uint64_t)order_bits(x) << 32) | (uint32_t)(~(uint32_t)id);
}
__device__ __forceinline__ float key_value(uint64_t k) { return value_of_bits((uint32_t)(k >> 32)); }
__device__ __forceinline__ int key_index(uint64_t k) { return (int)(~(uint32_t)k); }
__device__ __forceinline__ uint64_t kmax(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t kmin(uint64_t a, uint64_t b) { return a > b ? b : a; }

// Float threshold equivalent to "order_bits(x) >= b" for non-NaN x: every image at or below
// that of -inf (0x007fffff; in practice the empty key 0) accepts all values.
__device__ __forceinline__ float threshold_of_bits(uint32_t b) {
    return b <= 0x007fffffu ? kNegInf : value_of_bits(b);
}

template <int K>
struct TopList {
    static_assert(K == 1 || K == 2 || K == 4 || K == 8, "K must be a power of two <= 8");
    uint64_t key[K];  // descending

    __device__ __forceinline__ void clear() {
#pragma unroll
        for (int j = 0; j < K; ++j) key[j] = 0;
    }
    // Sorted insertion by a max/min bubble; the displaced tail entry drops out.
    __device__ __forceinline__ void insert(uint64_t x) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const uint64_t hi = kmax(x, key[j]);
            x = kmin(x, key[j]);
            key[j] = hi;
        }
    }
    // Keeps the K best of this list and another sorted list: the elementwise max of
    // key[j] and o[K-1-j] holds exactly the K best and is bitonic; half-cleaners sort it.
    __device__ __forceinline__ void merge(const uint64_t (&o)[K]) {
#pragma unroll
        for (int j = 0; j < K; ++j) key[j] = kmax(key[j], o[K - 1 - j]);
#pragma unroll
        for (int st = K / 2; st >= 1; st /= 2) {
#pragma unroll
            for (int j = 0; j < K; ++j) {
                if ((j & st) == 0) {
                    const uint64_t hi = kmax(key[j], key[j + st]);
                    const uint64_t lo = kmin(key[j], key[j + st]);
                    key[j] = hi;
                    key[j + st] = lo;
                }
            }
        }
    }
};

__device__ __forceinline__ void lane_pair64(int step, uint64_t v, uint64_t& a, uint64_t& b) {
    uint32_t ah, bh, al, bl;
    lane_pair(step, (uint32_t)(v >> 32), ah, bh);
    lane_pair(step, (uint32_t)v, al, bl);
    a = ((uint64_t)ah << 32) | al;
    b = ((uint64_t)bh << 32) | bl;
}
// Unsigned maxima over the wave, in every lane.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        uint32_t a, b;
        lane_pair(t, v, a, b);
        v = a > b ? a : b;
    }
    return v;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int t = 0; t < 6; ++t) {
        uint64_t a, b;
        lane_pair64(t, v, a, b);
        v = kmax(a, b);
    }
    return v;
}

// Merge two (reference, sum) pairs, each sum relative to its own reference; the result is
// relative to the larger reference.
__device__ __forceinline__ void merge_ms(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    const float Ms = fmaxf(M, -1e30f);
    s = s * fast_exp2((m - Ms) * kLog2e) + s2 * fast_exp2((m2 - Ms) * kLog2e);
    m = M;
}

// (reference, sum) pairs combined over exchange steps 0 .. STEPS-1 (6: the wave, 4: each row of
// 16 lanes).  Lanes may round differently (the combination order differs); lane 0 holds a result.
template <int STEPS>
__device__ __forceinline__ void lanes_merge_ms(float& m, float& s) {
#pragma unroll
    for (int t = 0; t < STEPS; ++t) {
        uint32_t am, bm, as, bs;
        lane_pair(t, __builtin_bit_cast(uint32_t, m), am, bm);
        lane_pair(t, __builtin_bit_cast(uint32_t, s), as, bs);
        m = __builtin_bit_cast(float, am);
        s = __builtin_bit_cast(float, as);
        merge_ms(m, s, __builtin_bit_cast(float, bm), __builtin_bit_cast(float, bs));
    }
}

// Lower bound on the k-th largest value of a row from the lanes' maxima: the k-th largest lane
// maximum (all copies of each round's maximum are dropped, which can only lower the bound).
// Returned in order_bits form; 0 when fewer than k lanes hold a value.  (K >= k bounds the
// rounds at compile time: no inner loop, which keeps the compiler's load-wait placement exact in
// the streaming loop around it.)
template <int K>
__device__ __forceinline__ uint32_t wave_kth_floor(float lane_max, int k) {
    uint32_t cur = lane_max == kNegInf ? 0u : order_bits(lane_max);
    uint32_t best = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
        if (r < k) {
            best = wave_max_u32(cur);
            if (cur == best) cur = 0u;
        }
    }
    return best;
}

// The k <= K best keys of a wave (descending, in every lane; the others 0) from the lanes' sorted
// lists, by k rounds of a wave-wide maximum over the list heads; the lane holding the winner
// drops it (keys are unique: the index is part of the key).
template <int K>
__device__ __forceinline__ void wave_top_keys(TopList<K>& tl, uint64_t (&best)[K], int k) {
#pragma unroll
    for (int r = 0; r < K; ++r) {
        best[r] = 0ull;
        if (r >= k) continue;  // wave-uniform
        const uint64_t head = tl.key[0];
        const uint64_t mk = wave_max_u64(head);
        best[r] = mk;
        if (r + 1 < K && head == mk && mk != 0ull) {
#pragma unroll
            for (int j = 0; j + 1 < K; ++j) tl.key[j] = tl.key[j + 1];
            tl.key[K - 1] = 0ull;
        }
    }
}

// Running state of one lane.
template <int K>
struct TopkLane {
    float ref;   // reference: an element value of this lane (-inf before the first finite one)
    float nrl;   // -ref * log2(e) (0 before the first reference)
    float rthr;  // ref + kTopkLazyLog2 / log2(e): a larger vector maximum moves the reference
    float s;     // sum of exp2(x log2e + nrl) over the lane's values
    float lmax;  // largest value of the lane so far (for the wave floor)
    float ins;   // insertion threshold: max(wave floor, the lane's K-th key) as a float
    TopList<K> tl;

    __device__ __forceinline__ void init() {
        ref = kNegInf;
        nrl = 0.f;
        rthr = kNegInf;
        s = 0.f;
        lmax = kNegInf;
        ins = kNegInf;
        tl.clear();
    }
    __device__ __forceinline__ void refresh(uint32_t floor_bits) {
        const uint32_t own = (uint32_t)(tl.key[K - 1] >> 32);
        ins = threshold_of_bits(floor_bits > own ? floor_bits : own);
    }
};

template <int NV>
__device__ __forceinline__ float vec_max(const float (&x)[NV]) {
    float m = x[0];
    int j = 1;
#pragma unroll
    for (; j + 1 < NV; j += 2) m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, x[j]), x[j + 1]);
#pragma unroll
    for (; j < NV; ++j) m = __builtin_elementwise_maximum(m, x[j]);
    return m;
}

// Absorbs NV values x (vocabulary indices id0 ..) whose maximum is vmax.  Values are never NaN
// (an ABI precondition), so the NaN-propagating maxima above are exact.
template <int K, int NV>
__device__ __forceinline__ void absorb(const float (&x)[NV], float vmax, int id0, TopkLane<K>& st, uint32_t floor_bits) {
    const bool up = vmax > st.rthr;
    if (ballot64(up) != 0ull) {  // wave-uniform branch, rare after the first vectors
        const float nr = -vmax * kLog2e;
        const float f = fast_exp2(__builtin_fmaf(st.ref, kLog2e, nr));  // 0 while ref is -inf
        st.s = up ? st.s * f : st.s;
        st.ref = up ? vmax : st.ref;
        st.nrl = up ? nr : st.nrl;
        st.rthr = up ? vmax + kTopkLazyLog2 / kLog2e : st.rthr;
    }
    st.lmax = __builtin_elementwise_maximum(st.lmax, vmax);
    float acc = fast_exp2(__builtin_fmaf(x[0], kLog2e, st.nrl));
#pragma unroll
    for (int j = 1; j < NV; ++j) acc += fast_exp2(__builtin_fmaf(x[j], kLog2e, st.nrl));
    st.s += acc;
    if (vmax >= st.ins) {  // rare once the floor is set
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            // A value below the threshold is below the row's k-th largest (the wave floor) or below
            // the lane's own K-th key: it can change neither the result nor the list, so it skips
            // the key and the insertion network (a branch per value, taken by few lanes).
            if (x[j] >= st.ins) {
                const uint64_t key = make_key(x[j], id0 + j);
                if (key > st.tl.key[K - 1]) st.tl.insert(key);
            }
        }
        st.refresh(floor_bits);
    }
}

// Elements of type T per 16-byte vector.
template <typename T> struct VecOf;
template <> struct VecOf<uint16_t> { static constexpr int n = 8; };
template <> struct VecOf<float> { static constexpr int n = 4; };

__device__ __forceinline__ void unpack(const u32x4_t& w, float (&x)[8]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        x[2 * j] = bf16_lo(w[j]);
        x[2 * j + 1] = bf16_hi(w[j]);
    }
}
__device__ __forceinline__ void unpack(const u32x4_t& w, float (&x)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t u = w[j];  // copy out first: bit_cast of a vector element reads element 0
        x[j] = __builtin_bit_cast(float, u);
    }
}

__device__ __forceinline__ float load_scalar(const uint16_t* p) { return bf16_bits_to_float(*p); }
__device__ __forceinline__ float load_scalar(const float* p) { return *p; }

// grid.x = rows * splits; workgroup (row, split) covers [split * chunk, min(V, (split + 1) * chunk)).
// VECTOR selects 16-byte loads (row base and chunk are then 16-byte aligned); without it every
// value is a scalar load (rows of any alignment).
template <typename T, int K, int THREADS, int U, int DEPTH, bool VECTOR>
__global__ __launch_bounds__(THREADS) void conf_topk_kernel(const T* __restrict__ logits, int64_t row_stride, int V,
                                                            int k, int splits, int chunk, float* __restrict__ conf,
                                                            int32_t* __restrict__ idx, float* __restrict__ partial) {
    constexpr int NV = VecOf<T>::n;
    constexpr int SW = THREADS * U;  // vectors per sweep of the workgroup
    const int row = blockIdx.x / splits;
    const int split = blockIdx.x - row * splits;
    const int begin = split * chunk;
    const int end = min(V, begin + chunk);
    const T* base = logits + (int64_t)row * row_stride;
    const int tid = threadIdx.x;

    TopkLane<K> st;
    st.init();
    uint32_t floor_bits = 0;
    int scalar_from = begin;
    // The waves of a workgroup share their floors through LDS: each floor is a lower bound on the
    // row's k-th largest value, so the largest of them is one too and gates every wave's
    // insertions.  A value read before another wave updates its word is merely a weaker bound,
    // so no barrier orders the accesses (only the initial zeros).
    constexpr int NWR = THREADS / 64;
    __shared__ uint32_t sh_floor[NWR];
    if (NWR > 1) {
        if ((tid & 63) == 0) sh_floor[tid >> 6] = 0u;
        __syncthreads();
    }
    auto share_floor = [&](uint32_t fb) {  // publish fb, return the largest floor of the workgroup
        if (NWR > 1) {
            if ((tid & 63) == 0)
                __hip_atomic_store(&sh_floor[tid >> 6], fb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
            for (int w = 0; w < NWR; ++w) {
                const uint32_t o = __hip_atomic_load(&sh_floor[w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                fb = o > fb ? o : fb;
            }
        }
        return fb;
    };
    if (VECTOR) {
        const int nvec = (end - begin) / NV;
        const int nfull = nvec / SW;
        const bool tail = nvec > nfull * SW;  // a last, partial sweep (fewer than SW vectors)
        const int nsw = nfull + (tail ? 1 : 0);
        const u32x4_t* vp = reinterpret_cast<const u32x4_t*>(base + begin);
        // Vector indices past the row are clamped to its last vector: such loads (the partial
        // sweep's missing vectors, the ring's loads beyond the last sweep) hit one cache line
        // and are never absorbed.
        auto load = [&](int sweep, u32x4_t (&b)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int v = sweep * SW + u * THREADS + tid;
                b[u] = __builtin_nontemporal_load(vp + (v < nvec ? v : nvec - 1));
            }
        };
        // PARTIAL: only the row's last sweep, whose vectors past the row are skipped.
        auto absorb_sweep = [&](int sweep, const u32x4_t (&b)[U], auto partial_tag) {
            constexpr bool PARTIAL = decltype(partial_tag)::value;
            float x[U][NV];
            float vm[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                unpack(b[u], x[u]);
                vm[u] = vec_max<NV>(x[u]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int v = sweep * SW + u * THREADS + tid;
                if (!PARTIAL || v < nvec) absorb<K, NV>(x[u], vm[u], begin + v * NV, st, floor_bits);
            }
            // after sweeps 1, 3, 7, ... (after sweep 0 the lane maxima are those the first floor
            // was taken from)
            if (sweep != 0 && (sweep & (sweep + 1)) == 0) {
                const uint32_t own = wave_kth_floor<K>(st.lmax, k);
                floor_bits = share_floor(own > floor_bits ? own : floor_bits);
                st.refresh(floor_bits);
            } else if (NWR > 1) {  // pick up the other waves' floors every sweep
                const uint32_t f = share_floor(floor_bits);
                if (f != floor_bits) {  // wave-uniform
                    floor_bits = f;
                    st.refresh(floor_bits);
                }
            }
        };
        using Full = std::integral_constant<bool, false>;
        using Partial = std::integral_constant<bool, true>;
        if (nsw > 0) {
            u32x4_t buf[DEPTH][U];
#pragma unroll
            for (int d = 0; d + 1 < DEPTH; ++d) load(d, buf[d]);
            {  // a first floor from sweep 0's lane maxima, so that sweep 0 already inserts rarely
                float lm = kNegInf;
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    float x0[NV];
                    unpack(buf[0][u], x0);
                    const bool in_row = u * THREADS + tid < nvec;  // false only in a partial sweep 0
                    lm = __builtin_elementwise_maximum(lm, in_row ? vec_max<NV>(x0) : kNegInf);
                }
                floor_bits = share_floor(wave_kth_floor<K>(lm, k));
                st.refresh(floor_bits);
            }
            int it = 0;
            for (; it + DEPTH <= nfull; it += DEPTH) {
#pragma unroll
                for (int j = 0; j < DEPTH; ++j) {
                    load(it + j + DEPTH - 1, buf[(j + DEPTH - 1) % DEPTH]);
                    __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the absorb
                    absorb_sweep(it + j, buf[j], Full{});
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // The remaining nfull - it < DEPTH full sweeps and the partial one: one more group of
            // the same shape (its loads unconditional, so the load waits stay exact), the partial
            // sweep in flight behind the last full one.
#pragma unroll
            for (int j = 0; j < DEPTH; ++j) {
                load(it + j + DEPTH - 1, buf[(j + DEPTH - 1) % DEPTH]);
                __builtin_amdgcn_sched_barrier(0);
                if (it + j < nfull) {
                    absorb_sweep(it + j, buf[j], Full{});
                } else if (it + j < nsw) {
                    absorb_sweep(it + j, buf[j], Partial{});
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        scalar_from = begin + nvec * NV;
    }
    for (int e = scalar_from + tid; e < end; e += THREADS) {
        const float x[1] = {load_scalar(base + e)};
        absorb<K, 1>(x, x[0], e, st, floor_bits);
    }

    // lanes -> wave: (reference, sum) over the exchange network, the keys by k rounds of a wave
    // maximum
    float m = st.ref, s = st.s;
    lanes_merge_ms<6>(m, s);
    uint64_t best[K];
    wave_top_keys<K>(st.tl, best, k);
    // waves -> workgroup
    constexpr int NW = THREADS / 64;
    TopList<K> tl;
#pragma unroll
    for (int j = 0; j < K; ++j) tl.key[j] = best[j];
    const int lane = tid & 63;
    if (NW > 1) {
        __shared__ float sh_m[NW], sh_s[NW];
        __shared__ uint64_t sh_k[NW][K];
        const int wave = tid >> 6;
        if (lane == 0) {
            sh_m[wave] = m;
            sh_s[wave] = s;
#pragma unroll
            for (int j = 0; j < K; ++j) sh_k[wave][j] = best[j];
        }
        __syncthreads();
        if (wave != 0) return;
        if (lane < NW) {
            m = sh_m[lane];
            s = sh_s[lane];
#pragma unroll
            for (int j = 0; j < K; ++j) tl.key[j] = sh_k[lane][j];
        } else {
            m = kNegInf;
            s = 0.f;
            tl.clear();
        }
        // lanes 0 .. NW-1 hold the waves' results, lanes NW .. 15 neutral ones: a reduction over
        // the quad steps (NW <= 4) or the row of 16 leaves the workgroup's in lane 0
        constexpr int STEPS = NW <= 2 ? 1 : NW <= 4 ? 2 : 4;
        static_assert(NW <= 16, "the row reduction covers at most 16 waves");
        lanes_merge_ms<STEPS>(m, s);
#pragma unroll
        for (int t = 0; t < STEPS; ++t) {
            uint64_t b[K];
#pragma unroll
            for (int j = 0; j < K; ++j) lane_pair64(t, tl.key[j], tl.key[j], b[j]);
            tl.merge(b);
        }
    }
    if (lane != 0) return;
    if (partial != nullptr) {
        float* rec = partial + ((int64_t)row * splits + split) * kTopkRecord;
        rec[0] = m;
        rec[1] = s;
        uint64_t* rk = reinterpret_cast<uint64_t*>(rec + 2);
#pragma unroll
        for (int j = 0; j < 8; ++j) rk[j] = j < K ? tl.key[j] : 0ull;
        return;
    }
    const float inv = 1.0f / s;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        if (j < k) {
            conf[(int64_t)row * k + j] = fast_exp2((key_value(tl.key[j]) - m) * kLog2e) * inv;
            idx[(int64_t)row * k + j] = key_index(tl.key[j]);
        }
    }
}

// One wave per row merges `splits` partial records.
template <int K>
__global__ __launch_bounds__(64) void conf_topk_merge_kernel(const float* __restrict__ partial, int rows,
                                                             int splits, int k, float* __restrict__ conf,
                                                             int32_t* __restrict__ idx) {
    const int row = blockIdx.x;
    if (row >= rows) return;  // the grid is exactly `rows`; kept for any other launch shape
    const int lane = threadIdx.x;
    float m = kNegInf, s = 0.f;
    TopList<K> tl;
    tl.clear();
    for (int sp = lane; sp < splits; sp += 64) {
        const float* rec = partial + ((int64_t)row * splits + sp) * kTopkRecord;
        merge_ms(m, s, rec[0], rec[1]);
        const uint64_t* rk = reinterpret_cast<const uint64_t*>(rec + 2);
        uint64_t o[K];
#pragma unroll
        for (int j = 0; j < K; ++j) o[j] = rk[j];
        tl.merge(o);
    }
    lanes_merge_ms<6>(m, s);
    uint64_t best[K];
    wave_top_keys<K>(tl, best, k);
    if (lane != 0) return;
    const float inv = 1.0f / s;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        if (j < k) {
            conf[(int64_t)row * k + j] = fast_exp2((key_value(best[j]) - m) * kLog2e) * inv;
            idx[(int64_t)row * k + j] = key_index(best[j]);
        }
    }
}

// Launch shape of the pass.  threads: lanes per row slice; unroll / depth: the register ring
// (vectors per sweep, sweeps held); splits / chunk: slices per row and their length.
struct TopkPlan {
    int threads, unroll, depth;
    int splits, chunk;
};

// Measured on the 8B shapes (vocab 126464-152064, bf16; every shape checked against the library's
// output): with many rows one wave per row and a 3-sweep ring of 2 vectors streams fastest
// (32768 rows: 6.8 TB/s); 1024 rows run best with 4 waves per row and 2-vector sweeps (4 waves
// per SIMD), 256 rows with 8 waves per row and 4-vector sweeps (2 waves per SIMD).  Fewer rows
// than 128 run 8 waves per row and also split each row, so that the launch keeps about 128
// workgroups.
inline TopkPlan plan_conf_topk(int64_t rows, int64_t vocab, int vec) {
    TopkPlan p{64, 2, 3, 1, (int)vocab};
    if (rows >= 4096) return p;
    if (rows >= 512) return TopkPlan{256, 2, 2, 1, (int)vocab};
    if (rows >= 128) return TopkPlan{512, 4, 2, 1, (int)vocab};
    p = TopkPlan{512, 2, 2, 1, (int)vocab};
    const int64_t target = 128;
    if (rows <= 0 || rows >= target) return p;
    const int64_t align = (int64_t)p.threads * vec;  // one vector per lane
    const int64_t want = (target + rows - 1) / rows;
    const int64_t max_by_len = (vocab + 4 * align - 1) / (4 * align);  // >= 4 vectors per lane and slice
    int64_t splits = want < max_by_len ? want : max_by_len;
    if (splits > 64) splits = 64;
    if (splits <= 1) return p;
    int64_t chunk = (vocab + splits - 1) / splits;
    chunk = (chunk + align - 1) / align * align;
    p.splits = (int)((vocab + chunk - 1) / chunk);
    p.chunk = (int)chunk;
    return p;
}

}  // namespace trajspec
