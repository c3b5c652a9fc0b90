// Confidence / top-k pass over vocabulary logits (Sec. 3.2, Eq. 2 and candidate
// collection): per row, m = max, s = sum exp(l - m), the k largest entries (lower index
// first on equal values) and conf_j = exp(l_j - m) / s.
//
// HBM-bound streaming design for gfx950:
//   * one 256-thread workgroup streams one row (or one slice of a row when there are too
//     few rows to fill 256 CUs) with 16-byte non-temporal loads: full sweeps of the
//     workgroup load unconditionally, two vectors per lane per sweep, and the next sweep's
//     loads are issued before the current sweep is absorbed (a guard per load would put each
//     load in its own branch and serialise them); only the last, partial sweep checks bounds;
//   * each lane keeps a running (max, rescaled sum) and a sorted top-K list; a vector of 8
//     bf16 costs one max-tree, one rescale test, 8 fma+exp2+add and one compare against
//     the lane's current K-th value (insertions are rare after the first few vectors);
//   * lanes merge through cross-lane shuffles, waves through LDS; row slices write
//     (max, sum, top-K) partials that a second one-wave-per-row kernel merges with the
//     same associative rule.
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kTopkThreads = 256;
constexpr int kTopkUnroll = 2;
constexpr int kTopkRecord = 2 + 2 * 8;  // floats per partial record: m, s, 8 64-bit keys

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

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t x, int off) {
    const uint32_t lo = __shfl_xor((uint32_t)x, off);
    const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), off);
    return ((uint64_t)hi << 32) | lo;
}

// Merge two (max, sum) pairs expressed in log2-domain-free form: sums are relative to
// their own max; the result is relative to the larger max.
__device__ __forceinline__ void merge_ms(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    const float Ms = fmaxf(M, -1e30f);
    s = s * fast_exp2((m - Ms) * kLog2e) + s2 * fast_exp2((m2 - Ms) * kLog2e);
    m = M;
}

template <int K>
__device__ __forceinline__ void wave_merge(float& m, float& s, TopList<K>& tl) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float m2 = __shfl_xor(m, off);
        const float s2 = __shfl_xor(s, off);
        merge_ms(m, s, m2, s2);
        uint64_t o[K];
#pragma unroll
        for (int j = 0; j < K; ++j) o[j] = shfl_xor64(tl.key[j], off);
        tl.merge(o);
    }
}

// Running update with one vector of NV values starting at vocabulary index id0.
// `floor_bits` is a lower bound (order_bits form) on the row's k-th largest value shared by
// the wave: values below it can never reach the row's top-k, so only vectors holding a
// value >= max(floor, this lane's K-th) take the insertion path.
template <int K, int NV>
__device__ __forceinline__ void absorb(const float (&x)[NV], int id0, float& m, float& s, TopList<K>& tl,
                                       uint32_t floor_bits) {
    float vmax = x[0];
#pragma unroll
    for (int j = 1; j < NV; ++j) vmax = fmaxf(vmax, x[j]);
    if (vmax > m) {
        s *= fast_exp2((m - vmax) * kLog2e);
        m = vmax;
    }
    const float mL = fmaxf(m, -1e30f) * kLog2e;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) acc += fast_exp2(__builtin_fmaf(x[j], kLog2e, -mL));
    s += acc;
    const uint32_t lane_floor = (uint32_t)(tl.key[K - 1] >> 32);
    const uint32_t thr = floor_bits > lane_floor ? floor_bits : lane_floor;
    if (order_bits(vmax) >= thr) {
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const uint64_t key = make_key(x[j], id0 + j);
            if (key > tl.key[K - 1]) tl.insert(key);
        }
    }
}

// Lower bound on the k-th largest value of a row from the lanes' running maxima: the k-th
// largest lane maximum (all copies of each round's maximum are dropped, which can only
// lower the bound).  Returned in order_bits form; 0 when fewer than k lanes hold a value.
// (K >= k bounds the rounds at compile time: no inner loop, which keeps the compiler's
// load-wait placement exact in the streaming loop around it.)
template <int K>
__device__ __forceinline__ uint32_t wave_kth_floor(float lane_max, int k) {
    uint32_t cur = lane_max == kNegInf ? 0u : order_bits(lane_max);
    uint32_t best = 0;
#pragma unroll
    for (int r = 0; r < K; ++r) {
        if (r < k) {
            best = cur;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                const uint32_t o = __shfl_xor(best, off);
                best = o > best ? o : best;
            }
            if (cur == best) cur = 0u;
        }
    }
    return best;
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

// grid.x = rows * splits; workgroup (row, split) covers [split*chunk, min(V, (split+1)*chunk)).
// VECTOR selects 16-byte loads (row base and chunk are then 16-byte aligned).
template <typename T, int K, bool VECTOR>
__global__ __launch_bounds__(kTopkThreads) void conf_topk_kernel(
    const T* __restrict__ logits, int64_t row_stride, int V, int k, int splits, int chunk,
    float* __restrict__ conf, int32_t* __restrict__ idx, float* __restrict__ partial) {
    constexpr int NV = VecOf<T>::n;
    const int row = blockIdx.x / splits;
    const int split = blockIdx.x - row * splits;
    const int begin = split * chunk;
    const int end = min(V, begin + chunk);
    const T* base = logits + (int64_t)row * row_stride;
    const int tid = threadIdx.x;

    float m = kNegInf, s = 0.f;
    TopList<K> tl;
    tl.clear();

    int scalar_from = begin;
    uint32_t floor_bits = 0;
    if (VECTOR) {
        const int nvec = (end - begin) / NV;
        const u32x4_t* vp = reinterpret_cast<const u32x4_t*>(base + begin);
        constexpr int SW = kTopkThreads * kTopkUnroll;  // vectors per sweep of the workgroup
        const int nfull = nvec / SW;
        int it = 0;
        // Full sweeps: unconditional loads, the next sweep's loads in flight while the current
        // one is absorbed (two register sets, so the loop is unrolled by two).
        auto load_sweep = [&](int sweep, u32x4_t (&buf)[kTopkUnroll]) {
#pragma unroll
            for (int u = 0; u < kTopkUnroll; ++u) buf[u] = __builtin_nontemporal_load(vp + sweep * SW + u * kTopkThreads + tid);
        };
        auto absorb_sweep = [&](int sweep, const u32x4_t (&buf)[kTopkUnroll]) {
#pragma unroll
            for (int u = 0; u < kTopkUnroll; ++u) {
                float x[NV];
                unpack(buf[u], x);
                absorb<K, NV>(x, begin + (sweep * SW + u * kTopkThreads + tid) * NV, m, s, tl, floor_bits);
            }
            // refresh the wave floor after sweeps 0, 1, 3, 7, 15, ...
            if ((sweep & (sweep + 1)) == 0) floor_bits = wave_kth_floor<K>(m, k);
        };
        if (nfull > 0) {
            u32x4_t bufa[kTopkUnroll], bufb[kTopkUnroll];
            load_sweep(0, bufa);
            for (; it + 2 <= nfull; it += 2) {
                load_sweep(it + 1, bufb);
                __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the absorb
                absorb_sweep(it, bufa);
                if (it + 2 < nfull) load_sweep(it + 2, bufa);
                __builtin_amdgcn_sched_barrier(0);
                absorb_sweep(it + 1, bufb);
            }
            if (it < nfull) {  // odd count: the last full sweep is already loaded in bufa
                absorb_sweep(it, bufa);
                ++it;
            }
        }
        // Last, partial sweep: per-vector bounds.
        for (int vb = nfull * SW; vb < nvec; vb += SW, ++it) {
            u32x4_t buf[kTopkUnroll];
#pragma unroll
            for (int u = 0; u < kTopkUnroll; ++u) {
                const int vi = vb + u * kTopkThreads + tid;
                if (vi < nvec) buf[u] = __builtin_nontemporal_load(vp + vi);
            }
#pragma unroll
            for (int u = 0; u < kTopkUnroll; ++u) {
                const int vi = vb + u * kTopkThreads + tid;
                if (vi < nvec) {
                    float x[NV];
                    unpack(buf[u], x);
                    absorb<K, NV>(x, begin + vi * NV, m, s, tl, floor_bits);
                }
            }
            if ((it & (it + 1)) == 0) floor_bits = wave_kth_floor<K>(m, k);
        }
        scalar_from = begin + nvec * NV;
    }
    for (int e = scalar_from + tid; e < end; e += kTopkThreads) {
        float x[1] = {load_scalar(base + e)};
        absorb<K, 1>(x, e, m, s, tl, floor_bits);
    }

    // lanes -> wave
    wave_merge<K>(m, s, tl);
    // waves -> workgroup
    constexpr int NW = kTopkThreads / 64;
    __shared__ float sh_m[NW], sh_s[NW];
    __shared__ uint64_t sh_k[NW][K];
    const int lane = tid & 63, wave = tid >> 6;
    if (lane == 0) {
        sh_m[wave] = m;
        sh_s[wave] = s;
#pragma unroll
        for (int j = 0; j < K; ++j) sh_k[wave][j] = tl.key[j];
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
    wave_merge<K>(m, s, tl);
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
    wave_merge<K>(m, s, tl);
    if (lane != 0) return;
    const float inv = 1.0f / s;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        if (j < k) {
            conf[(int64_t)row * k + j] = fast_exp2((key_value(tl.key[j]) - m) * kLog2e) * inv;
            idx[(int64_t)row * k + j] = key_index(tl.key[j]);
        }
    }
}

struct TopkPlan {
    int splits;
    int chunk;
};

// Splits short batches so that at least ~512 workgroups stream the rows.  More, shorter
// slices cost more than they gain: each slice pays a workgroup reduction and a partial record,
// and the merge kernel grows with them (measured on 256-1024-row batches: a 2048 target was
// 15-25% slower than 512).
inline TopkPlan plan_conf_topk(int64_t rows, int64_t vocab, int vec) {
    TopkPlan p{1, (int)vocab};
    const int64_t target = 512;
    if (rows <= 0 || rows >= target) return p;
    const int64_t align = (int64_t)kTopkThreads * vec;  // one full sweep of the workgroup
    int64_t want = (target + rows - 1) / rows;
    int64_t max_by_len = (vocab + 4 * align - 1) / (4 * align);  // >= 4 sweeps per slice
    int64_t splits = want < max_by_len ? want : max_by_len;
    if (splits > 64) splits = 64;
    if (splits <= 1) return p;
    int64_t chunk = (vocab + splits - 1) / splits;
    chunk = (chunk + align - 1) / align * align;
    splits = (vocab + chunk - 1) / chunk;
    p.splits = (int)splits;
    p.chunk = (int)chunk;
    return p;
}

}  // namespace trajspec
