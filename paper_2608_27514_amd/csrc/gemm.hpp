// Dense bf16 projection GEMM of the verification layer: D[M,N] = A[M,K] W[K,N] (+ D), all
// row-major bf16, fp32 accumulation on v_mfma_f32_32x32x16_bf16, one bf16 rounding (nearest
// even) of each result.  A holds the packed draft tokens (M = B N L rows), W a weight matrix.
//
// Two tilings, chosen by the host: gemm_tile256_kernel (256 x 256 tiles, 8 waves) for grids
// that fill the chip, gemm_ring128_kernel (128 x 128 tiles, 4 waves, a deeper stage ring)
// for the few-sequence shapes whose k loops are latency-bound.
//
// Fragments: the MFMA takes 8 k-values per lane; lane half h = lane / 32 holds k = 8h .. 8h+7
// of each 16-wide k slice, for row (A) or column (W) lane % 32.  A is k-contiguous, so an A
// fragment is one 16-byte LDS read.  W is n-contiguous: a W fragment is two transposing
// reads (ds_read_b64_tr_b16) of slice rows 8h .. 8h+3 and 8h+4 .. 8h+7; in each group of 16
// lanes, lane i addresses 4 columns of row (i / 4) and receives column i of the 4 rows.
//
// LDS layouts (16-byte chunks permuted per row; conflict-free for each reader and writer):
//   A stage [rows][64]: chunk c of row r at c ^ ((r >> 1) & 7)   (16 rows of one chunk: 64 banks)
//   W stage [64][cols]: chunk c of row r at c ^ ((r & 3) << 2)   (4 rows x 64 bytes: 64 banks;
//                       with 256 columns the permutation stays within each 16-chunk half)
//
// Loads: operand tiles go global -> LDS directly (buffer_load_dwordx4 ... lds, 1 KB per
// wave-wide load, each lane fetching the chunk that the row permutation puts in its slot).
// Buffer descriptors bound A to the tile's rows and W to the rows below K; chunks past K or N
// get an offset beyond every descriptor's size.  Out-of-range buffer loads return zeros, so
// the edges contribute nothing.  N and K are multiples of 8, M is arbitrary.
//
// Tile order: consecutive logical tiles run on one XCD (one L2) at about the same time; they
// are grouped kGemmGroupM row tiles at a time, so both A and W tiles are reused from L2 (a plain
// row- or column-major order re-reads one operand from HBM once per tile of the other).
//
// Epilogue: the tile's results go through LDS (bf16, row-major) so that global reads of the old
// D (accumulate) and the stores are whole 16-byte chunks, predicated on row < M and
// column < N; with accumulate each result is added to the old value in fp32 and rounded once.
#pragma once

#include "common.hpp"

namespace trajspec {

constexpr int kGemmBM = 128;
constexpr int kGemmBN = 128;
constexpr int kGemmBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kGemmGroupM = 8;  // row tiles per ordering group
constexpr int kGemmAElems = kGemmBM * kGemmBK;
constexpr int kGemmWElems = kGemmBK * kGemmBN;

typedef __attribute__((address_space(3))) bf16x4_t gemm_lds_bf16x4_t;
typedef __attribute__((address_space(3))) void gemm_lds_void_t;

struct GemmParams {
    const uint16_t* A;  // [M, K]
    const uint16_t* W;  // [K, N]
    uint16_t* D;        // [M, N]
    int M, N, K;
    int tiles_m;        // row tiles
    int tiles_n;        // column tiles; the grid holds tiles_m * tiles_n workgroups (x)
    float* partial;     // split-K: [splits][M][N] fp32 partial products (grid y = split)
    int k_split;        // split-K: k per split, a multiple of 64
};

// Host-side choice between the two tilings, and the limits of their 32-bit buffer offsets.
constexpr int64_t kGemmBigGridMin = 256;            // 256 x 256 tiles: at least one per CU
constexpr int64_t kGemmMaxK = 1 << 22;              // 256 rows of A below 2^31 bytes
constexpr int64_t kGemmMaxN = 1 << 24;              // 64 rows of W below 2^31 bytes
constexpr int64_t kGemmMaxRecords = 0xFFFFFF00u;    // descriptor sizes stay below the outside offset
constexpr unsigned kGemmOutside = 0xFFFFFFF0u;      // a buffer offset past every descriptor's size
// Word 3 of a raw buffer descriptor on gfx950: 32-bit data format, no swizzle.
constexpr int kGemmBufferFlags = 0x00020000;

// s_waitcnt immediate (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt at
// their maxima) waiting until at most n vector-memory loads are outstanding.
constexpr int wait_vmcnt_imm(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }

// Logical tile of workgroup `bid` in the grouped, XCD-aware order.
__device__ __forceinline__ void gemm_tile_origin(const GemmParams& P, int bm, int bn, int& m0, int& n0) {
    const int tile = xcd_logical_id(blockIdx.x, gridDim.x);
    const int per_group = kGemmGroupM * P.tiles_n;
    const int group = tile / per_group;
    const int first_m = group * kGemmGroupM;
    const int group_m = min(P.tiles_m - first_m, kGemmGroupM);
    const int in_group = tile - group * per_group;
    m0 = (first_m + in_group % group_m) * bm;
    n0 = (in_group / group_m) * bn;
}

__device__ __forceinline__ int gemm_a_slot(int r, int c) { return r * kGemmBK + ((c ^ ((r >> 1) & 7)) << 3); }
__device__ __forceinline__ int gemm_w_slot(int r, int c) { return r * kGemmBN + ((c ^ ((r & 3) << 2)) << 3); }

// Raw buffer descriptor (gfx950): base address, no stride, num_records bytes, word 3 flags.
typedef int32_t gemm_i32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ gemm_i32x4_t gemm_descriptor(const void* base, unsigned num_records) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return gemm_i32x4_t{(int32_t)(uint32_t)a, (int32_t)((a >> 32) & 0xFFFFu), (int32_t)num_records, kGemmBufferFlags};
}

// ---------------------------------------------------------------- 128 x 128 tiles, stage ring
// For grids too small to fill the chip with 256 x 256 tiles (a few sequences' drafts: M in the
// hundreds).  There a workgroup's k loop is a chain of dependent steps, and with one stage in
// flight each step waits a full memory latency; here K advances in steps of 64 through a ring
// of kR1Stages LDS buffers (32 KB each), so the loads of the next kR1Stages - 1 steps are in
// flight while a step multiplies.  4 waves (2 x 2) of 64 x 64 each (2 x 2 MFMA blocks).
constexpr int kR1Stages = 4;
constexpr int kR1StageElems = kGemmAElems + kGemmWElems;   // 32 KB
constexpr int kR1Loads = kGemmAElems / 512 / 4;            // 1 KB wave loads per operand and step: 4
static_assert(kGemmWElems / 512 / 4 == kR1Loads, "equal A and W loads");
constexpr int kR1WaitAhead = wait_vmcnt_imm(2 * kR1Loads * (kR1Stages - 2));  // all but S - 2 steps
static_assert(2 * kR1Loads * (kR1Stages - 2) < 64, "vmcnt has 6 bits");

// One wave-wide 16-byte-per-lane load from a buffer straight into LDS (lane i -> bytes 16 i ..
// 16 i + 15 after `lds_dst`, which must be wave-uniform).  Issued through asm so that the
// compiler does not track it: with loads into several ring buffers outstanding, its own wait
// insertion cannot tell which buffer they write and would wait for all of them before every
// LDS read.  Completion is the caller's explicit s_waitcnt vmcnt; a compiler-tracked load
// issued earlier only sees stricter waits because of these (loads complete in order).
// M0 (the LDS destination of the load) is a register the compiler reserves: the statement
// saves it in a scratch SGPR and restores it after the load, so no code around it sees a
// changed M0.  On gfx9 an SALU write of M0 needs one wait state before an LDS-DMA load reads
// it (the compiler's hazard recognizer does not look inside asm), hence the s_nop.
__device__ __forceinline__ void gemm_dma16(const gemm_i32x4_t& rsrc, unsigned voffset, uint16_t* lds_dst) {
    const unsigned lds = __builtin_amdgcn_readfirstlane((unsigned)(size_t)((gemm_lds_void_t*)lds_dst));
    unsigned saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds), "v"(voffset), "s"(rsrc)
        : "memory");
}

// Workgroup barrier for a stage ring.  __syncthreads() carries a workgroup release fence,
// which waits for every outstanding direct-to-LDS load and would leave one stage in flight.
// Here each wave first waits (s_waitcnt) for exactly the loads of the stage the next step
// reads; the bare s_barrier then makes them visible to every wave (LDS has no caches), and
// the empty asm statements with a memory clobber keep the compiler from moving LDS reads or
// writes across it.  Reads of a stage are consumed by MFMAs before the barrier, so they are
// complete before any wave refills that buffer.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// PARTIAL: split-K; workgroup (x, y) multiplies k in [y k_split, (y + 1) k_split) and writes its
// fp32 products to partial[y] (gemm_split_reduce_kernel adds the splits, the old D, and rounds).
template <bool ACCUMULATE, bool PARTIAL>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_ring128_kernel(GemmParams P) {
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[kR1StageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[kR1StageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf2[kR1StageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf3[kR1StageElems];
    static_assert(kR1Stages == 4, "the ring below is written out for four buffers");
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    int m0, n0;
    gemm_tile_origin(P, kGemmBM, kGemmBN, m0, n0);
    const int M = P.M, N = P.N, K = P.K;
    const int kb = PARTIAL ? (int)blockIdx.y * P.k_split : 0;  // this workgroup's k range
    const int ke = PARTIAL ? min(K, kb + P.k_split) : K;

    // A from row m0 (rows below min(M - m0, 128) in range); W one descriptor per k step, from
    // row k0 and column n0 (rows below ke in range; columns past N are sent outside explicitly)
    const int a_rows = min(M - m0, kGemmBM);
    const gemm_i32x4_t ars = gemm_descriptor(P.A + (int64_t)m0 * K, (unsigned)a_rows * (unsigned)K * 2u);

    // Load slots.  A: wave-load j fills stage rows 32 wave + 8 j .. +8; lane -> row lane >> 3,
    // slot chunk lane & 7, holding logical chunk (lane & 7) ^ ((row >> 1) & 7).  W: wave-load j
    // fills rows 16 wave + 4 j .. +4; lane -> row lane >> 4, slot chunk lane & 15, holding
    // logical chunk (lane & 15) ^ ((row & 3) << 2).
    unsigned a_off[kR1Loads], w_off[kR1Loads];
    int a_kc[kR1Loads];
    bool w_in[kR1Loads];
#pragma unroll
    for (int j = 0; j < kR1Loads; ++j) {
        const int ar = 32 * wave + 8 * j + (lane >> 3);
        const int ac = (lane & 7) ^ ((ar >> 1) & 7);
        a_kc[j] = 8 * ac;
        a_off[j] = (unsigned)ar * (unsigned)K * 2u + 16u * (unsigned)ac;
        const int wr = 16 * wave + 4 * j + (lane >> 4);
        const int wc = (lane & 15) ^ ((wr & 3) << 2);
        w_in[j] = n0 + 8 * wc < N;
        w_off[j] = (unsigned)wr * (unsigned)N * 2u + 16u * (unsigned)wc;
    }
    auto load_stage = [&](int t, uint16_t* stage) {
        const int k0 = kb + t * kGemmBK;
        const int64_t w_rem = ((int64_t)(ke - k0) * N - n0) * 2;
        const gemm_i32x4_t wrs = gemm_descriptor(P.W + (int64_t)k0 * N + n0, (unsigned)(w_rem < kGemmMaxRecords ? w_rem : kGemmMaxRecords));
#pragma unroll
        for (int j = 0; j < kR1Loads; ++j) {
            const unsigned ao = k0 + a_kc[j] < ke ? a_off[j] + 2u * (unsigned)k0 : kGemmOutside;
            gemm_dma16(ars, ao, stage + (32 * wave + 8 * j) * kGemmBK);
        }
#pragma unroll
        for (int j = 0; j < kR1Loads; ++j) {
            const unsigned wo = w_in[j] ? w_off[j] : kGemmOutside;
            gemm_dma16(wrs, wo, stage + kGemmAElems + (16 * wave + 4 * j) * kGemmBN);
        }
    };

    const int wm = wave >> 1, wn = wave & 1;
    const int r32 = lane & 31, h = lane >> 5, i16 = lane & 15, dsub = (lane >> 4) & 1;
    int a_off_f[2][4];
    int w_off_f[2];
#pragma unroll
    for (int am = 0; am < 2; ++am) {
        const int r = wm * 64 + am * 32 + r32;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) a_off_f[am][kk] = gemm_a_slot(r, 2 * kk + h);
    }
#pragma unroll
    for (int bn = 0; bn < 2; ++bn) {
        const int r = 8 * h + (i16 >> 2);  // +16 kk and +4 keep r & 3
        const int col = wn * 64 + bn * 32 + dsub * 16 + (i16 & 3) * 4;
        w_off_f[bn] = kGemmAElems + gemm_w_slot(r, col >> 3) + (col & 7);
    }

    f32x16_t acc[2][2];
#pragma unroll
    for (int am = 0; am < 2; ++am)
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) acc[am][bn] = f32x16_t{};

    const int nk = (ke - kb + kGemmBK - 1) / kGemmBK;
    // step t: load step t + 3 (if any) into the buffer step t - 1 read, multiply the stage in
    // `cur`, wait until this wave's loads of step t + 1 have landed, barrier
    auto step = [&](int t, const uint16_t* cur, uint16_t* ahead) {
        if (t + kR1Stages - 1 < nk) load_stage(t + kR1Stages - 1, ahead);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            bf16x8_t af[2], bf[2];
#pragma unroll
            for (int am = 0; am < 2; ++am) af[am] = *reinterpret_cast<const bf16x8_t*>(cur + a_off_f[am][kk]);
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const uint16_t* p = cur + w_off_f[bn] + 16 * kk * kGemmBN;
                const bf16x4_t b0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((gemm_lds_bf16x4_t*)(p));
                const bf16x4_t b1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((gemm_lds_bf16x4_t*)(p + 4 * kGemmBN));
                bf[bn] = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
            }
#pragma unroll
            for (int am = 0; am < 2; ++am)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn)
                    acc[am][bn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[am], bf[bn], acc[am][bn], 0, 0, 0);
        }
        // loads issued after step t + 1's: those of steps t + 2 .. min(t + 3, nk - 1)
        if (t + kR1Stages - 1 < nk)
            __builtin_amdgcn_s_waitcnt(kR1WaitAhead);
        else
            __builtin_amdgcn_s_waitcnt(wait_vmcnt_imm(0));
        ring_barrier();
    };
    load_stage(0, buf0);
    if (1 < nk) load_stage(1, buf1);
    if (2 < nk) load_stage(2, buf2);
    if (kR1Stages - 1 <= nk)
        __builtin_amdgcn_s_waitcnt(kR1WaitAhead);
    else
        __builtin_amdgcn_s_waitcnt(wait_vmcnt_imm(0));
    ring_barrier();
    for (int t0 = 0; t0 < nk; t0 += kR1Stages) {
        step(t0, buf0, buf3);
        if (t0 + 1 < nk) step(t0 + 1, buf1, buf0);
        if (t0 + 2 < nk) step(t0 + 2, buf2, buf1);
        if (t0 + 3 < nk) step(t0 + 3, buf3, buf2);
    }

    if (PARTIAL) {
        // fp32 products straight from the accumulators: for each e, 32 lanes store 128
        // contiguous bytes of one row
        float* out = P.partial + (int64_t)blockIdx.y * M * N;
#pragma unroll
        for (int am = 0; am < 2; ++am)
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const int col = n0 + wn * 64 + bn * 32 + r32;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = m0 + wm * 64 + am * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
                    if (row < M && col < N) out[(int64_t)row * N + col] = acc[am][bn][e];
                }
            }
        return;
    }

    // Epilogue through LDS (buf0, freed by the last barrier).
    static_assert(kGemmBM * kGemmBN <= kR1StageElems, "output tile fits one stage buffer");
    const int ec = tid & 15;
    const bool col_ok = n0 + 8 * ec < N;
    if (ACCUMULATE) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int r = (tid >> 4) + 16 * j;
            u32x4_t v = u32x4_t{0, 0, 0, 0};
            if (col_ok && m0 + r < M) v = *reinterpret_cast<const u32x4_t*>(P.D + (int64_t)(m0 + r) * N + n0 + 8 * ec);
            *reinterpret_cast<u32x4_t*>(buf0 + r * kGemmBN + 8 * ec) = v;
        }
        __syncthreads();
    }
#pragma unroll
    for (int am = 0; am < 2; ++am) {
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int c = wn * 64 + bn * 32 + r32;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                uint16_t* p = buf0 + (wm * 64 + am * 32 + 8 * (e >> 2) + 4 * h + (e & 3)) * kGemmBN + c;
                float v = acc[am][bn][e];
                if (ACCUMULATE) v += bf16_bits_to_float(*p);
                *p = __builtin_bit_cast(uint16_t, (__bf16)v);  // round to nearest even
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int r = (tid >> 4) + 16 * j;
        if (col_ok && m0 + r < M)
            *reinterpret_cast<u32x4_t*>(P.D + (int64_t)(m0 + r) * N + n0 + 8 * ec) =
                *reinterpret_cast<const u32x4_t*>(buf0 + r * kGemmBN + 8 * ec);
    }
}

// D = round(sum over splits of partial (+ D)), 8 columns per thread (N % 8 == 0, so a chunk
// stays in one row); grid-stride over the M x N / 8 chunks.
template <bool ACCUMULATE>
__global__ __launch_bounds__(256) void gemm_split_reduce_kernel(const float* __restrict__ partial, int splits,
                                                                uint16_t* __restrict__ D, int M, int N) {
    const int64_t MN = (int64_t)M * N;
    const int64_t chunks = MN / 8;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < chunks; q += (int64_t)gridDim.x * 256) {
        const int64_t e0 = 8 * q;
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
        for (int s2 = 0; s2 < splits; ++s2) {
            const float4 lo = *reinterpret_cast<const float4*>(partial + s2 * MN + e0);
            const float4 hi = *reinterpret_cast<const float4*>(partial + s2 * MN + e0 + 4);
            v[0] += lo.x; v[1] += lo.y; v[2] += lo.z; v[3] += lo.w;
            v[4] += hi.x; v[5] += hi.y; v[6] += hi.z; v[7] += hi.w;
        }
        u32x4_t o;
        if (ACCUMULATE) {
            const u32x4_t d = *reinterpret_cast<const u32x4_t*>(D + e0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] += bf16_lo(d[i]);
                v[2 * i + 1] += bf16_hi(d[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            o[i] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2 * i]) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2 * i + 1]) << 16);
        *reinterpret_cast<u32x4_t*>(D + e0) = o;
    }
}

// ---------------------------------------------------------------- 256 x 256 tiles
// For grids that fill the chip: 8 waves (2 x 4) own a 256 x 256 tile, 128 x 64 each
// (4 x 2 MFMA blocks, 128 fp32 accumulators per lane), so a wave reads 768 LDS bytes per MFMA
// and the workgroup moves half the global bytes per flop of the 128 x 128 tile.  Two 64 KB
// stages: step t + 1 is loaded while step t multiplies, one barrier per step (here the direct
// loads of this kernel are ordinary compiler-tracked builtins: with one other stage in flight,
// in a separate LDS array, the compiler's own waits are exact).
constexpr int kG2BM = 256;
constexpr int kG2BN = 256;
constexpr int kG2BK = 64;
constexpr int kG2Waves = 8;
constexpr int kG2Threads = kG2Waves * 64;
constexpr int kG2AElems = kG2BM * kG2BK;               // 32 KB
constexpr int kG2WElems = kG2BK * kG2BN;               // 32 KB
constexpr int kG2StageElems = kG2AElems + kG2WElems;   // 64 KB
constexpr int kG2LoadsPerWave = kG2AElems / 512 / kG2Waves;  // 1 KB wave loads per operand: 4
static_assert(kG2WElems / 512 / kG2Waves == kG2LoadsPerWave, "equal A and W loads");

__device__ __forceinline__ int g2_w_slot(int r, int c) { return r * kG2BN + ((c ^ ((r & 3) << 2)) << 3); }

template <bool ACCUMULATE>
__global__ __launch_bounds__(kG2Threads, 1) void gemm_tile256_kernel(GemmParams P) {
    // Two stage buffers as separate arrays: the compiler then knows that the direct loads into
    // one do not alias the fragment reads of the other and does not wait for them.
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[kG2StageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[kG2StageElems];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    int m0, n0;
    gemm_tile_origin(P, kG2BM, kG2BN, m0, n0);
    const int M = P.M, N = P.N, K = P.K;

    // Descriptors: A from row m0 (its rows below min(M - m0, 256) are in range); W one per k
    // step, from row k0 and column n0 (the rows below K are in range, columns past N are sent
    // outside explicitly), so every offset stays within a step's 64 rows.
    const int a_rows = min(M - m0, kG2BM);
    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.A + (int64_t)m0 * K), (short)0, (int)((unsigned)a_rows * (unsigned)K * 2u), kGemmBufferFlags);

    // This lane's load slots.  A: wave-load j fills tile rows 32 wave + 8 j .. +8; lane -> row
    // (lane >> 3), slot chunk lane & 7, which holds logical chunk (lane & 7) ^ ((row >> 1) & 7).
    // W: wave-load j fills tile rows 8 wave + 2 j .. +2; lane -> row (lane >> 5), slot chunk
    // lane & 31, holding logical chunk (lane & 31) ^ ((row & 3) << 2).
    unsigned a_off[kG2LoadsPerWave], w_off[kG2LoadsPerWave];
    int a_kc[kG2LoadsPerWave];  // logical k of the lane's A chunk within a step
    bool w_in[kG2LoadsPerWave];
#pragma unroll
    for (int j = 0; j < kG2LoadsPerWave; ++j) {
        const int ar = 32 * wave + 8 * j + (lane >> 3);
        const int ac = (lane & 7) ^ ((ar >> 1) & 7);
        a_kc[j] = 8 * ac;
        a_off[j] = (unsigned)ar * (unsigned)K * 2u + 16u * (unsigned)ac;
        const int wr = 8 * wave + 2 * j + (lane >> 5);
        const int wc = (lane & 31) ^ ((wr & 3) << 2);
        w_in[j] = n0 + 8 * wc < N;
        w_off[j] = (unsigned)wr * (unsigned)N * 2u + 16u * (unsigned)wc;
    }
    auto load_stage = [&](int t, uint16_t* stage) {
        const int k0 = t * kG2BK;
        const int64_t w_rem = ((int64_t)(K - k0) * N - n0) * 2;
        const __amdgpu_buffer_rsrc_t wrs =
            __builtin_amdgcn_make_buffer_rsrc((void*)(P.W + (int64_t)k0 * N + n0), (short)0,
                                              (int)(unsigned)(w_rem < kGemmMaxRecords ? w_rem : kGemmMaxRecords), kGemmBufferFlags);
#pragma unroll
        for (int j = 0; j < kG2LoadsPerWave; ++j) {
            const unsigned ao = k0 + a_kc[j] < K ? a_off[j] + 2u * (unsigned)k0 : kGemmOutside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ars, (gemm_lds_void_t*)(stage + (32 * wave + 8 * j) * kG2BK), 16,
                                                     ao, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kG2LoadsPerWave; ++j) {
            const unsigned wo = w_in[j] ? w_off[j] : kGemmOutside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                wrs, (gemm_lds_void_t*)(stage + kG2AElems + (8 * wave + 2 * j) * kG2BN), 16, wo, 0, 0, 0);
        }
    };

    // Fragment reads.  Wave (wm, wn) = (wave >> 2, wave & 3) owns rows 128 wm .. +128 and
    // columns 64 wn .. +64.  A row r = 128 wm + 32 am + lane % 32 keeps (r >> 1) & 7 equal for
    // every am, so the permuted chunk offset depends on kk only.
    const int wm = wave >> 2, wn = wave & 3;
    const int r32 = lane & 31, h = lane >> 5, i16 = lane & 15, dsub = (lane >> 4) & 1;
    const int a_row0 = (wm * 128 + r32) * kG2BK;
    int a_chunk[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) a_chunk[kk] = ((2 * kk + h) ^ ((r32 >> 1) & 7)) << 3;
    int b_off[2];
#pragma unroll
    for (int bn = 0; bn < 2; ++bn) {
        const int r = 8 * h + (i16 >> 2);  // +16 kk and +4 keep r & 3
        const int col = wn * 64 + bn * 32 + dsub * 16 + (i16 & 3) * 4;
        b_off[bn] = kG2AElems + g2_w_slot(r, col >> 3) + (col & 7);
    }

    f32x16_t acc[4][2];
#pragma unroll
    for (int am = 0; am < 4; ++am)
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) acc[am][bn] = f32x16_t{};

    const int nk = (K + kG2BK - 1) / kG2BK;
    // one k step: load step t + 1 into `nxt` (if any), multiply the stage in `cur`, then wait
    // for this wave's loads and meet at the barrier
    auto step = [&](int t, const uint16_t* cur, uint16_t* nxt) {
        if (t + 1 < nk) load_stage(t + 1, nxt);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            bf16x8_t af[4], bf[2];
#pragma unroll
            for (int am = 0; am < 4; ++am)
                af[am] = *reinterpret_cast<const bf16x8_t*>(cur + a_row0 + am * 32 * kG2BK + a_chunk[kk]);
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const uint16_t* p = cur + b_off[bn] + 16 * kk * kG2BN;
                const bf16x4_t b0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((gemm_lds_bf16x4_t*)(p));
                const bf16x4_t b1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((gemm_lds_bf16x4_t*)(p + 4 * kG2BN));
                bf[bn] = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
            }
#pragma unroll
            for (int am = 0; am < 4; ++am)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn)
                    acc[am][bn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[am], bf[bn], acc[am][bn], 0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(wait_vmcnt_imm(0));
        __syncthreads();
    };
    load_stage(0, buf0);
    __builtin_amdgcn_s_waitcnt(wait_vmcnt_imm(0));
    __syncthreads();
    for (int t = 0; t < nk; t += 2) {
        step(t, buf0, buf1);
        if (t + 1 < nk) step(t + 1, buf1, buf0);
    }

    // Epilogue through LDS (the last barrier above freed both buffers): the output tile is
    // staged as bf16 [256][256] row-major, rows 0..127 in buf0 and 128..255 in buf1, so global
    // traffic is 16-byte chunks (thread tid moves chunk tid & 31 of rows (tid >> 5) + 16 j).
    // With ACCUMULATE the old D tile is staged first and each lane adds its fp32 results to it
    // and rounds once.  Wave (wm, wn) touches only rows of buf{wm}.
    uint16_t* half = wm == 0 ? buf0 : buf1;
    const int ec = tid & 31;
    const bool col_ok = n0 + 8 * ec < N;
    if (ACCUMULATE) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int r = (tid >> 5) + 16 * j;
            uint16_t* dst = (j < 8 ? buf0 : buf1) + (r & 127) * kG2BN + 8 * ec;
            u32x4_t v = u32x4_t{0, 0, 0, 0};
            if (col_ok && m0 + r < M) v = *reinterpret_cast<const u32x4_t*>(P.D + (int64_t)(m0 + r) * N + n0 + 8 * ec);
            *reinterpret_cast<u32x4_t*>(dst) = v;
        }
        __syncthreads();
    }
    // acc[am][bn][e] is row 8 (e / 4) + 4 h + e % 4, column lane % 32 of its 32 x 32 block
#pragma unroll
    for (int am = 0; am < 4; ++am) {
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int c = wn * 64 + bn * 32 + r32;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                uint16_t* p = half + (am * 32 + 8 * (e >> 2) + 4 * h + (e & 3)) * kG2BN + c;
                float v = acc[am][bn][e];
                if (ACCUMULATE) v += bf16_bits_to_float(*p);
                *p = __builtin_bit_cast(uint16_t, (__bf16)v);  // round to nearest even
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int r = (tid >> 5) + 16 * j;
        const uint16_t* src = (j < 8 ? buf0 : buf1) + (r & 127) * kG2BN + 8 * ec;
        if (col_ok && m0 + r < M)
            *reinterpret_cast<u32x4_t*>(P.D + (int64_t)(m0 + r) * N + n0 + 8 * ec) =
                *reinterpret_cast<const u32x4_t*>(src);
    }
}

}  // namespace trajspec
