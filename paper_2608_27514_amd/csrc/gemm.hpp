// Dense bf16 projection GEMM of the verification layer: D[M,N] = A[M,K] W[K,N] (+ D), all
// row-major bf16, fp32 accumulation on v_mfma_f32_32x32x16_bf16, one bf16 rounding (nearest
// even) of each result.  A holds the packed draft tokens (M = B N L rows), W a weight matrix.
//
// Tiling: a workgroup of 4 waves owns a 128 x 128 output tile (2 x 2 waves of 64 x 64, each
// 2 x 2 MFMA blocks of 32 x 32) and walks K in steps of 64 through two LDS buffers: the
// global loads of step t + 1 are in flight while step t multiplies, one barrier per step.
//
// Fragments: the MFMA takes 8 k-values per lane; lane half h = lane / 32 holds k = 8h .. 8h+7
// of each 16-wide k slice, for row (A) or column (W) lane % 32.  A is k-contiguous, so an A
// fragment is one 16-byte LDS read.  W is n-contiguous: a W fragment is two transposing
// reads (ds_read_b64_tr_b16) of slice rows 8h .. 8h+3 and 8h+4 .. 8h+7; in each group of 16
// lanes, lane i addresses 4 columns of row (i / 4) and receives column i of the 4 rows.
//
// LDS layouts (16-byte chunks permuted per row; conflict-free for each reader and writer):
//   A tile [128][64]: chunk c of row r at c ^ ((r >> 1) & 7)   (16 rows of one chunk: 64 banks)
//   W tile [64][128]: chunk c of row r at c ^ ((r & 3) << 2)   (4 rows x 64 bytes: 64 banks)
//
// Edges: N and K are multiples of 8, M is arbitrary.  A 16-byte chunk outside the matrix is
// loaded as zeros on both operands (no contribution).
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
#ifndef TRAJ_GEMM_GROUP_M
#define TRAJ_GEMM_GROUP_M 8
#endif
constexpr int kGemmGroupM = TRAJ_GEMM_GROUP_M;  // row tiles per ordering group
constexpr int kGemmAElems = kGemmBM * kGemmBK;
constexpr int kGemmWElems = kGemmBK * kGemmBN;
constexpr int kGemmStageElems = kGemmAElems + kGemmWElems;
// 16-byte chunks per operand tile and thread: 1024 / 256
constexpr int kGemmLoads = kGemmAElems / 8 / kGemmThreads;
static_assert(kGemmWElems / 8 / kGemmThreads == kGemmLoads, "equal A and W tile loads");

typedef __attribute__((address_space(3))) bf16x4_t gemm_lds_bf16x4_t;

struct GemmParams {
    const uint16_t* A;  // [M, K]
    const uint16_t* W;  // [K, N]
    uint16_t* D;        // [M, N]
    int M, N, K;
    int tiles_m;        // ceil(M / 128)
    int tiles_n;        // ceil(N / 128); the grid holds tiles_m * tiles_n workgroups
};

__device__ __forceinline__ int gemm_a_slot(int r, int c) { return r * kGemmBK + ((c ^ ((r >> 1) & 7)) << 3); }
__device__ __forceinline__ int gemm_w_slot(int r, int c) { return r * kGemmBN + ((c ^ ((r & 3) << 2)) << 3); }

template <bool ACCUMULATE>
__global__ __launch_bounds__(kGemmThreads) void gemm_tile128_kernel(GemmParams P) {
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * kGemmStageElems];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // Consecutive logical tiles run on one XCD (one L2) at about the same time; they are
    // grouped kGemmGroupM row tiles x (64 / kGemmGroupM) column tiles, so A and W tiles are
    // both reused from L2 (a plain row-major or column-major order re-reads A or W from HBM
    // once per tile of the other operand).
    const int tile = xcd_logical_id(blockIdx.x, gridDim.x);
    const int per_group = kGemmGroupM * P.tiles_n;
    const int group = tile / per_group;
    const int first_m = group * kGemmGroupM;
    const int group_m = min(P.tiles_m - first_m, kGemmGroupM);
    const int in_group = tile - group * per_group;
    const int m0 = (first_m + in_group % group_m) * kGemmBM;
    const int n0 = (in_group / group_m) * kGemmBN;
    const int M = P.M, N = P.N, K = P.K;

    // loads: chunk tid + 256 j of each tile.  A: row (tid >> 3) + 32 j, chunk tid & 7.
    // W: row (tid >> 4) + 16 j, chunk tid & 15.
    const int a_r = tid >> 3, a_c = tid & 7;
    const int w_r = tid >> 4, w_c = tid & 15;
    const bool w_col_ok = n0 + 8 * w_c < N;
    const uint16_t* a_src = P.A + (int64_t)(m0 + a_r) * K + 8 * a_c;
    const uint16_t* w_src = P.W + (int64_t)w_r * N + n0 + 8 * w_c;
    u32x4_t ra[kGemmLoads], rw[kGemmLoads];

    auto load = [&](int t) {
        const int k0 = t * kGemmBK;
        const bool a_k_ok = k0 + 8 * a_c < K;
#pragma unroll
        for (int j = 0; j < kGemmLoads; ++j) {
            const bool ok = a_k_ok && m0 + a_r + 32 * j < M;
            ra[j] = ok ? *reinterpret_cast<const u32x4_t*>(a_src + (int64_t)(32 * j) * K + k0) : u32x4_t{0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < kGemmLoads; ++j) {
            const bool ok = w_col_ok && k0 + w_r + 16 * j < K;
            rw[j] = ok ? *reinterpret_cast<const u32x4_t*>(w_src + (int64_t)(k0 + 16 * j) * N) : u32x4_t{0, 0, 0, 0};
        }
    };
    auto store = [&](int buf) {
        uint16_t* sa = lds + buf * kGemmStageElems;
        uint16_t* sw = sa + kGemmAElems;
#pragma unroll
        for (int j = 0; j < kGemmLoads; ++j) *reinterpret_cast<u32x4_t*>(sa + gemm_a_slot(a_r + 32 * j, a_c)) = ra[j];
#pragma unroll
        for (int j = 0; j < kGemmLoads; ++j) *reinterpret_cast<u32x4_t*>(sw + gemm_w_slot(w_r + 16 * j, w_c)) = rw[j];
    };

    // fragment offsets within a stage (elements)
    const int wm = wave >> 1, wn = wave & 1;
    const int r32 = lane & 31, h = lane >> 5, i16 = lane & 15, dsub = (lane >> 4) & 1;
    int a_off[2][4];
    int w_off[2];
#pragma unroll
    for (int am = 0; am < 2; ++am) {
        const int r = wm * 64 + am * 32 + r32;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) a_off[am][kk] = gemm_a_slot(r, 2 * kk + h);
    }
#pragma unroll
    for (int bn = 0; bn < 2; ++bn) {
        const int r = 8 * h + (i16 >> 2);  // slice row; +16 kk and +4 keep r & 3
        const int col = wn * 64 + bn * 32 + dsub * 16 + (i16 & 3) * 4;
        w_off[bn] = kGemmAElems + gemm_w_slot(r, col >> 3) + (col & 7);
    }

    f32x16_t acc[2][2];
#pragma unroll
    for (int am = 0; am < 2; ++am)
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) acc[am][bn] = f32x16_t{};

    const int nk = (K + kGemmBK - 1) / kGemmBK;
    load(0);
    store(0);
    __syncthreads();
    for (int t = 0; t < nk; ++t) {
        if (t + 1 < nk) load(t + 1);
        const uint16_t* st = lds + (t & 1) * kGemmStageElems;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            bf16x8_t af[2], bf[2];
#pragma unroll
            for (int am = 0; am < 2; ++am) af[am] = *reinterpret_cast<const bf16x8_t*>(st + a_off[am][kk]);
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const uint16_t* p = st + w_off[bn] + 16 * kk * kGemmBN;
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
        if (t + 1 < nk) store((t + 1) & 1);
        __syncthreads();
    }

    // Epilogue through LDS (the last barrier above freed it): the output tile is staged as bf16
    // [128][128] row-major, so global traffic is 16-byte chunks (thread tid moves chunk tid & 15
    // of rows (tid >> 4) + 16 j).  With ACCUMULATE the old D tile is staged first and each lane
    // adds its fp32 results to it and rounds once.
    const int ec = tid & 15;
    const bool col_ok = n0 + 8 * ec < N;
    if (ACCUMULATE) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int r = (tid >> 4) + 16 * j;
            u32x4_t v = u32x4_t{0, 0, 0, 0};
            if (col_ok && m0 + r < M) v = *reinterpret_cast<const u32x4_t*>(P.D + (int64_t)(m0 + r) * N + n0 + 8 * ec);
            *reinterpret_cast<u32x4_t*>(lds + r * kGemmBN + 8 * ec) = v;
        }
        __syncthreads();
    }
    // acc[am][bn][e] is row 8 (e / 4) + 4 h + e % 4, column lane % 32 of its 32 x 32 block
#pragma unroll
    for (int am = 0; am < 2; ++am) {
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int c = wn * 64 + bn * 32 + r32;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                uint16_t* p = lds + (wm * 64 + am * 32 + 8 * (e >> 2) + 4 * h + (e & 3)) * kGemmBN + c;
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
                *reinterpret_cast<const u32x4_t*>(lds + r * kGemmBN + 8 * ec);
    }
}

// ---------------------------------------------------------------- 256 x 256 tiles
// For grids that fill the chip: 8 waves (2 x 4) own a 256 x 256 tile, 128 x 64 each
// (4 x 2 MFMA blocks, 128 fp32 accumulators per lane), so a wave reads 768 LDS bytes per MFMA
// and the workgroup moves half the global bytes per flop of the 128 x 128 tile.  Operand
// tiles go global -> LDS directly (buffer_load_dwordx4 ... lds, 1 KB per wave-wide load, each
// lane fetching the chunk that the row permutation puts in its slot); loads past the matrix
// return zeros (rows through the descriptor's size, chunks past K or N through an offset
// beyond it).  Two 64 KB stages: step t + 1 is loaded while step t multiplies, one barrier
// per step.  LDS layouts as above with 256-element W rows (32 chunks; the permutation only
// touches chunk bits 2..3, so a row's chunks stay in place modulo 16).
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
constexpr unsigned kG2Outside = 0xFFFFFFF0u;  // a buffer offset past every descriptor's size
// Word 3 of a raw buffer descriptor on gfx950: 32-bit data format, no swizzle.
constexpr int kG2BufferFlags = 0x00020000;
// s_waitcnt immediate (gfx9 encoding) for vector-memory loads only: vmcnt = 0.
constexpr int kG2WaitVmcnt0 = 0x0F70;

typedef __attribute__((address_space(3))) void gemm_lds_void_t;

// Host-side choice between the two tilings.
constexpr int64_t kGemmBigGridMin = 256;            // 256 x 256 tiles: at least one per CU
constexpr int64_t kGemmBigMaxK = 1 << 22;           // 256 rows of A below 2^31 bytes
constexpr int64_t kGemmBigMaxWBytes = 0xFFFFFF00u;  // all of W below the outside offset

__device__ __forceinline__ int g2_w_slot(int r, int c) { return r * kG2BN + ((c ^ ((r & 3) << 2)) << 3); }

template <bool ACCUMULATE>
__global__ __launch_bounds__(kG2Threads, 1) void gemm_tile256_kernel(GemmParams P) {
    // Two stage buffers as separate arrays: the compiler then knows that the direct loads into
    // one do not alias the fragment reads of the other and does not wait for them.
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[kG2StageElems];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[kG2StageElems];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int tile = xcd_logical_id(blockIdx.x, gridDim.x);
    const int per_group = kGemmGroupM * P.tiles_n;
    const int group = tile / per_group;
    const int first_m = group * kGemmGroupM;
    const int group_m = min(P.tiles_m - first_m, kGemmGroupM);
    const int in_group = tile - group * per_group;
    const int m0 = (first_m + in_group % group_m) * kG2BM;
    const int n0 = (in_group / group_m) * kG2BN;
    const int M = P.M, N = P.N, K = P.K;

    // Descriptors: A from row m0 (its rows below min(M - m0, 256) are in range), W from column
    // n0 (rows below K are in range; columns past N are sent outside explicitly).
    const int a_rows = min(M - m0, kG2BM);
    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.A + (int64_t)m0 * K), (short)0, (int)((unsigned)a_rows * (unsigned)K * 2u), kG2BufferFlags);
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(P.W + n0), (short)0, (int)(((unsigned)K * (unsigned)N - (unsigned)n0) * 2u), kG2BufferFlags);

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
#pragma unroll
        for (int j = 0; j < kG2LoadsPerWave; ++j) {
            const unsigned ao = k0 + a_kc[j] < K ? a_off[j] + 2u * (unsigned)k0 : kG2Outside;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ars, (gemm_lds_void_t*)(stage + (32 * wave + 8 * j) * kG2BK), 16,
                                                     ao, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kG2LoadsPerWave; ++j) {
            const unsigned wo = w_in[j] ? w_off[j] + (unsigned)k0 * (unsigned)N * 2u : kG2Outside;
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
        __builtin_amdgcn_s_waitcnt(kG2WaitVmcnt0);
        __syncthreads();
    };
    load_stage(0, buf0);
    __builtin_amdgcn_s_waitcnt(kG2WaitVmcnt0);
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
