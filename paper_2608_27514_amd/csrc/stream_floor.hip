// libtrajfloor: measurement aids (not part of the verification step and not declared in the
// library's C ABI): the streaming-read floor of the logit pass, and the rate the matrix cores
// sustain on the attention's own operand data.
//
// The kernel reads rows of bytes with exactly the launch shape and load pattern of the logit pass
// (conf_topk.hpp): one workgroup per row, THREADS lanes, 16-byte non-temporal loads held in a ring
// of DEPTH sweeps of U vectors per lane, unconditional loads in a loop over whole groups of DEPTH
// sweeps, the row's last partial sweep loaded through the same ring.  Instead of the softmax and
// the top-k it only XORs the words it reads (so the loads stay live) and writes one word per
// wave.  Its duration on the same rows is what the memory system
// delivers to that access pattern: the logit pass's time against it separates the cost of the
// arithmetic from the cost of the reads.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "conf_topk.hpp"  // the logit pass's launch plan (plan_conf_topk)

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// grid.x = rows * splits; workgroup (row, split) reads vectors [split * chunk, min(nvec, (split + 1) * chunk))
template <int THREADS, int U, int DEPTH>
__global__ __launch_bounds__(THREADS) void stream_floor_kernel(const u32x4* __restrict__ data, int64_t row_stride_vec,
                                                               int nvec_row, int splits, int chunk,
                                                               uint32_t* __restrict__ sink) {
    constexpr int SW = THREADS * U;
    const int row = blockIdx.x / splits;
    const int split = blockIdx.x - row * splits;
    const int begin = split * chunk;
    const int nvec = min(nvec_row, begin + chunk) - begin;
    const u32x4* vp = data + (int64_t)row * row_stride_vec + begin;
    const int tid = threadIdx.x;
    const int nfull = nvec / SW;
    const bool tail = nvec > nfull * SW;
    const int nsw = nfull + (tail ? 1 : 0);
    uint32_t acc = 0;
    auto take = [&](const u32x4& w) { acc ^= w[0] ^ w[1] ^ w[2] ^ w[3]; };
    if (nsw > 0) {
        u32x4 buf[DEPTH][U];
        auto load = [&](int sweep, u32x4 (&b)[U]) {  // indices past the row clamped to its last vector
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int v = sweep * SW + u * THREADS + tid;
                b[u] = __builtin_nontemporal_load(vp + (v < nvec ? v : nvec - 1));
            }
        };
        auto take_sweep = [&](int sweep, const u32x4 (&b)[U], bool partial) {
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (!partial || sweep * SW + u * THREADS + tid < nvec) take(b[u]);
        };
#pragma unroll
        for (int d = 0; d + 1 < DEPTH; ++d) load(d, buf[d]);
        int it = 0;
        for (; it + DEPTH <= nfull; it += DEPTH) {
#pragma unroll
            for (int j = 0; j < DEPTH; ++j) {
                load(it + j + DEPTH - 1, buf[(j + DEPTH - 1) % DEPTH]);
                __builtin_amdgcn_sched_barrier(0);
                take_sweep(it + j, buf[j], false);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // the remaining full sweeps and the partial one, as one more group with unconditional loads
#pragma unroll
        for (int j = 0; j < DEPTH; ++j) {
            load(it + j + DEPTH - 1, buf[(j + DEPTH - 1) % DEPTH]);
            __builtin_amdgcn_sched_barrier(0);
            if (it + j < nsw) take_sweep(it + j, buf[j], it + j >= nfull);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int t = 0; t < 6; ++t) {  // the wave's XOR on the exchange network, as the pass's reductions
        uint32_t a, b;
        trajspec::lane_pair(t, acc, a, b);
        acc = a ^ b;
    }
    if ((tid & 63) == 0) sink[((int64_t)blockIdx.x * (THREADS / 64) + (tid >> 6)) & 4095] = acc;
}

// The sustained bf16 MFMA rate: each wave loads four A and four B fragments (16 bytes per lane)
// from the two operand arrays it is given (the attention's cache K and Q), then issues `iters`
// rounds of 16 v_mfma_f32_32x32x16_bf16 on four independent accumulators -- the matrix cores'
// own issue rate, with the data toggling as the attention's does (the power the multiplies draw,
// and so the clock the part holds, depends on the operands).  Two 4-wave workgroups per CU, as
// the attention.  Wave 0 of workgroup 0 records shader-clock cycles (s_memtime) and 100 MHz
// reference ticks (s_memrealtime) around its loop.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint64_t shader_cycles() {
    uint64_t t;
    asm volatile("s_memtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t)::"memory");
    return t;
}
__device__ __forceinline__ uint64_t ref_ticks() {
    uint64_t t;
    asm volatile("s_memrealtime %0\n\ts_waitcnt lgkmcnt(0)" : "=s"(t)::"memory");
    return t;
}

__global__ __launch_bounds__(256, 2) void mfma_rate_kernel(const u32x4* __restrict__ a_src, int64_t a_vecs,
                                                           const u32x4* __restrict__ b_src, int64_t b_vecs, int iters,
                                                           float* __restrict__ sink, uint64_t* __restrict__ clock) {
    const int64_t gl = (int64_t)blockIdx.x * 256 + threadIdx.x;
    bf16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = __builtin_bit_cast(bf16x8, a_src[(gl * 4 + i) % a_vecs]);
        b[i] = __builtin_bit_cast(bf16x8, b_src[(gl * 4 + i) % b_vecs]);
    }
    f32x16 c[4] = {{}, {}, {}, {}};
    uint64_t t0 = 0, r0 = 0;
    const bool timer = blockIdx.x == 0 && threadIdx.x == 0;
    if (timer) {
        t0 = shader_cycles();
        r0 = ref_ticks();
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                c[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + k) & 3], b[(3 * i + k) & 3], c[i], 0, 0, 0);
    }
    if (timer) {
        clock[0] = shader_cycles() - t0;
        clock[1] = ref_ticks() - r0;
    }
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc += c[i][v];
    if ((threadIdx.x & 63) == 0) sink[(gl >> 6) & 4095] = acc;  // keeps the products live
}

template <int THREADS, int U, int DEPTH>
void launch(const void* data, int64_t rows, int64_t stride_vec, int nvec, int splits, int chunk, uint32_t* sink,
            hipStream_t s) {
    hipLaunchKernelGGL((stream_floor_kernel<THREADS, U, DEPTH>), dim3((unsigned)(rows * splits)), dim3(THREADS), 0, s,
                       static_cast<const u32x4*>(data), stride_vec, nvec, splits, chunk, sink);
}

}  // namespace

extern "C" {

// Reads the logit rows that traj_confidence_topk would read for this shape (rows x vocab elements
// of elem_bytes (2: bf16, 4: fp32), row r at data + r * row_stride elements), with the launch shape
// the logit pass plans for it (workgroup size, load ring, row slices).  data 16-byte aligned,
// vocab * elem_bytes and row_stride * elem_bytes multiples of 16 (the pass's vector path); sink:
// 4096 uint32 (device).  shape_out (host, may be NULL) receives threads, unroll, depth, splits.
// Returns 0, or -1 when the arguments do not meet these conditions (nothing launched).
int traj_floor_logit_read(const void* data, int64_t rows, int64_t vocab, int64_t row_stride, int32_t elem_bytes,
                          uint32_t* sink, int32_t* shape_out, void* stream) {
    if (data == nullptr || sink == nullptr || rows < 1 || vocab < 1 || row_stride < vocab) return -1;
    if (elem_bytes != 2 && elem_bytes != 4) return -1;
    if ((vocab * elem_bytes) % 16 != 0 || (row_stride * elem_bytes) % 16 != 0) return -1;
    if ((reinterpret_cast<uintptr_t>(data) & 15u) != 0 || vocab >= ((int64_t)1 << 31) || rows >= ((int64_t)1 << 31) / 64)
        return -1;
    const int vec = 16 / elem_bytes;
    const trajspec::TopkPlan plan = trajspec::plan_conf_topk(rows, vocab, vec);
    if (shape_out != nullptr) {
        shape_out[0] = plan.threads;
        shape_out[1] = plan.unroll;
        shape_out[2] = plan.depth;
        shape_out[3] = plan.splits;
    }
    const int nvec = (int)(vocab / vec);
    const int chunk = plan.splits > 1 ? plan.chunk / vec : nvec;  // chunks are whole sweeps, so whole vectors
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t stride_vec = row_stride * elem_bytes / 16;
    if (plan.threads == 64 && plan.unroll == 2 && plan.depth == 3) {
        launch<64, 2, 3>(data, rows, stride_vec, nvec, plan.splits, chunk, sink, s);
    } else if (plan.threads == 256 && plan.unroll == 2 && plan.depth == 2) {
        launch<256, 2, 2>(data, rows, stride_vec, nvec, plan.splits, chunk, sink, s);
    } else if (plan.threads == 512 && plan.unroll == 4 && plan.depth == 2) {
        launch<512, 4, 2>(data, rows, stride_vec, nvec, plan.splits, chunk, sink, s);
    } else if (plan.threads == 512 && plan.unroll == 2 && plan.depth == 2) {
        launch<512, 2, 2>(data, rows, stride_vec, nvec, plan.splits, chunk, sink, s);
    } else {
        return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Sustained bf16 MFMA rate on operand data: grid workgroups of 256 threads (two per CU), each
// wave running iters x 16 MFMAs of 32x32x16 (32768 FLOP each) on fragments read from a (a_bytes)
// and b (b_bytes), both 16-byte aligned device arrays of at least 16 bytes.  sink: 4096 floats,
// clock: 2 uint64 (device; shader cycles and 100 MHz ticks of wave 0 of workgroup 0).  Returns
// 0, or -1 on bad arguments (nothing launched).
int traj_floor_mfma_rate(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes, int32_t grid, int32_t iters,
                         float* sink, uint64_t* clock, void* stream) {
    if (a == nullptr || b == nullptr || sink == nullptr || clock == nullptr || a_bytes < 16 || b_bytes < 16 ||
        grid < 1 || iters < 1)
        return -1;
    if (((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b)) & 15u) != 0) return -1;
    hipLaunchKernelGGL(mfma_rate_kernel, dim3(grid), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                       static_cast<const u32x4*>(a), a_bytes / 16, static_cast<const u32x4*>(b), b_bytes / 16, iters,
                       sink, clock);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // extern "C"
