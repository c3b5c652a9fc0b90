// libtrajfloor: the streaming-read floor of the logit pass, a measurement aid (not part of the
// verification step and not declared in the library's C ABI).
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

}  // extern "C"
