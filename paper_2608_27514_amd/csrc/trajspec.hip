// libtrajspec: C ABI of the gfx950 trajectory-verification step (see include/traj_spec.h).
// One translation unit: the kernels live in the headers included below.
#include <hip/hip_runtime.h>

#include <cmath>
#include <algorithm>
#include <climits>
#include <cstdint>
#include <mutex>

#include "../../include/traj_spec.h"
#include "accept.hpp"
#include "common.hpp"
#include "conf_topk.hpp"
#include "gemm.hpp"
#include "interblock.hpp"
#include "layer.hpp"
#include "tree.hpp"
#include "verify_attn.hpp"
#include "verify_attn16.hpp"

// Fixed device scratch of traj_confidence_topk_noalloc: the split records of short batches
// (at most TRAJ_TOPK_SCRATCH_BYTES).  Host code must not pass this name to a kernel or a copy: on
// the host it is only a handle; the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[TRAJ_TOPK_SCRATCH_BYTES];

namespace {

using namespace trajspec;

// Device address of `scratch` on the current device, looked up once per device.
constexpr int kScratchMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kScratchMaxDevices];

traj_status device_scratch(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchMaxDevices) return TRAJ_E_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return TRAJ_E_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return TRAJ_OK;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline traj_status launched() { return hipGetLastError() == hipSuccess ? TRAJ_OK : TRAJ_E_HIP; }

// ------------------------------------------------------------------ attention
traj_status check_attn(const traj_attn_shape* sh) {
    if (sh->B < 1 || sh->N < 1 || sh->L < 1 || sh->Hq < 1 || sh->Hkv < 1 || sh->S < 0) return TRAJ_E_SHAPE;
    if (sh->N > 64) return TRAJ_E_SHAPE;
    if (sh->Hq % sh->Hkv != 0) return TRAJ_E_SHAPE;
    if (sh->D != 64 && sh->D != 128) return TRAJ_E_UNSUPPORTED;
    if (!(sh->scale == sh->scale) || std::isinf(sh->scale)) return TRAJ_E_ARG;
    // flattened element counts must fit the kernels' 64-bit offsets and 32-bit row math
    const int64_t rows_per_group = (int64_t)(sh->Hq / sh->Hkv) * sh->N * sh->L;
    if (rows_per_group > (int64_t)1 << 30) return TRAJ_E_SHAPE;
    if ((int64_t)sh->S * sh->Hkv * sh->D > ((int64_t)1 << 40)) return TRAJ_E_SHAPE;
    // one sequence's cache slice is addressed through 32-bit buffer offsets
    if ((int64_t)sh->S * sh->Hkv * sh->D * 2 >= ((int64_t)1 << 31)) return TRAJ_E_UNSUPPORTED;
    return TRAJ_OK;
}

// Compute units of the current device (0 when the query fails).
int device_cu_count() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

// p describes the 32-row launch (4 waves x 32 rows per workgroup).  A grid that still has at
// most one workgroup per CU with 16-row waves (4 waves x 16 rows per workgroup, twice the
// workgroups) runs that way: each wave's chain of steps is half as long.  Larger grids keep
// 32-row waves: with two 16-row workgroups per CU the doubled LDS fragment reads and stage loads
// per MFMA cost more than the second wave per SIMD gains.
template <int D>
traj_status launch_attn(AttnParams p, hipStream_t st) {
    const int wg16 = (p.rows_per_group + kAttnWaves * 16 - 1) / (kAttnWaves * 16);
    const int64_t nwg16 = (int64_t)p.B * p.Hkv * wg16;
    if (nwg16 <= device_cu_count()) {
        p.wg_per_group = wg16;
        p.num_wg = (int)nwg16;
        hipLaunchKernelGGL(verify_attn16_kernel<D>, dim3(p.num_wg), dim3(kAttnThreads), 0, st, p);
    } else {
        hipLaunchKernelGGL(verify_attn_kernel<D>, dim3(p.num_wg), dim3(kAttnThreads), 0, st, p);
    }
    return launched();
}

// ------------------------------------------------------------------ confidence / top-k
int vec_of(int32_t dtype) { return dtype == TRAJ_BF16 ? 8 : 4; }
int size_of(int32_t dtype) { return dtype == TRAJ_BF16 ? 2 : 4; }

traj_status check_logits(const traj_logits_shape* sh, int32_t k) {
    if (sh->dtype != TRAJ_BF16 && sh->dtype != TRAJ_F32) return TRAJ_E_DTYPE;
    if (sh->rows < 0 || sh->vocab < 1 || sh->vocab >= ((int64_t)1 << 31)) return TRAJ_E_SHAPE;
    if (sh->row_stride < sh->vocab) return TRAJ_E_SHAPE;
    if (sh->rows >= ((int64_t)1 << 31) / 64) return TRAJ_E_SHAPE;
    if (k < 1 || k > 8 || k > sh->vocab) return TRAJ_E_ARG;
    return TRAJ_OK;
}

template <typename T, int K, int THREADS, int U, int DEPTH, bool VECTOR>
void launch_conf_kernel(const T* lg, const traj_logits_shape* sh, int k, const TopkPlan& plan, float* conf,
                        int32_t* idx, float* partial, hipStream_t st) {
    const dim3 grid((unsigned)(sh->rows * plan.splits));
    hipLaunchKernelGGL((conf_topk_kernel<T, K, THREADS, U, DEPTH, VECTOR>), grid, dim3(THREADS), 0, st, lg,
                       sh->row_stride, (int)sh->vocab, k, plan.splits, plan.chunk, conf, idx, partial);
}

// The plan's split records go to `ws` (at least traj_confidence_topk_workspace_size() bytes);
// without one the rows run unsplit.
template <typename T, int K>
traj_status launch_topk_k(const void* logits, const traj_logits_shape* sh, int k, float* conf, int32_t* idx,
                          void* ws, size_t ws_bytes, hipStream_t st) {
    const bool vector_ok = aligned16(logits) && ((sh->row_stride * (int64_t)sizeof(T)) % 16 == 0);
    TopkPlan plan = plan_conf_topk(sh->rows, sh->vocab, VecOf<T>::n);
    const size_t need = (size_t)sh->rows * plan.splits * kTopkRecord * sizeof(float);
    if (plan.splits > 1 && (ws == nullptr || ws_bytes < need || !aligned16(ws))) {
        plan.splits = 1;
        plan.chunk = (int)sh->vocab;
    }
    if (sh->rows == 0) return TRAJ_OK;
    float* partial = plan.splits > 1 ? static_cast<float*>(ws) : nullptr;
    const T* lg = static_cast<const T*>(logits);
    if (!vector_ok) {
        launch_conf_kernel<T, K, 256, 1, 1, false>(lg, sh, k, plan, conf, idx, partial, st);
    } else if (plan.threads == 64) {
        launch_conf_kernel<T, K, 64, 2, 3, true>(lg, sh, k, plan, conf, idx, partial, st);
    } else if (plan.threads == 256) {
        launch_conf_kernel<T, K, 256, 2, 2, true>(lg, sh, k, plan, conf, idx, partial, st);
    } else if (plan.unroll == 4) {
        launch_conf_kernel<T, K, 512, 4, 2, true>(lg, sh, k, plan, conf, idx, partial, st);
    } else {
        launch_conf_kernel<T, K, 512, 2, 2, true>(lg, sh, k, plan, conf, idx, partial, st);
    }
    if (plan.splits > 1) {
        hipLaunchKernelGGL((conf_topk_merge_kernel<K>), dim3((unsigned)sh->rows), dim3(64), 0, st, partial,
                           (int)sh->rows, plan.splits, k, conf, idx);
    }
    return launched();
}

template <typename T>
traj_status launch_topk(const void* logits, const traj_logits_shape* sh, int k, float* conf, int32_t* idx,
                        void* ws, size_t ws_bytes, hipStream_t st) {
    switch (k) {
        case 1: return launch_topk_k<T, 1>(logits, sh, k, conf, idx, ws, ws_bytes, st);
        case 2: return launch_topk_k<T, 2>(logits, sh, k, conf, idx, ws, ws_bytes, st);
        case 3:
        case 4: return launch_topk_k<T, 4>(logits, sh, k, conf, idx, ws, ws_bytes, st);
        default: return launch_topk_k<T, 8>(logits, sh, k, conf, idx, ws, ws_bytes, st);
    }
}

// ------------------------------------------------------------------ verification layer
// Split-K for grids of 128 x 128 tiles that leave CUs idle: up to kGemmMaxSplits k ranges of
// at least kGemmMinSplitK each, so that tiles x splits stays within one workgroup per CU.
constexpr int kGemmMaxSplits = 8;
constexpr int64_t kGemmMinSplitK = 512;

struct GemmSplit {
    int splits;
    int k_split;
};

GemmSplit plan_split(int64_t M, int64_t N, int64_t K) {
    const int64_t big = ((M + kG2BM - 1) / kG2BM) * ((N + kG2BN - 1) / kG2BN);
    const int64_t tiles = ((M + kGemmBM - 1) / kGemmBM) * ((N + kGemmBN - 1) / kGemmBN);
    if (big >= kGemmBigGridMin || tiles >= 256) return {1, 0};
    int64_t S = std::min<int64_t>(256 / tiles, kGemmMaxSplits);
    while (S > 1 && K / S < kGemmMinSplitK) --S;
    if (S <= 1) return {1, 0};
    const int64_t k_split = ((K + S - 1) / S + kGemmBK - 1) / kGemmBK * kGemmBK;
    return {(int)((K + k_split - 1) / k_split), (int)k_split};
}

// fp32 partial products of a split GEMM (0 when the shape is not split)
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M < 1 || N < 8 || K < 8 || K > kGemmMaxK || N > kGemmMaxN) return 0;
    const GemmSplit sp = plan_split(M, N, K);
    return sp.splits > 1 ? (size_t)sp.splits * (size_t)M * (size_t)N * sizeof(float) : 0;
}

// D[M,N] = A[M,K] W[K,N] (+ D when accumulate), bf16 row-major, fp32 accumulation.  `ws` (may
// be null) holds the split-K partials when the shape is split and it is large enough.
traj_status gemm(const uint16_t* A, const uint16_t* W, uint16_t* D, int64_t M, int64_t N, int64_t K, bool accumulate,
                 void* ws, size_t ws_bytes, hipStream_t st) {
    if (M < 1 || N < 8 || K < 8 || N % 8 != 0 || K % 8 != 0) return TRAJ_E_SHAPE;
    if (M > INT_MAX - kG2BM) return TRAJ_E_SHAPE;
    if (K > kGemmMaxK || N > kGemmMaxN) return TRAJ_E_UNSUPPORTED;  // 32-bit buffer offsets
    if (!aligned16(A) || !aligned16(W) || !aligned16(D)) return TRAJ_E_SHAPE;
    // 256 x 256 tiles when they alone fill the chip, else 128 x 128 tiles with the stage ring
    const int64_t big_m = (M + kG2BM - 1) / kG2BM, big_n = (N + kG2BN - 1) / kG2BN;
    if (big_m * big_n >= kGemmBigGridMin) {
        const GemmParams p{A, W, D, (int)M, (int)N, (int)K, (int)big_m, (int)big_n, nullptr, 0};
        const dim3 grid((unsigned)(big_m * big_n));
        if (accumulate)
            hipLaunchKernelGGL((gemm_tile256_kernel<true>), grid, dim3(kG2Threads), 0, st, p);
        else
            hipLaunchKernelGGL((gemm_tile256_kernel<false>), grid, dim3(kG2Threads), 0, st, p);
        return launched();
    }
    const int64_t tiles_m = (M + kGemmBM - 1) / kGemmBM, tiles_n = (N + kGemmBN - 1) / kGemmBN;
    const dim3 grid((unsigned)(tiles_m * tiles_n));  // fewer than 4 x 256 tiles
    const GemmSplit sp = plan_split(M, N, K);
    const size_t need = gemm_workspace_bytes(M, N, K);
    if (sp.splits > 1 && ws != nullptr && ws_bytes >= need && aligned16(ws)) {
        const GemmParams p{A, W, D, (int)M, (int)N, (int)K, (int)tiles_m, (int)tiles_n, static_cast<float*>(ws),
                           sp.k_split};
        hipLaunchKernelGGL((gemm_ring128_kernel<false, true>), dim3(grid.x, (unsigned)sp.splits), dim3(kGemmThreads),
                           0, st, p);
        traj_status rs = launched();
        if (rs != TRAJ_OK) return rs;
        const int64_t chunks = M * N / 8;
        const dim3 rgrid((unsigned)std::min<int64_t>((chunks + 255) / 256, 4096));
        if (accumulate)
            hipLaunchKernelGGL((gemm_split_reduce_kernel<true>), rgrid, dim3(256), 0, st,
                               static_cast<const float*>(ws), sp.splits, D, (int)M, (int)N);
        else
            hipLaunchKernelGGL((gemm_split_reduce_kernel<false>), rgrid, dim3(256), 0, st,
                               static_cast<const float*>(ws), sp.splits, D, (int)M, (int)N);
        return launched();
    }
    const GemmParams p{A, W, D, (int)M, (int)N, (int)K, (int)tiles_m, (int)tiles_n, nullptr, 0};
    if (accumulate)
        hipLaunchKernelGGL((gemm_ring128_kernel<true, false>), grid, dim3(kGemmThreads), 0, st, p);
    else
        hipLaunchKernelGGL((gemm_ring128_kernel<false, false>), grid, dim3(kGemmThreads), 0, st, p);
    return launched();
}

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

struct LayerPlan {
    size_t xn, qkv, q, kd, vd, a, gu, act, split, split_bytes, total;
};

LayerPlan plan_layer(const traj_attn_shape* sh, const traj_layer_dims* dm) {
    const size_t T = (size_t)sh->B * sh->N * sh->L;
    LayerPlan p{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align256(bytes);
        return at;
    };
    p.xn = take(T * dm->hidden * 2);
    p.qkv = take(T * (size_t)(sh->Hq + 2 * sh->Hkv) * sh->D * 2);
    p.q = take(T * (size_t)sh->Hq * sh->D * 2);
    p.kd = take(T * (size_t)sh->Hkv * sh->D * 2);
    p.vd = take(T * (size_t)sh->Hkv * sh->D * 2);
    p.a = take(T * (size_t)sh->Hq * sh->D * 2);
    p.gu = take(T * 2 * (size_t)dm->inter * 2);
    p.act = take(T * (size_t)dm->inter * 2);
    const int64_t hid = dm->hidden, qkv_w = (int64_t)(sh->Hq + 2 * sh->Hkv) * sh->D;
    p.split_bytes = std::max(std::max(gemm_workspace_bytes(T, qkv_w, hid), gemm_workspace_bytes(T, hid, (int64_t)sh->Hq * sh->D)),
                             std::max(gemm_workspace_bytes(T, 2 * (int64_t)dm->inter, hid),
                                      gemm_workspace_bytes(T, hid, dm->inter)));
    p.split = take(p.split_bytes);
    p.total = off;
    return p;
}

traj_status check_layer(const traj_attn_shape* sh, const traj_layer_dims* dm) {
    if (sh == nullptr || dm == nullptr) return TRAJ_E_NULL;
    const traj_status st = check_attn(sh);
    if (st != TRAJ_OK) return st;
    if (dm->hidden != sh->Hq * sh->D || dm->hidden % 8 != 0 || dm->inter < 8 || dm->inter % 8 != 0) return TRAJ_E_SHAPE;
    if (!(dm->rms_eps >= 0.f) || !(dm->rope_theta > 0.f)) return TRAJ_E_ARG;
    return TRAJ_OK;
}

traj_status check_weights(const void* x, const traj_layer_weights* w) {
    if (w == nullptr || w->attn_norm == nullptr || w->w_qkv == nullptr || w->w_o == nullptr ||
        w->mlp_norm == nullptr || w->w_gate_up == nullptr || w->w_down == nullptr)
        return TRAJ_E_NULL;
    if (!aligned16(x) || !aligned16(w->attn_norm) || !aligned16(w->mlp_norm) || !aligned16(w->w_qkv) ||
        !aligned16(w->w_o) || !aligned16(w->w_gate_up) || !aligned16(w->w_down))
        return TRAJ_E_SHAPE;
    return TRAJ_OK;
}

// The refresh's layer runs over B whole sequences of T = S + L tokens; `as` receives the
// equivalent attention shape (one "draft" of T tokens, the sequence's own K / V as its cache).
traj_status check_refresh(const traj_refresh_shape* sh, const traj_layer_dims* dm, traj_attn_shape* as) {
    if (sh == nullptr || dm == nullptr) return TRAJ_E_NULL;
    if (sh->B < 1 || sh->S < 0 || sh->L < 1 || (int64_t)sh->S + sh->L > 0x7fffffff / 2) return TRAJ_E_SHAPE;
    *as = traj_attn_shape{sh->B, 1, sh->S + sh->L, sh->Hq, sh->Hkv, sh->D, sh->S + sh->L, sh->scale};
    return check_layer(as, dm);
}

// Cache-only attention: every query row of q [B, T, Hq, D] attends to the S keys of k / v
// [B, S, Hkv, D] (the attention kernel with empty draft visible sets, N = 1, L = T).
traj_status attn_cache_only(const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* out, int B, int T,
                            int S, int Hq, int Hkv, int D, float scale_in, hipStream_t s) {
    const traj_attn_shape sh{B, 1, T, Hq, Hkv, D, S, scale_in};
    const traj_status st = check_attn(&sh);
    if (st != TRAJ_OK) return st;
    AttnParams p{};
    p.q = q;
    p.kc = k;
    p.vc = v;
    p.kd = k;  // never read: no draft is visible
    p.vd = v;
    p.parent = nullptr;
    p.peers = nullptr;
    p.out = out;
    p.B = B;
    p.N = 1;
    p.L = T;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.S = S;
    p.group = Hq / Hkv;
    p.rows_per_group = p.group * T;
    const int rb = (p.rows_per_group + 31) / 32;
    p.wg_per_group = (rb + kAttnWaves - 1) / kAttnWaves;
    const int64_t nwg = (int64_t)B * Hkv * p.wg_per_group;
    if (nwg > 0x7fffffff) return TRAJ_E_SHAPE;
    p.num_wg = (int)nwg;
    const float scale = scale_in > 0.f ? scale_in : 1.0f / std::sqrt((float)D);
    p.scale_log2 = scale * 1.4426950408889634f;
    p.drafts_visible = 0;
    return D == 128 ? launch_attn<128>(p, s) : launch_attn<64>(p, s);
}

// One pre-norm decoder layer over T packed tokens (x [T, hidden], updated in place).  The rotary
// position of token t is pos0[t / rope_nl] + t % rope_l (pos0 may be null = 0); `attend` runs
// between the rotary split and the O projection: it reads the q / k / v rows and writes the
// attention output a [T, Hq D].
template <typename Attend>
traj_status run_layer(uint16_t* xs, const traj_layer_weights* w, const traj_layer_dims* dims, int64_t T, int Hq,
                      int Hkv, int D, const int32_t* pos0, int rope_nl, int rope_l, const LayerPlan& plan, char* ws,
                      hipStream_t s, Attend attend) {
    auto buf = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
    const int hidden = dims->hidden, inter = dims->inter;
    const int qkv_w = (Hq + 2 * Hkv) * D;
    void* split = ws + plan.split;
    const size_t split_bytes = plan.split_bytes;
    traj_status st;
    // attention block
    hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)T), dim3(kLayerThreads), 0, s, xs,
                       static_cast<const uint16_t*>(w->attn_norm), buf(plan.xn), hidden, dims->rms_eps);
    if ((st = launched()) != TRAJ_OK) return st;
    if ((st = gemm(buf(plan.xn), static_cast<const uint16_t*>(w->w_qkv), buf(plan.qkv), T, qkv_w, hidden, false, split,
                   split_bytes, s)) != TRAJ_OK)
        return st;
    hipLaunchKernelGGL(rope_split_kernel, dim3((unsigned)T), dim3(kLayerThreads), 0, s, buf(plan.qkv), pos0,
                       buf(plan.q), buf(plan.kd), buf(plan.vd), rope_nl, rope_l, Hq, Hkv, D,
                       std::log2(dims->rope_theta));
    if ((st = launched()) != TRAJ_OK) return st;
    if ((st = attend(buf(plan.q), buf(plan.kd), buf(plan.vd), buf(plan.a))) != TRAJ_OK) return st;
    if ((st = gemm(buf(plan.a), static_cast<const uint16_t*>(w->w_o), xs, T, hidden, (int64_t)Hq * D, true, split,
                   split_bytes, s)) != TRAJ_OK)
        return st;
    // MLP block
    hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)T), dim3(kLayerThreads), 0, s, xs,
                       static_cast<const uint16_t*>(w->mlp_norm), buf(plan.xn), hidden, dims->rms_eps);
    if ((st = launched()) != TRAJ_OK) return st;
    if ((st = gemm(buf(plan.xn), static_cast<const uint16_t*>(w->w_gate_up), buf(plan.gu), T, 2 * (int64_t)inter, hidden,
                   false, split, split_bytes, s)) != TRAJ_OK)
        return st;
    const int64_t chunks = T * (inter / 8);
    hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)std::min<int64_t>((chunks + kLayerThreads - 1) / kLayerThreads, 16384)),
                       dim3(kLayerThreads), 0, s, buf(plan.gu), buf(plan.act), T, inter);
    if ((st = launched()) != TRAJ_OK) return st;
    return gemm(buf(plan.act), static_cast<const uint16_t*>(w->w_down), xs, T, hidden, inter, true, split, split_bytes, s);
}

}  // namespace

extern "C" {

size_t traj_verify_attn_workspace_size(const traj_attn_shape* shape) {
    (void)shape;
    return 0;  // the attention kernels use no scratch memory; the workspace argument is reserved
}

traj_status traj_verify_attn(const void* q, const void* k_cache, const void* v_cache, const void* k_draft,
                             const void* v_draft, const int32_t* draft_parent, void* out,
                             const traj_attn_shape* shape, void* workspace, size_t workspace_bytes, void* stream) {
    return traj_verify_attn_peers(q, k_cache, v_cache, k_draft, v_draft, draft_parent, nullptr, out, shape,
                                  workspace, workspace_bytes, stream);
}

traj_status traj_verify_attn_peers(const void* q, const void* k_cache, const void* v_cache, const void* k_draft,
                                   const void* v_draft, const int32_t* draft_parent, const uint64_t* draft_peers,
                                   void* out, const traj_attn_shape* shape, void* workspace, size_t workspace_bytes,
                                   void* stream) {
    (void)workspace;
    (void)workspace_bytes;
    if (shape == nullptr || q == nullptr || k_draft == nullptr || v_draft == nullptr || draft_parent == nullptr ||
        out == nullptr)
        return TRAJ_E_NULL;
    if (shape->S > 0 && (k_cache == nullptr || v_cache == nullptr)) return TRAJ_E_NULL;
    traj_status st = check_attn(shape);
    if (st != TRAJ_OK) return st;
    if (!aligned16(q) || !aligned16(k_draft) || !aligned16(v_draft) || !aligned16(out) ||
        (shape->S > 0 && (!aligned16(k_cache) || !aligned16(v_cache))))
        return TRAJ_E_SHAPE;

    AttnParams p{};
    p.q = static_cast<const uint16_t*>(q);
    p.kc = static_cast<const uint16_t*>(k_cache);
    p.vc = static_cast<const uint16_t*>(v_cache);
    p.kd = static_cast<const uint16_t*>(k_draft);
    p.vd = static_cast<const uint16_t*>(v_draft);
    p.parent = draft_parent;
    p.peers = draft_peers;
    p.out = static_cast<uint16_t*>(out);
    p.B = shape->B;
    p.N = shape->N;
    p.L = shape->L;
    p.Hq = shape->Hq;
    p.Hkv = shape->Hkv;
    p.S = shape->S;
    p.group = shape->Hq / shape->Hkv;
    p.rows_per_group = p.group * p.N * p.L;
    const int rb = (p.rows_per_group + 31) / 32;
    p.wg_per_group = (rb + kAttnWaves - 1) / kAttnWaves;
    const int64_t nwg = (int64_t)p.B * p.Hkv * p.wg_per_group;
    if (nwg > 0x7fffffff) return TRAJ_E_SHAPE;
    p.num_wg = (int)nwg;
    const float scale = shape->scale > 0.f ? shape->scale : 1.0f / std::sqrt((float)shape->D);
    p.scale_log2 = scale * 1.4426950408889634f;
    p.drafts_visible = 1;
    hipStream_t s = as_stream(stream);
    return shape->D == 128 ? launch_attn<128>(p, s) : launch_attn<64>(p, s);
}

size_t traj_confidence_topk_workspace_size(const traj_logits_shape* shape, int32_t k) {
    if (shape == nullptr || check_logits(shape, k) != TRAJ_OK) return 0;
    const TopkPlan plan = plan_conf_topk(shape->rows, shape->vocab, vec_of(shape->dtype));
    if (plan.splits <= 1) return 0;
    return (size_t)shape->rows * plan.splits * kTopkRecord * sizeof(float);
}

traj_status traj_confidence_topk(const void* logits, int32_t k, float* conf, int32_t* idx,
                                 const traj_logits_shape* shape, void* workspace, size_t workspace_bytes,
                                 void* stream) {
    if (shape == nullptr) return TRAJ_E_NULL;
    traj_status st = check_logits(shape, k);
    if (st != TRAJ_OK) return st;
    if (shape->rows == 0) return TRAJ_OK;  // nothing to do; pointers may be NULL
    if (logits == nullptr || conf == nullptr || idx == nullptr) return TRAJ_E_NULL;
    if (workspace != nullptr && !aligned16(workspace)) return TRAJ_E_WORKSPACE;
    const size_t need = traj_confidence_topk_workspace_size(shape, k);
    if (workspace != nullptr && workspace_bytes > 0 && workspace_bytes < need) return TRAJ_E_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (shape->dtype == TRAJ_BF16) return launch_topk<uint16_t>(logits, shape, k, conf, idx, workspace, workspace_bytes, s);
    return launch_topk<float>(logits, shape, k, conf, idx, workspace, workspace_bytes, s);
}

traj_status traj_confidence_topk_noalloc(const void* logits, int32_t k, float* conf, int32_t* idx,
                                         const traj_logits_shape* shape, void* stream) {
    if (shape == nullptr) return TRAJ_E_NULL;
    traj_status st = check_logits(shape, k);
    if (st != TRAJ_OK) return st;
    if (shape->rows == 0) return TRAJ_OK;
    if (logits == nullptr || conf == nullptr || idx == nullptr) return TRAJ_E_NULL;
    const size_t need = traj_confidence_topk_workspace_size(shape, k);
    if (need > (size_t)TRAJ_TOPK_SCRATCH_BYTES) return TRAJ_E_WORKSPACE;  // split records beyond the fixed scratch
    void* ws = nullptr;
    if (need > 0 && (st = device_scratch(&ws)) != TRAJ_OK) return st;
    hipStream_t s = as_stream(stream);
    if (shape->dtype == TRAJ_BF16) return launch_topk<uint16_t>(logits, shape, k, conf, idx, ws, need, s);
    return launch_topk<float>(logits, shape, k, conf, idx, ws, need, s);
}

traj_status traj_accept(const float* conf, const int32_t* idx, const traj_drafts* drafts, float threshold,
                        const traj_accepted* accepted, void* stream) {
    if (drafts == nullptr || accepted == nullptr || conf == nullptr || idx == nullptr) return TRAJ_E_NULL;
    if (drafts->tokens == nullptr || drafts->parent == nullptr || drafts->committed == nullptr ||
        drafts->conf0 == nullptr || drafts->idx0 == nullptr)
        return TRAJ_E_NULL;
    if (accepted->leaf == nullptr || accepted->on_path == nullptr || accepted->n_accepted == nullptr ||
        accepted->out_tokens == nullptr || accepted->hi == nullptr)
        return TRAJ_E_NULL;
    if (drafts->B < 1 || drafts->N < 1 || drafts->N > kMaxDrafts || drafts->L < 1 || drafts->L > kMaxBlock)
        return TRAJ_E_SHAPE;
    if (drafts->k < 1 || drafts->k > 8) return TRAJ_E_ARG;
    if (drafts->mode < TRAJ_MODE_EXACT || drafts->mode > TRAJ_MODE_TOPK) return TRAJ_E_ARG;
    if (drafts->traversal != TRAJ_GREEDY && drafts->traversal != TRAJ_LONGEST) return TRAJ_E_ARG;
    if (!(threshold == threshold)) return TRAJ_E_ARG;
    AcceptParams p{};
    p.conf = conf;
    p.idx = idx;
    p.tokens = drafts->tokens;
    p.parent = drafts->parent;
    p.committed = drafts->committed;
    p.conf0 = drafts->conf0;
    p.idx0 = drafts->idx0;
    p.leaf = accepted->leaf;
    p.on_path = accepted->on_path;
    p.n_accepted = accepted->n_accepted;
    p.out_tokens = accepted->out_tokens;
    p.hi = accepted->hi;
    p.B = drafts->B;
    p.N = drafts->N;
    p.L = drafts->L;
    p.k = drafts->k;
    p.mode = drafts->mode;
    p.traversal = drafts->traversal;
    p.tau = threshold;
    hipLaunchKernelGGL(accept_kernel, dim3(p.B), dim3(kAcceptThreads), 0, as_stream(stream), p);
    return launched();
}

traj_status traj_interblock_trigger(const int32_t* state, const float* conf, int32_t B, int32_t L, int32_t k,
                                    float threshold, uint8_t* trigger, float* c_cur, float* c_next, void* stream) {
    if (state == nullptr || conf == nullptr || trigger == nullptr) return TRAJ_E_NULL;
    if (B < 1 || L < 1 || L > kTriggerMaxBlock) return TRAJ_E_SHAPE;
    if (k < 1 || k > 8 || !(threshold == threshold)) return TRAJ_E_ARG;
    TriggerParams p{state, conf, trigger, c_cur, c_next, B, L, k, threshold};
    hipLaunchKernelGGL(interblock_trigger_kernel, dim3(B), dim3(64), 0, as_stream(stream), p);
    return launched();
}

traj_status traj_joint_peers(int32_t B, int32_t n_cur, int32_t n_next, const int32_t* root_cur,
                             const int32_t* root_next, uint64_t* peers, void* stream) {
    if (peers == nullptr) return TRAJ_E_NULL;
    if (B < 1 || n_cur < 1 || n_next < 1 || n_cur + n_next > 64) return TRAJ_E_SHAPE;
    const int64_t total = (int64_t)B * (n_cur + n_next);
    if (total > ((int64_t)1 << 31) - 256) return TRAJ_E_SHAPE;
    static_assert(kDevBadRoot == TRAJ_DEV_BAD_ROOT, "device status bit");
    const JointPeersParams p{root_cur, root_next, peers, B, n_cur, n_next};
    hipLaunchKernelGGL(joint_peers_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, as_stream(stream), p);
    return launched();
}

int32_t traj_tree_max_nodes(const traj_tree_shape* sh) {
    if (sh == nullptr || sh->B < 1 || sh->L < 1 || sh->L > kTreeMaxBlock || sh->k < 1 || sh->k > kTreeMaxK ||
        sh->branch < 1 || sh->branch > sh->k || sh->branch_deep < 1 || sh->branch_deep > sh->k || sh->width < 1 ||
        sh->depth < 0 || sh->n_prev < 0 || (sh->full != 0 && sh->full != 1))
        return -1;
    int64_t total = 1, cnt = 0;
    const int levels = sh->depth < sh->L ? sh->depth : sh->L;
    for (int l = 1; l <= levels; ++l) {
        const int64_t w = sh->full ? sh->width : (sh->width - l + 1 > 1 ? sh->width - l + 1 : 1);
        const int64_t gen = l == 1 ? sh->branch : cnt * sh->branch_deep;
        cnt = gen < w ? gen : w;
        total += cnt;
        if (total > 0x7fffffff) return -1;
    }
    return (int32_t)total;
}

traj_status traj_build_tree(const int32_t* state, const int32_t* leaf, const float* conf, const int32_t* idx,
                            const float* conf0, const int32_t* idx0, const traj_tree_shape* shape, float threshold,
                            int32_t* tokens, int32_t* parent, int32_t* n_nodes, float* score, float* conf_next,
                            int32_t* idx_next, void* stream) {
    if (shape == nullptr || state == nullptr || conf0 == nullptr || idx0 == nullptr || tokens == nullptr ||
        parent == nullptr || n_nodes == nullptr)
        return TRAJ_E_NULL;
    if (leaf != nullptr && shape->n_prev > 0 && (conf == nullptr || idx == nullptr)) return TRAJ_E_NULL;
    if ((conf_next == nullptr) != (idx_next == nullptr)) return TRAJ_E_NULL;
    if (shape->k < 1 || shape->k > kTreeMaxK || shape->branch < 1 || shape->branch > shape->k ||
        shape->branch_deep < 1 || shape->branch_deep > shape->k || (shape->full != 0 && shape->full != 1))
        return TRAJ_E_ARG;
    if (!(threshold == threshold)) return TRAJ_E_ARG;
    const int32_t need = traj_tree_max_nodes(shape);
    if (need < 0 || shape->n_max < need || shape->n_max > kTreeMaxNodes) return TRAJ_E_SHAPE;
    TreeParams p{};
    p.state = state;
    p.leaf = leaf;
    p.conf = conf;
    p.idx = idx;
    p.conf0 = conf0;
    p.idx0 = idx0;
    p.tokens = tokens;
    p.parent = parent;
    p.n_nodes = n_nodes;
    p.score = score;
    p.conf_next = conf_next;
    p.idx_next = idx_next;
    p.B = shape->B;
    p.L = shape->L;
    p.k = shape->k;
    p.n_prev = leaf != nullptr ? shape->n_prev : 0;
    p.width = shape->width;
    p.depth = shape->depth;
    p.branch = shape->branch;
    p.branch_deep = shape->branch_deep;
    p.full = shape->full;
    p.n_max = shape->n_max;
    p.tau = threshold;
    hipLaunchKernelGGL(build_tree_kernel, dim3(p.B), dim3(kTreeThreads), 0, as_stream(stream), p);
    return launched();
}

size_t traj_verify_layer_workspace_size(const traj_attn_shape* shape, const traj_layer_dims* dims) {
    if (check_layer(shape, dims) != TRAJ_OK) return 0;
    return plan_layer(shape, dims).total;
}

traj_status traj_verify_layer(void* x, const traj_layer_weights* w, const traj_layer_dims* dims, const void* k_cache,
                              const void* v_cache, const int32_t* draft_parent, const int32_t* pos0,
                              const traj_attn_shape* shape, void* workspace, size_t workspace_bytes, void* stream) {
    traj_status st = check_layer(shape, dims);
    if (st != TRAJ_OK) return st;
    if (x == nullptr || draft_parent == nullptr || workspace == nullptr) return TRAJ_E_NULL;
    if ((st = check_weights(x, w)) != TRAJ_OK) return st;
    if (shape->S > 0 && (k_cache == nullptr || v_cache == nullptr)) return TRAJ_E_NULL;
    const LayerPlan plan = plan_layer(shape, dims);
    if (workspace_bytes < plan.total || reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return TRAJ_E_WORKSPACE;
    const int64_t T = (int64_t)shape->B * shape->N * shape->L;
    // every draft's token p sits at position pos0[b] + p
    return run_layer(static_cast<uint16_t*>(x), w, dims, T, shape->Hq, shape->Hkv, shape->D, pos0,
                     shape->N * shape->L, shape->L, plan, static_cast<char*>(workspace), as_stream(stream),
                     [&](const uint16_t* q, const uint16_t* kd, const uint16_t* vd, uint16_t* a) {
                         return traj_verify_attn(q, k_cache, v_cache, kd, vd, draft_parent, a, shape, nullptr, 0, stream);
                     });
}

size_t traj_refresh_layer_workspace_size(const traj_refresh_shape* shape, const traj_layer_dims* dims) {
    traj_attn_shape as{};
    if (check_refresh(shape, dims, &as) != TRAJ_OK) return 0;
    return plan_layer(&as, dims).total;
}

traj_status traj_refresh_layer(void* x, const traj_layer_weights* w, const traj_layer_dims* dims,
                               const int32_t* block_start, void* k_cache, void* v_cache,
                               const traj_refresh_shape* shape, void* workspace, size_t workspace_bytes, void* stream) {
    traj_attn_shape as{};
    traj_status st = check_refresh(shape, dims, &as);
    if (st != TRAJ_OK) return st;
    if (x == nullptr || block_start == nullptr || workspace == nullptr) return TRAJ_E_NULL;
    if ((st = check_weights(x, w)) != TRAJ_OK) return st;
    if (shape->S > 0 && (k_cache == nullptr || v_cache == nullptr)) return TRAJ_E_NULL;
    if (shape->S > 0 && (!aligned16(k_cache) || !aligned16(v_cache))) return TRAJ_E_SHAPE;
    const LayerPlan plan = plan_layer(&as, dims);
    if (workspace_bytes < plan.total || reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return TRAJ_E_WORKSPACE;
    const int Tseq = shape->S + shape->L;
    const int64_t T = (int64_t)shape->B * Tseq;
    hipStream_t s = as_stream(stream);
    // positions 0 .. T - 1 of each sequence; attention over the sequence's own K / V (the
    // kernel's cache-only mode), after the rows outside the block have been copied to the cache
    return run_layer(static_cast<uint16_t*>(x), w, dims, T, shape->Hq, shape->Hkv, shape->D, nullptr, Tseq, Tseq,
                     plan, static_cast<char*>(workspace), s,
                     [&](const uint16_t* q, const uint16_t* kd, const uint16_t* vd, uint16_t* a) -> traj_status {
                         if (shape->S > 0) {
                             const int width = shape->Hkv * shape->D;
                             const int64_t chunks = (int64_t)shape->B * shape->S * (width / 8);
                             const unsigned grid = (unsigned)std::min<int64_t>((chunks + kLayerThreads - 1) / kLayerThreads, 8192);
                             hipLaunchKernelGGL(cache_gather_kernel, dim3(grid), dim3(kLayerThreads), 0, s, kd, vd,
                                                block_start, static_cast<uint16_t*>(k_cache),
                                                static_cast<uint16_t*>(v_cache), shape->B, shape->S, shape->L, width);
                             const traj_status gs = launched();
                             if (gs != TRAJ_OK) return gs;
                         }
                         return attn_cache_only(q, kd, vd, a, shape->B, Tseq, Tseq, shape->Hq, shape->Hkv, shape->D,
                                                shape->scale, s);
                     });
}

size_t traj_linear_workspace_size(int64_t M, int64_t K, int64_t N) { return gemm_workspace_bytes(M, N, K); }

traj_status traj_linear(const void* x, const void* w, void* y, int64_t M, int64_t K, int64_t N, int32_t accumulate,
                        void* workspace, size_t workspace_bytes, void* stream) {
    if (M < 0 || K < 8 || N < 8 || K % 8 != 0 || N % 8 != 0) return TRAJ_E_SHAPE;
    if (M == 0) return TRAJ_OK;
    if (x == nullptr || w == nullptr || y == nullptr) return TRAJ_E_NULL;
    if (workspace != nullptr && (workspace_bytes < gemm_workspace_bytes(M, N, K) || !aligned16(workspace)))
        return TRAJ_E_WORKSPACE;
    return gemm(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), static_cast<uint16_t*>(y), M, N, K,
                accumulate != 0, workspace, workspace_bytes, as_stream(stream));
}

const char* traj_status_string(int32_t status) {
    switch (status) {
        case TRAJ_OK: return "ok";
        case TRAJ_E_NULL: return "a required pointer is NULL";
        case TRAJ_E_SHAPE: return "a size is out of range, inconsistent or misaligned";
        case TRAJ_E_DTYPE: return "unknown element type";
        case TRAJ_E_UNSUPPORTED: return "supported by the ABI but not implemented (head_dim must be 64 or 128; one sequence's cache below 2 GiB)";
        case TRAJ_E_WORKSPACE: return "workspace too small or misaligned";
        case TRAJ_E_HIP: return "HIP runtime error";
        case TRAJ_E_ARG: return "an enumerated or scalar argument has an invalid value";
        default: return "unknown status";
    }
}

// TRAJ_SOURCE_DIGEST: sha256 of the sources and flags, stamped by the package's build script.
#ifndef TRAJ_SOURCE_DIGEST
#define TRAJ_SOURCE_DIGEST "unstamped"
#endif
const char* traj_version(void) { return "libtrajspec 0.2.0 gfx950 sources " TRAJ_SOURCE_DIGEST; }

traj_status traj_get_device_status(int32_t* host_flags, int32_t reset, void* stream) {
    if (host_flags == nullptr) return TRAJ_E_NULL;
    hipStream_t s = as_stream(stream);
    if (hipStreamSynchronize(s) != hipSuccess) return TRAJ_E_HIP;
    int32_t v = 0;
    if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_device_status), sizeof(v), 0, hipMemcpyDeviceToHost) != hipSuccess)
        return TRAJ_E_HIP;
    *host_flags = v;
    if (reset) {
        const int32_t zero = 0;
        if (hipMemcpyToSymbol(HIP_SYMBOL(g_device_status), &zero, sizeof(zero), 0, hipMemcpyHostToDevice) !=
            hipSuccess)
            return TRAJ_E_HIP;
    }
    return TRAJ_OK;
}

}  // extern "C"
