"""Benchmark of one trajectory-verification step on one MI355X.

A step is the whole hot path over one batch of synthetic input already resident in
HBM: trajectory-masked attention (traj_verify_attn), the confidence/top-k logit pass
(traj_confidence_topk) and acceptance (traj_accept), launched back to back on one
stream.  Metric: verified draft tokens per second = B*N*L / step time.

Default workload: "8b-batched" -- 16 sequences, 64 tree-structured drafts of 32
tokens each (3-ary, levels 3+9+27+25), 32 heads of dim 128, a 4096-token dual
cache (3584 prefix + 512 suffix), 32768 logit rows over a 126464-token vocabulary.
Other workloads: --workload 1..5 (see synthetic/workloads.py).

Prints ONE JSON line.  Timing: W warm-up steps, then K timed steps bracketed by
synchronisation; per-kernel durations come from HIP events recorded on the launch
stream around every call.  Small workloads rotate several input copies so that the
reads come from HBM rather than the 256 MB Infinity Cache.
"""

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import paper_2608_27514_amd as tsp  # noqa: E402
from synthetic import WORKLOADS, attention_inputs, decode_inputs, make_logits, seed_for, torch_dtype  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
MALL_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {
    "verify_attn": ("common.hpp", "verify_attn.hpp", "verify_attn16.hpp"),
    "confidence_topk": ("common.hpp", "conf_topk.hpp"),
}


def kernel_source_hash(kernel):
    """sha256 over the sources a kernel is built from (traffic figures are only valid for
    the exact code they were measured on)."""
    import hashlib
    h = hashlib.sha256()
    for fn in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2608_27514_amd", "csrc", fn), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE passes, or
    None when they are missing or were taken on different kernel code."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)[kernel][workload]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return rec["bytes_per_launch"]


def log(msg):
    """Progress on stderr (the result line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def depths(parent_row):
    out = []
    for n in range(len(parent_row)):
        d, j = 1, int(parent_row[n])
        while j != -1:
            d += 1
            j = int(parent_row[j])
        out.append(d)
    return out


def attn_flops(wl, parent):
    """Algorithmic FLOP: 4*L*D*(S + L*|anc*(i)|) per (sequence, head, draft)."""
    tot = 0
    for b in range(wl.B):
        for dep in depths(parent[b]):
            tot += 4 * wl.L * wl.D * (wl.S + wl.L * dep) * wl.Hq
    return tot


def attn_bytes(wl):
    """Each tensor read or written once: K/V cache, q, out, draft K/V (bf16)."""
    return 2 * wl.D * wl.B * (2 * wl.S * wl.Hkv + wl.N * wl.L * (2 * wl.Hq + 2 * wl.Hkv))


def logit_bytes(wl):
    elem = 2 if wl.logits_dtype == "bf16" else 4
    return wl.rows * wl.V * elem + wl.rows * wl.k * 8


class StepInputs:
    def __init__(self, wl, seed, tau, dev):
        self.wl = wl
        self.d = decode_inputs(wl, seed, tau=tau)
        self.q, self.kc, self.vc, self.kd, self.vd = attention_inputs(wl, seed, device=dev)
        self.parent = torch.as_tensor(self.d["parent"], dtype=torch.int32, device=dev)
        self.logits = make_logits(self.d["row_margin"], self.d["row_top"], wl.V, torch_dtype(wl.logits_dtype),
                                  seed + 17, device=dev, row_chunk=2048)
        self.tokens = torch.as_tensor(self.d["tokens"], device=dev)
        self.committed = torch.as_tensor(self.d["committed"], device=dev)
        self.conf0 = torch.as_tensor(self.d["conf0"], device=dev)
        self.idx0 = torch.as_tensor(self.d["idx0"], device=dev)

    def nbytes(self):
        ts = [self.q, self.kc, self.vc, self.kd, self.vd, self.logits]
        return sum(t.numel() * t.element_size() for t in ts)

    def replant(self, seed, tau):
        """Re-plant tree tokens and logits for another threshold (attention unchanged)."""
        wl = self.wl
        dev = self.q.device
        self.d = decode_inputs(wl, seed, tau=tau, parent=self.d["parent"], rank=self.d["rank"],
                               level=self.d["level"])
        make_logits(self.d["row_margin"], self.d["row_top"], wl.V, torch_dtype(wl.logits_dtype), seed + 17,
                    device=dev, row_chunk=2048, out=self.logits)
        self.tokens = torch.as_tensor(self.d["tokens"], device=dev)
        self.committed = torch.as_tensor(self.d["committed"], device=dev)
        self.conf0 = torch.as_tensor(self.d["conf0"], device=dev)
        self.idx0 = torch.as_tensor(self.d["idx0"], device=dev)


class Buffers:
    def __init__(self, wl, dev, logits):
        self.out = torch.empty((wl.B, wl.N, wl.L, wl.Hq, wl.D), dtype=torch.bfloat16, device=dev)
        self.conf = torch.empty((wl.rows, wl.k), dtype=torch.float32, device=dev)
        self.idx = torch.empty((wl.rows, wl.k), dtype=torch.int32, device=dev)
        n = tsp.confidence_topk_workspace_size(logits, wl.k)
        self.ws = torch.empty(max(n, 16), dtype=torch.uint8, device=dev) if n > 0 else None
        self.acc = {
            "leaf": torch.empty(wl.B, dtype=torch.int32, device=dev),
            "on_path": torch.empty((wl.B, wl.N), dtype=torch.uint8, device=dev),
            "n_accepted": torch.empty(wl.B, dtype=torch.int32, device=dev),
            "out_tokens": torch.empty((wl.B, wl.L), dtype=torch.int32, device=dev),
            "hi": torch.empty((wl.B, wl.N, wl.L), dtype=torch.uint8, device=dev),
        }


def run_step(x, buf, tau, stream, ev=None):
    if ev is not None:
        ev[0].record(stream)
    tsp.verify_attn(x.q, x.kc, x.vc, x.kd, x.vd, x.parent, out=buf.out, stream=stream)
    if ev is not None:
        ev[1].record(stream)
    tsp.confidence_topk(x.logits, x.wl.k, conf=buf.conf, idx=buf.idx, workspace=buf.ws, stream=stream)
    if ev is not None:
        ev[2].record(stream)
    tsp.accept(buf.conf, buf.idx, x.tokens, x.parent, x.committed, x.conf0, x.idx0, tau, out=buf.acc,
               stream=stream)
    if ev is not None:
        ev[3].record(stream)


def cpu_workers():
    """Host threads for the oracle: the process's CPU affinity set, capped at the 16-core
    share of one GPU on the shared hosts this runs on."""
    return max(1, min(len(os.sched_getaffinity(0)), 16))


def cpu_baseline(x, buf, wl, tau, n_seq):
    """The oracle, as it stands, on the first n_seq sequences of the same inputs, run on a pool
    of host threads (one BLAS thread each; numpy releases the interpreter lock in its array
    kernels): attention one query head per task, the logit pass in equal contiguous row ranges,
    acceptance as one call.  Also checks the GPU outputs of those sequences against it."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    from threadpoolctl import threadpool_limits
    workers = cpu_workers()
    sl = slice(0, n_seq)
    f64 = lambda t: t[sl].float().cpu().numpy().astype(np.float64)  # noqa: E731
    q, kc, vc, kd, vd = (f64(t) for t in (x.q, x.kc, x.vc, x.kd, x.vd))
    rows = n_seq * wl.N * wl.L
    lg = x.logits[:rows].float().cpu().numpy()
    parent = x.d["parent"][sl]
    G = wl.Hq // wl.Hkv
    ref_out = np.empty(q.shape, dtype=np.float64)

    def attn_head(h):
        g = h // G
        ref_out[:, :, :, h:h + 1] = oracle.verify_attention(q[:, :, :, h:h + 1], kc[:, :, g:g + 1], vc[:, :, g:g + 1],
                                                            kd[:, :, :, g:g + 1], vd[:, :, :, g:g + 1], parent)

    bounds = np.linspace(0, rows, workers + 1).astype(int)
    parts = [None] * workers

    def conf_part(i):
        parts[i] = oracle.confidence_topk(lg[bounds[i]:bounds[i + 1]], wl.k)

    with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
        t0 = time.perf_counter()
        list(ex.map(attn_head, range(wl.Hq)))
        t1 = time.perf_counter()
        list(ex.map(conf_part, range(workers)))
        rc = np.concatenate([p_[0] for p_ in parts])
        ri = np.concatenate([p_[1] for p_ in parts])
        t2 = time.perf_counter()
        shp = (n_seq, wl.N, wl.L, wl.k)
        ref_acc = oracle.accept_batch(x.d["tokens"][sl], parent, x.d["committed"][sl],
                                      x.d["conf0"][sl].astype(np.float64), x.d["idx0"][sl], rc.reshape(shp),
                                      ri.reshape(shp), tau)
        t3 = time.perf_counter()
    # sample parity of the timed GPU outputs
    g_out = buf.out[sl].float().cpu().numpy()
    attn_ok = bool((np.abs(g_out - ref_out) <= 2e-3 + 2e-2 * np.abs(ref_out)).all())
    idx_ok = bool(np.array_equal(buf.idx[:rows].cpu().numpy(), ri))
    conf_err = float(np.abs(buf.conf[:rows].cpu().numpy() - rc).max())
    leaf_ok = bool(np.array_equal(buf.acc["leaf"][sl].cpu().numpy(), ref_acc["leaf"]))
    fragile = sum(int(oracle.fragile_states(x.d["tokens"][b], x.d["committed"][b], x.d["conf0"][b],
                                            rc.reshape(shp)[b], tau).any()) for b in range(n_seq))
    total = t3 - t0
    return {
        "value": rows / total,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": (f"first {n_seq} of {wl.B} sequences ({rows} draft tokens: all {wl.Hq} heads of "
                   f"attention, {rows} logit rows, acceptance); fp64 numpy on a pool of {workers} host threads "
                   f"(affinity set {len(os.sched_getaffinity(0))} CPUs), one BLAS thread each"),
        "pool": {"threads": workers, "attention_tasks": wl.Hq, "logit_tasks": workers, "accept_tasks": 1},
        "seconds": {"attention": t1 - t0, "confidence_topk": t2 - t1, "accept": t3 - t2, "total": total},
        "sample_parity": {"attention_within_tol": attn_ok, "topk_idx_exact": idx_ok,
                          "conf_max_abs_err": conf_err, "leaf_exact": leaf_ok,
                          "fragile_sequences_excluded": fragile},
    }


def sharp_sample_parity(wl, parent, stream, b=None, h=None):
    """The timed attention launch (full batch and heads, the workload's parent array) on sharp
    inputs (q ~ 3 N(0,1), k, v ~ N(0,1)), where a wrong mask moves outputs far outside the
    tolerance: one sampled (sequence, head) slice is checked against the oracle, and the same slice
    must fail against oracles with a wrong mask (ancestors dropped; siblings chained)."""
    import oracle
    from synthetic import attention_inputs as ai
    seed = seed_for(wl.cid, salt=3)
    q, kc, vc, kd, vd = ai(wl, seed, "sharp", device="cuda")
    out = tsp.verify_attn(q, kc, vc, kd, vd, torch.as_tensor(parent, dtype=torch.int32, device="cuda"),
                          stream=stream)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed)
    b = int(rng.integers(wl.B)) if b is None else b
    h = int(rng.integers(wl.Hq)) if h is None else h
    g = h // (wl.Hq // wl.Hkv)
    f64 = lambda t: t.float().cpu().numpy().astype(np.float64)  # noqa: E731
    sub = [f64(q[b:b + 1, :, :, h:h + 1]), f64(kc[b:b + 1, :, g:g + 1]), f64(vc[b:b + 1, :, g:g + 1]),
           f64(kd[b:b + 1, :, :, g:g + 1]), f64(vd[b:b + 1, :, :, g:g + 1])]
    got = f64(out[b:b + 1, :, :, h:h + 1])
    del q, kc, vc, kd, vd, out

    def within(par):
        ref = oracle.verify_attention(*sub, par)
        aw = oracle.verify_attention(sub[0], sub[1], np.abs(sub[2]), sub[3], np.abs(sub[4]), par)
        lim = 2e-3 + 2e-2 * np.abs(ref) + 2 * 2.0 ** -9 * aw
        bad = np.abs(got - ref) > lim
        return (not bad.any()), float(bad.mean())

    pr = np.asarray(parent)[b:b + 1]
    ok, _ = within(pr)
    wrong = {"siblings_chained": np.arange(-1, wl.N - 1, dtype=np.int32)[None]}
    if (pr >= 0).any():
        wrong["ancestors_dropped"] = np.full_like(pr, -1)
    rejected = {}
    for name, wp in wrong.items():
        ok_w, frac_w = within(wp)
        rejected[name] = {"rejected": not ok_w, "fraction_outside": frac_w}
    return {"sequence": b, "head": h, "within_sharp_bound": ok, "wrong_masks": rejected}


def time_warm(x, buf, tau, stream, steps):
    """The same step repeated on one input copy, so that its inputs stay resident in the 256 MB
    Infinity Cache (MALL); reported beside the cold, rotated-copy measurement."""
    for _ in range(3):
        run_step(x, buf, tau, stream)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(steps):
        run_step(x, buf, tau, stream, evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    k = {name: sum(e[a].elapsed_time(e[a + 1]) for e in evs) / steps
         for a, name in enumerate(("verify_attn", "confidence_topk", "accept"))}
    wl = x.wl
    return {"ms_per_step": ms, "tokens_per_s": wl.B * wl.N * wl.L / (ms * 1e-3), "kernels_ms": k}


def time_steps(copies, buf, tau, stream, steps, warmup):
    """W warm-up steps, then K steps over the rotated input copies between two synchronisations,
    HIP events recorded on the launch stream around every call.  Returns (ms per step, per-kernel
    ms averages)."""
    n = len(copies)
    for i in range(warmup):
        run_step(copies[i % n], buf, tau, stream)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(steps):
        run_step(copies[i % n], buf, tau, stream, evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    kernels = {name: sum(e[a].elapsed_time(e[a + 1]) for e in evs) / steps
               for a, name in enumerate(("verify_attn", "confidence_topk", "accept"))}
    return start.elapsed_time(stop) / steps, kernels


def make_copies(wl, tau, dev):
    """Input copies rotated through the timed steps so that together they exceed twice the
    256 MB Infinity Cache and every step reads its inputs from HBM."""
    seed = seed_for(wl.cid)
    x = StepInputs(wl, seed, tau, dev)
    copies = [x]
    n_copies = max(1, min(8, math.ceil(2 * MALL_BYTES / x.nbytes())))
    for c in range(1, n_copies):
        copies.append(StepInputs(wl, seed + 101 * c, tau, dev))
    return copies


def describe(wl, tau):
    return (f"{wl.name}: B{wl.B} N{wl.N} L{wl.L} Hq{wl.Hq} Hkv{wl.Hkv} D{wl.D} S{wl.S}({wl.S_prefix}+{wl.S_suffix}) "
            f"V{wl.V} {wl.logits_dtype} logits, k{wl.k}, tau {tau}")


def step_record(wl, x, ms_step, kernels, n_copies, steps):
    """Throughput and roofline fractions of one workload's timed steps."""
    flops = attn_flops(wl, x.d["parent"])
    t_attn, t_conf = kernels["verify_attn"], kernels["confidence_topk"]
    a_tflops = flops / (t_attn * 1e-3) / 1e12
    a_gbs = attn_bytes(wl) / (t_attn * 1e-3) / 1e9
    l_gbs = logit_bytes(wl) / (t_conf * 1e-3) / 1e9
    return {
        "workload": describe(wl, wl.tau),
        "draft_tokens_per_step": wl.B * wl.N * wl.L,
        "input_copies_rotated": n_copies,
        "steps": steps,
        "step_us": ms_step * 1e3,
        "tokens_per_s": wl.B * wl.N * wl.L / (ms_step * 1e-3),
        "kernel_us": {k: v * 1e3 for k, v in kernels.items()},
        "verify_attn": {"algorithmic_flop_per_launch": flops, "tflops": a_tflops,
                        "frac_of_bf16_peak": a_tflops / PEAK_BF16_TFLOPS,
                        "algorithmic_bytes_per_launch": attn_bytes(wl), "gbs": a_gbs,
                        "frac_of_hbm": a_gbs / PEAK_HBM_GBS,
                        "bound": "hbm" if flops / attn_bytes(wl) < PEAK_BF16_TFLOPS / PEAK_HBM_GBS * 1e3 else "mfma"},
        "logit_pass": {"algorithmic_bytes_per_launch": logit_bytes(wl), "gbs": l_gbs,
                       "frac_of_hbm": l_gbs / PEAK_HBM_GBS},
    }


FLOOR_LIB = os.path.join(ROOT, "paper_2608_27514_amd", "libtrajfloor.so")


def logit_floor(copies, stream, reps):
    """The logit pass's streaming-read floor on the same logit rows: libtrajfloor's read-only kernel
    with the launch shape the pass plans for this shape (workgroup size, load ring, row slices),
    `reps` back-to-back launches over the rotated copies replayed as one HIP graph (graph_time),
    like the pass in the configuration records.  None when the library is not built or the rows
    are not on the pass's 16-byte vector path."""
    import ctypes
    if not os.path.exists(FLOOR_LIB):
        return None
    lib = ctypes.CDLL(FLOOR_LIB)
    fn = lib.traj_floor_logit_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p]
    lg0 = copies[0].logits
    wl = copies[0].wl
    sink = torch.zeros(4096, dtype=torch.int32, device=lg0.device)
    shape = (ctypes.c_int32 * 4)()

    def call(x, s):
        lg = x.logits
        return fn(ctypes.c_void_p(lg.data_ptr()), lg.shape[0], lg.shape[1], lg.stride(0), lg.element_size(),
                  ctypes.c_void_p(sink.data_ptr()), shape, ctypes.c_void_p(s.cuda_stream))

    n = len(copies)
    if call(copies[0], stream) != 0:
        return None
    ms = graph_time(lambda i, s: call(copies[i % n], s), stream, reps)
    gbs = logit_bytes(wl) / (ms * 1e-3) / 1e9
    return {"kernel": "read-only floor (libtrajfloor), same launch shape and loads as the pass",
            "launch": {"threads": shape[0], "unroll": shape[1], "depth": shape[2], "row_slices": shape[3]},
            "us": ms * 1e3, "gbs": gbs, "frac_of_hbm": gbs / PEAK_HBM_GBS}


def mfma_rate(x, stream, reps, flop_target):
    """What the matrix cores sustain on the attention's own operand data: libtrajfloor's MFMA-rate
    kernel (two 4-wave workgroups per CU, each wave issuing back-to-back 32x32x16 bf16 MFMAs on
    fragments read from the cache K and the queries), sized to about the attention's FLOP per
    launch and timed like it (graph_time).  The part holds a lower clock when the multiplies draw
    more power, which depends on the operand bits; this is the ceiling of any kernel's MFMA rate
    on such data, beside the nominal 2.5 PFLOP/s.  None when the library is not built."""
    import ctypes
    if not os.path.exists(FLOOR_LIB):
        return None
    lib = ctypes.CDLL(FLOOR_LIB)
    fn = lib.traj_floor_mfma_rate
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    dev = x.q.device
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    grid = 2 * cus
    per_iter = grid * 4 * 16 * 32768  # FLOP of one round: 16 MFMAs of 2 x 32 x 32 x 16 per wave, 4 waves per workgroup
    iters = max(1, int(round(flop_target / per_iter)))
    sink = torch.zeros(4096, dtype=torch.float32, device=dev)
    clock = torch.zeros(2, dtype=torch.int64, device=dev)

    def call(i, s):
        r = fn(ctypes.c_void_p(x.kc.data_ptr()), x.kc.numel() * 2, ctypes.c_void_p(x.q.data_ptr()), x.q.numel() * 2,
               grid, iters, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(clock.data_ptr()),
               ctypes.c_void_p(s.cuda_stream))
        if r != 0:
            raise RuntimeError("traj_floor_mfma_rate rejected its arguments")

    ms = graph_time(call, stream, reps)
    cyc, ticks = (int(v) for v in clock.cpu().tolist())
    tflops = per_iter * iters / (ms * 1e-3) / 1e12
    return {"kernel": "sustained MFMA rate (libtrajfloor): 32x32x16 bf16 MFMAs back to back on the attention's "
                      "cache K / query data, two 4-wave workgroups per CU",
            "flop_per_launch": per_iter * iters, "us": ms * 1e3, "tflops": tflops,
            "frac_of_peak": tflops / PEAK_BF16_TFLOPS,
            "clock_ghz": cyc / (ticks / 100e6) / 1e9 if ticks > 0 else None}


def graph_time(launch, stream, reps, replays=5):
    """Per-launch ms of `reps` back-to-back launches (launch(i, s) enqueues the i-th on torch
    stream s), captured once in a HIP graph on a side stream and replayed between two HIP events
    on `stream`: the time the kernel takes in a steady stream of launches, without the host issue
    of each call or the dispatch gap between separately issued launches (both matter for kernels
    of tens of microseconds).  One replay of a few milliseconds varies by several percent from
    one replay to the next (clock and memory state), so the median over `replays` timed replays
    (after one untimed) is reported.  The library's entry points only enqueue kernels, so they
    are capturable."""
    for i in range(3):
        launch(i, stream)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for i in range(reps):
            launch(i, side)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    times = []
    for _ in range(replays):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / reps)
    del g
    return statistics.median(times)


def time_kernels_apart(copies, buf, tau, stream, reps):
    """Each kernel of the step on its own: `reps` back-to-back launches over the rotated copies,
    timed as one replayed HIP graph (graph_time).  Returns per-launch ms."""
    n = len(copies)
    calls = {
        "verify_attn": lambda x, s: tsp.verify_attn(x.q, x.kc, x.vc, x.kd, x.vd, x.parent, out=buf.out, stream=s),
        "confidence_topk": lambda x, s: tsp.confidence_topk(x.logits, x.wl.k, conf=buf.conf, idx=buf.idx,
                                                            workspace=buf.ws, stream=s),
        "accept": lambda x, s: tsp.accept(buf.conf, buf.idx, x.tokens, x.parent, x.committed, x.conf0, x.idx0, tau,
                                          out=buf.acc, stream=s),
    }
    return {name: graph_time(lambda i, s, fn=fn: fn(copies[i % n], s), stream, reps) for name, fn in calls.items()}


def time_config(cid, stream, steps, warmup):
    """A workload other than the headline one, timed in the same run: the step exactly as the
    headline step (rotated copies, HIP events on the launch stream around every call), and each
    kernel in back-to-back launches of its own (the fractions of the roofline use these)."""
    wl = WORKLOADS[cid]
    dev = torch.device("cuda:0")
    copies = make_copies(wl, wl.tau, dev)
    buf = Buffers(wl, dev, copies[0].logits)
    torch.cuda.synchronize()
    ms_step, in_step = time_steps(copies, buf, wl.tau, stream, steps, warmup)
    kernels = time_kernels_apart(copies, buf, wl.tau, stream, steps)
    rec = step_record(wl, copies[0], ms_step, kernels, len(copies), steps)
    rec["kernel_us_in_step"] = {k: v * 1e3 for k, v in in_step.items()}
    # the same step captured once as a HIP graph of `steps` back-to-back steps over the rotated
    # copies and replayed (graph_time): what a serving loop that captures its step gets, without
    # the host issue of three calls per step and the events around them
    n = len(copies)
    ms_graph = graph_time(lambda i, s: run_step(copies[i % n], buf, wl.tau, s), stream, steps)
    rec["step_us_graph"] = ms_graph * 1e3
    rec["tokens_per_s_graph"] = wl.B * wl.N * wl.L / (ms_graph * 1e-3)
    fl = logit_floor(copies, stream, steps)
    if fl is not None:
        fl["logit_pass_over_floor"] = kernels["confidence_topk"] * 1e3 / fl["us"]
    rec["logit_pass"]["floor"] = fl
    run_step(copies[0], buf, wl.tau, stream)
    torch.cuda.synchronize()
    rec["accepted_tokens_per_step"] = float(buf.acc["n_accepted"].sum().item())
    del copies, buf
    torch.cuda.empty_cache()
    return rec


TREE_WIDTH, TREE_DEPTH = 3, 3  # the paper's adopted W3D3 hybrid tree


def time_tree_build(x, buf, tau, stream, reps=50):
    """The next step's drafts from this step's acceptance (traj_build_tree, Alg. 1), timed
    with HIP events on the launch stream; not part of the verification step above."""
    wl = x.wl
    k = wl.k
    conf = buf.conf.view(wl.B, wl.N, wl.L, k)
    idx = buf.idx.view(wl.B, wl.N, wl.L, k)
    args = (buf.acc["out_tokens"], x.conf0, x.idx0, tau, TREE_WIDTH, TREE_DEPTH, k)
    kw = dict(leaf=buf.acc["leaf"], conf=conf, idx=idx, stream=stream)
    out = tsp.build_tree(*args, **kw)
    kw["out"] = out
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        tsp.build_tree(*args, **kw)
    e1.record(stream)
    torch.cuda.synchronize()
    n_nodes = out["n_nodes"].cpu().numpy()
    return {"ms": e0.elapsed_time(e1) / reps, "tree": f"W{TREE_WIDTH}D{TREE_DEPTH} hybrid, branch {k}",
            "node_slots": int(out["parent"].shape[1]), "mean_nodes": float(n_nodes.mean())}


def time_interblock(x, buf, tau, stream, reps=5, trig_reps=50):
    """Inter-block speculation pieces on the same inputs (not part of the step): attention with
    root-to-root peer visibility for a joint packing (the last drafts form the next block's tree,
    the first draft of each tree is its root), and the trigger on two blocks' states."""
    wl = x.wl
    n_next = min(4, wl.N - 1)
    if n_next < 1:
        return None
    peers = tsp.joint_peers(wl.B, wl.N - n_next, n_next, device=x.q.device, stream=stream)
    scratch = torch.empty_like(buf.out)  # buf.out stays the step's output
    times = {"plain": 0.0, "peers": 0.0}
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2 * reps)]
    for r in range(2 * reps + 2):  # alternate the two variants; the first pair warms up
        name = "plain" if r % 2 == 0 else "peers"
        kw = dict(out=scratch, stream=stream, peers=peers if name == "peers" else None)
        if r >= 2:
            evs[r - 2][0].record(stream)
        tsp.verify_attn(x.q, x.kc, x.vc, x.kd, x.vd, x.parent, **kw)
        if r >= 2:
            evs[r - 2][1].record(stream)
    torch.cuda.synchronize()
    for r in range(2 * reps):
        times["plain" if r % 2 == 0 else "peers"] += evs[r][0].elapsed_time(evs[r][1]) / reps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # trigger: the accepted block state followed by the committed state as the next block
    state2 = torch.cat([buf.acc["out_tokens"], x.committed], 1).contiguous()
    conf2 = buf.conf.view(wl.B, wl.N * wl.L, wl.k)[:, :2 * wl.L].contiguous()
    out = tsp.interblock_trigger(state2, conf2, tau, stream=stream)
    e0.record(stream)
    for _ in range(trig_reps):
        tsp.interblock_trigger(state2, conf2, tau, out=out, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    return {"joint_drafts": f"{wl.N - n_next}+{n_next}, root-to-root peers", "attn_peers_ms": times["peers"],
            "attn_plain_ms": times["plain"], "trigger_ms": e0.elapsed_time(e1) / trig_reps,
            "triggered_sequences": int(out["trigger"].sum().item())}


W3D3_PARENTS = [-1, 0, 0, 0, 1, 2, 4]  # hybrid W3D3 tree: root + 3 + 2 + 1 drafts


def time_layer(x, stream, reps=5):
    """One verification decoder layer (traj_verify_layer) over the workload's packed drafts, with
    random-init weights of the layer shape (MLP width 3 x hidden, as in the 8B models), and its
    four projection GEMMs alone (traj_linear), timed with HIP events on the launch stream; not
    part of the verification step above."""
    wl = x.wl
    return _time_layer(wl.B, wl.N, wl.L, wl.Hq, wl.Hkv, wl.D, wl.S, wl.S_prefix, x.kc, x.vc, x.parent,
                       seed_for(wl.cid, salt=31), stream, reps)


def time_layer_one_sequence(wl, stream, reps=20):
    """The same layer for one sequence's W3D3 hybrid tree (7 drafts of the block), the paper's
    single-sequence decoding setting: 224 draft tokens, cache 512 + 224."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed_for(wl.cid, salt=37))
    S_prefix, S = 512, 512 + 7 * wl.L
    kc = torch.randn(1, S, wl.Hkv, wl.D, device=dev, generator=g).to(torch.bfloat16)
    vc = torch.randn(1, S, wl.Hkv, wl.D, device=dev, generator=g).to(torch.bfloat16)
    parent = torch.tensor([W3D3_PARENTS], dtype=torch.int32, device=dev)
    return _time_layer(1, len(W3D3_PARENTS), wl.L, wl.Hq, wl.Hkv, wl.D, S, S_prefix, kc, vc, parent,
                       seed_for(wl.cid, salt=41), stream, reps)


def time_refresh(wl, stream, reps=3):
    """The dual-cache refresh at a block boundary (traj_refresh_layer: one decoder layer over
    whole sequences, bidirectional attention, prefix / suffix K and V written to the cache), for
    one sequence (prefix 512, block 32, suffix 224) and for the workload's batch (its prefix,
    block and suffix), random-init weights of the 8B layer shape."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed_for(wl.cid, salt=43))
    hidden, inter = wl.Hq * wl.D, 3 * wl.Hq * wl.D
    qkv = (wl.Hq + 2 * wl.Hkv) * wl.D

    def r(*shape, scale=1.0):
        return (torch.randn(*shape, device=dev, generator=g) * scale).to(torch.bfloat16)

    w = {"attn_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16), "w_qkv": r(hidden, qkv, scale=hidden ** -0.5),
         "w_o": r(wl.Hq * wl.D, hidden, scale=hidden ** -0.5),
         "mlp_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16),
         "w_gate_up": r(hidden, 2 * inter, scale=hidden ** -0.5), "w_down": r(inter, hidden, scale=inter ** -0.5)}
    out = {}
    for name, B, prefix, suffix in (("one_sequence", 1, 512, 224), ("batch", wl.B, wl.S_prefix, wl.S_suffix)):
        S, L = prefix + suffix, wl.L
        x0 = r(B, S + L, hidden)
        x = x0.clone()
        starts = torch.full((B,), prefix, dtype=torch.int32, device=dev)
        kc = torch.empty(B, S, wl.Hkv, wl.D, dtype=torch.bfloat16, device=dev)
        vc = torch.empty_like(kc)
        ws = torch.empty(tsp.refresh_layer_workspace_size(B, S, L, wl.Hq, wl.Hkv, wl.D, hidden, inter),
                         dtype=torch.uint8, device=dev)
        total = 0.0
        for i in range(reps + 1):  # the first call warms up
            x.copy_(x0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            tsp.refresh_layer(x, w, starts, wl.Hq, wl.Hkv, L, k_cache=kc, v_cache=vc, workspace=ws, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            if i > 0:
                total += e0.elapsed_time(e1)
        T = B * (S + L)
        out[name] = {"sequences": B, "tokens": T, "cache_rows": S, "ms_per_layer": total / reps,
                     "gemm_tflop": 2.0 * T * hidden * (qkv + hidden + 3 * inter) / 1e12,
                     "attention_tflop": 4.0 * B * (S + L) ** 2 * wl.D * wl.Hq / 1e12}
        del x0, x, kc, vc, ws
    return out


FORWARD_LAYERS = 32  # decoder layers of the 8B models


def time_forward_one_sequence(wl, stream, reps=20):
    """Per-step latency of one sequence's whole verification forward against its number of draft
    blocks (in kind the per-step latency the paper plots against draft blocks, Sec. 4,
    computational overhead analysis): 32 verification layers of the 8B
    shape (random-init weights, one dual cache per layer: prefix 512 + suffix 224), the LM head
    (traj_linear), the logit pass, acceptance and the next tree (W3D3), captured once as a HIP
    graph and replayed; the eager time (one Python call per entry point) is given beside it.
    Drafts 1, 2, 4, 7 are prefixes of the W3D3 hybrid tree.  The final RMSNorm before the LM
    head is not a library call and is left out (one pass over the draft rows)."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed_for(wl.cid, salt=53))
    Hq, Hkv, D, L, k, V = wl.Hq, wl.Hkv, wl.D, wl.L, wl.k, wl.V
    hidden, inter = Hq * D, 3 * Hq * D
    qkv = (Hq + 2 * Hkv) * D
    S_prefix, S = 512, 512 + 224

    def r(*shape, scale=1.0):
        return (torch.randn(*shape, device=dev, generator=g) * scale).to(torch.bfloat16)

    layers = []
    for _ in range(FORWARD_LAYERS):
        layers.append({"w": {"attn_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16),
                             "w_qkv": r(hidden, qkv, scale=hidden ** -0.5), "w_o": r(Hq * D, hidden, scale=hidden ** -0.5),
                             "mlp_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16),
                             "w_gate_up": r(hidden, 2 * inter, scale=hidden ** -0.5),
                             "w_down": r(inter, hidden, scale=inter ** -0.5)},
                       "kc": r(1, S, Hkv, D), "vc": r(1, S, Hkv, D)})
    lm_head = r(hidden, V, scale=hidden ** -0.5)
    pos0 = torch.full((1,), S_prefix, dtype=torch.int32, device=dev)
    committed = torch.where(torch.rand(1, L, device=dev, generator=g) < 0.75,
                            torch.full((1, L), -1, dtype=torch.int32, device=dev),
                            torch.randint(0, V, (1, L), device=dev, generator=g, dtype=torch.int32))
    conf0 = torch.rand(1, L, k, device=dev, generator=g)
    idx0 = torch.randint(0, V, (1, L, k), device=dev, generator=g, dtype=torch.int32)
    out = {"layers": FORWARD_LAYERS, "cache_rows": S, "per_drafts": {}}
    base = None
    for n in (1, 2, 4, 7):
        parent = torch.tensor([W3D3_PARENTS[:n]], dtype=torch.int32, device=dev)
        tokens = torch.randint(0, V, (1, n, L), device=dev, generator=g, dtype=torch.int32)
        x0 = r(1, n, L, hidden)
        x = x0.clone()
        T = n * L
        ws = torch.empty(tsp.layer_workspace_size(1, n, L, Hq, Hkv, D, S, hidden, inter), dtype=torch.uint8,
                         device=dev)
        logits = torch.empty(T, V, dtype=torch.bfloat16, device=dev)
        lws = torch.empty(max(tsp.linear_workspace_size(T, hidden, V), 16), dtype=torch.uint8, device=dev)
        conf = torch.empty(T, k, dtype=torch.float32, device=dev)
        idx = torch.empty(T, k, dtype=torch.int32, device=dev)
        cws = torch.empty(max(tsp.confidence_topk_workspace_size(logits, k), 16), dtype=torch.uint8, device=dev)
        acc = {"leaf": torch.empty(1, dtype=torch.int32, device=dev),
               "on_path": torch.empty((1, n), dtype=torch.uint8, device=dev),
               "n_accepted": torch.empty(1, dtype=torch.int32, device=dev),
               "out_tokens": torch.empty((1, L), dtype=torch.int32, device=dev),
               "hi": torch.empty((1, n, L), dtype=torch.uint8, device=dev)}
        acc["leaf"].fill_(-1)  # before the first forward: no accepted draft, the committed state
        acc["out_tokens"].copy_(committed)
        targs = (acc["out_tokens"], conf0, idx0, wl.tau, TREE_WIDTH, TREE_DEPTH, k)
        tkw = dict(leaf=acc["leaf"], conf=conf.view(1, n, L, k), idx=idx.view(1, n, L, k))
        tkw["out"] = tsp.build_tree(*targs, **tkw)

        def forward(s):
            x.copy_(x0)
            for ly in layers:
                tsp.verify_layer(x, ly["w"], ly["kc"], ly["vc"], parent, Hq, pos0=pos0, workspace=ws, stream=s)
            tsp.linear(x.view(T, hidden), lm_head, y=logits, workspace=lws, stream=s)
            tsp.confidence_topk(logits, k, conf=conf, idx=idx, workspace=cws, stream=s)
            tsp.accept(conf, idx, tokens, parent, committed, conf0, idx0, wl.tau, out=acc, stream=s)
            tsp.build_tree(*targs, **tkw, stream=s)

        def timed(fn):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            fn()
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        eager_ms = timed(lambda: forward(stream))
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            forward(torch.cuda.current_stream())
        torch.cuda.synchronize()
        graph_ms = timed(graph.replay)
        base = graph_ms if base is None else base
        out["per_drafts"][str(n)] = {"draft_tokens": T, "graph_ms": graph_ms, "eager_ms": eager_ms,
                                     "vs_one_draft": graph_ms / base}
        del graph, ws, logits, lws, x, x0
    del layers, lm_head
    torch.cuda.empty_cache()
    return out


def _time_layer(B, N, L, Hq, Hkv, D, S, S_prefix, kc, vc, parent, seed, stream, reps):
    dev = kc.device
    hidden, inter = Hq * D, 3 * Hq * D
    qkv = (Hq + 2 * Hkv) * D
    T = B * N * L
    g = torch.Generator(device=dev)
    g.manual_seed(seed)

    def r(*shape, scale=1.0):
        return (torch.randn(*shape, device=dev, generator=g) * scale).to(torch.bfloat16)

    w = {"attn_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16), "w_qkv": r(hidden, qkv, scale=hidden ** -0.5),
         "w_o": r(Hq * D, hidden, scale=hidden ** -0.5),
         "mlp_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16),
         "w_gate_up": r(hidden, 2 * inter, scale=hidden ** -0.5), "w_down": r(inter, hidden, scale=inter ** -0.5)}
    h0 = r(B, N, L, hidden)
    h = h0.clone()
    pos0 = torch.full((B,), S_prefix, dtype=torch.int32, device=dev)
    ws = torch.empty(tsp.layer_workspace_size(B, N, L, Hq, Hkv, D, S, hidden, inter), dtype=torch.uint8, device=dev)

    def timed(fn, before=None):
        total = 0.0
        for i in range(reps + 1):  # the first call warms up
            if before is not None:
                before()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            if i > 0:
                total += e0.elapsed_time(e1)
        return total / reps

    layer_ms = timed(lambda: tsp.verify_layer(h, w, kc, vc, parent, Hq, pos0=pos0, workspace=ws, stream=stream),
                     before=lambda: h.copy_(h0))
    gemms = {}
    a = h0.view(T, hidden)
    for name, K, Nn, acc in (("qkv", hidden, qkv, False), ("o", Hq * D, hidden, True),
                             ("gate_up", hidden, 2 * inter, False), ("down", inter, hidden, True)):
        src = a if K == hidden else r(T, K)
        y = torch.zeros(T, Nn, dtype=torch.bfloat16, device=dev)
        lws = torch.empty(max(tsp.linear_workspace_size(T, K, Nn), 16), dtype=torch.uint8, device=dev)
        ms = timed(lambda: tsp.linear(src, w["w_" + name], y=y, accumulate=acc, workspace=lws, stream=stream))
        tflops = 2.0 * T * K * Nn / (ms * 1e-3) / 1e12
        weight_tbs = K * Nn * 2 / (ms * 1e-3) / 1e12
        gemms[name] = {"M": T, "K": K, "N": Nn, "ms": ms, "tflops": tflops,
                       "frac_of_bf16_peak": tflops / PEAK_BF16_TFLOPS, "weight_read_tb_s": weight_tbs}
        del y
    gemm_flops = 2.0 * T * hidden * (qkv + hidden + 3 * inter)
    weight_bytes = 2.0 * hidden * (qkv + hidden + 3 * inter)
    return {"shape": f"hidden {hidden}, {Hq} q / {Hkv} kv heads x {D}, MLP {inter}, {T} draft tokens, cache {S}",
            "weights": "synthetic (random init)", "ms_per_layer": layer_ms,
            "weight_bytes_per_layer": weight_bytes, "gemm_ms": sum(v["ms"] for v in gemms.values()),
            "gemm_tflops": gemm_flops / (sum(v["ms"] for v in gemms.values()) * 1e-3) / 1e12, "gemms": gemms}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=5, choices=sorted(WORKLOADS))
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-seqs", type=int, default=8)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the measurements beside the step (warm cache, tree build, inter-block), e.g. "
                         "for a kernel trace of the step alone")
    ap.add_argument("--with-floor", action="store_true",
                    help="time the logit pass's streaming-read floor even with --no-extras")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip timing the other workloads (the 'configs' record)")
    ap.add_argument("--config-steps", type=int, default=50, help="timed steps of each other workload")
    ap.add_argument("--no-sharp-parity", action="store_true",
                    help="skip the sharp-input attention check at the timed launch")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run three 1 GiB device-to-device copies (for scaling rocprofv3 FETCH_SIZE / "
                         "WRITE_SIZE readings) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        src = torch.ones((1 << 30) // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 1 << 30, "copy_bytes_written": 1 << 30, "copies": 3}))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs the verification step on exactly one GPU; "
                                   "sequences shard across GPUs with no exchange, so N>1 is N independent "
                                   "copies of this benchmark and is not launched here"}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(2)
    tsp.load()  # fails loudly when the HIP library is missing

    wl = WORKLOADS[args.workload]
    tau = wl.tau if args.tau is None else args.tau
    dev = torch.device("cuda:0")
    seed = seed_for(wl.cid)
    log(f"inputs: {wl.name}")
    copies = make_copies(wl, tau, dev)
    x = copies[0]
    n_copies = len(copies)
    buf = Buffers(wl, dev, x.logits)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    ms_step, kern = time_steps(copies, buf, tau, stream, args.steps, args.warmup)
    log(f"step {ms_step:.4f} ms")
    t_attn, t_conf, t_acc = kern["verify_attn"], kern["confidence_topk"], kern["accept"]

    tokens = wl.B * wl.N * wl.L
    flops = attn_flops(wl, x.d["parent"])
    a_tflops = flops / (t_attn * 1e-3) / 1e12
    l_gbs = logit_bytes(wl) / (t_conf * 1e-3) / 1e9
    warm = time_warm(x, buf, tau, stream, args.steps) if n_copies > 1 and not args.no_extras else None
    # the last timed step used copies[(K-1) % n]; rerun copy 0 so outputs match x
    run_step(x, buf, tau, stream)
    torch.cuda.synchronize()
    acc_main = buf.acc["n_accepted"].cpu().numpy()
    if not args.no_extras:
        log("extras: tree build, layer, refresh, inter-block, one-sequence forward")
    tree = None if args.no_extras else time_tree_build(x, buf, tau, stream)
    layer = None if args.no_extras else time_layer(x, stream)
    layer_one = None if args.no_extras else time_layer_one_sequence(wl, stream)
    refresh = None if args.no_extras else time_refresh(wl, stream)
    inter = None if args.no_extras else time_interblock(x, buf, tau, stream)
    forward = None if args.no_extras else time_forward_one_sequence(wl, stream)
    if not args.no_sharp_parity:
        log("sharp-input attention check at the timed launch")
    sharp = None if args.no_sharp_parity else sharp_sample_parity(wl, x.d["parent"], stream)
    configs = None
    if not args.no_configs:
        configs = {}
        for cid in sorted(WORKLOADS):
            if cid != wl.cid:
                log(f"config {WORKLOADS[cid].name}")
                configs[WORKLOADS[cid].name] = time_config(cid, stream, args.config_steps, args.warmup)
    floor = logit_floor(copies, stream, args.steps) if (args.with_floor or not args.no_extras) else None
    if floor is not None:
        floor["logit_pass_over_floor"] = t_conf * 1e3 / floor["us"]
    sustained = None
    if args.with_floor or not args.no_extras:
        log("sustained MFMA rate on the attention's operands")
        sustained = mfma_rate(copies[0], stream, args.steps, flops)
        if sustained is not None:
            sustained["attention_over_sustained"] = a_tflops / sustained["tflops"]
    status = tsp.device_status(reset=True)

    result = {
        "metric": "verified draft tokens/sec/GPU",
        "value": tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; stands in for the paper's benchmarks and LLaDA/Dream activations)",
        "config": {
            "workload": describe(wl, tau),
            "draft_tokens_per_step": tokens,
            "tree": "levels " + "+".join(map(str, wl.level_sizes)) if wl.level_sizes else "explicit parents",
            "input_copies_rotated": n_copies,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "verify_attn",
            "achieved": a_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": a_tflops / PEAK_BF16_TFLOPS,
            "traffic": measured_traffic("verify_attn", wl.name),
            "algorithmic_flop_per_launch": flops,
            "sustained_mfma": sustained,
        },
        "kernels_ms": {"verify_attn": t_attn, "confidence_topk": t_conf, "accept": t_acc},
        "logit_pass": {"bound": "hbm", "achieved": l_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                       "frac": l_gbs / PEAK_HBM_GBS, "algorithmic_bytes_per_launch": logit_bytes(wl),
                       "traffic": measured_traffic("confidence_topk", wl.name), "floor": floor},
        "attention_hbm_bytes_per_launch": attn_bytes(wl),
        "accepted_tokens_per_step": {str(tau): float(acc_main.sum())},
        "mean_accepted_per_sequence": {str(tau): float(acc_main.mean())},
        "warm": warm if warm is not None or args.no_extras else
                "inputs exceed the 256 MB Infinity Cache: every step reads HBM",
        "tree_build": tree,
        "interblock": inter,
        "verify_layer": layer,
        "verify_layer_one_sequence": layer_one,
        "refresh_layer": refresh,
        "forward_one_sequence": forward,
        "device_status": status,
    }
    if configs is not None:
        result["configs"] = configs
    if sharp is not None:
        result["attention_sharp_parity"] = sharp
    if wl.cid == 5 and not args.no_sweep:
        for t2 in (0.7, 0.8):
            x.replant(seed, t2)
            run_step(x, buf, t2, stream)
            torch.cuda.synchronize()
            a = buf.acc["n_accepted"].cpu().numpy()
            result["accepted_tokens_per_step"][str(t2)] = float(a.sum())
            result["mean_accepted_per_sequence"][str(t2)] = float(a.mean())
        x.replant(seed, tau)
        run_step(x, buf, tau, stream)
        torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        log("oracle baseline on the host")
        result["cpu_baseline"] = cpu_baseline(x, buf, wl, tau, min(args.cpu_sample_seqs, wl.B))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
