"""GPU parity: traj_build_tree against the tree-construction oracle (Alg. 1).

Tokens, parents and node counts are integer outputs and must be bit-exact; the kernel and
the oracle take every decision on the same fp32 confidences (the threshold rounded to fp32,
as the kernel compares it).  Path scores are fp32 sums of logf against fp64 sums of log:
|gpu - ref| <= 1e-5 (1 + |ref|).  A closed loop (build, accept, build ...) with a static
candidate table runs the multi-step decode of one block entirely on the GPU and must follow
the oracle's loop step for step.
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from helpers import cuda
from oracle.tree import build_tree_batch

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_build.json")


def _random_batch(rng, B, L, k, p_mask=0.7, ties=False, n_prev=0):
    state = np.where(rng.random((B, L)) < p_mask, -1, rng.integers(0, 50000, (B, L))).astype(np.int32)

    def table(shape):
        top = rng.random(shape) ** 0.5
        if ties:
            top = np.round(top * 4) / 4
        conf = np.empty(shape + (k,), dtype=np.float32)
        conf[..., 0] = top
        rest = np.sort(rng.random(shape + (max(k - 1, 1),)), axis=-1)[..., ::-1] * (1 - top)[..., None] / max(k - 1, 1)
        if k > 1:  # a top-k row is non-increasing
            conf[..., 1:] = np.minimum(rest[..., : k - 1], top[..., None])
        idx = np.argsort(rng.random(shape + (64,)), axis=-1)[..., :k].astype(np.int32) + 100
        return conf, idx

    conf0, idx0 = table((B, L))
    conf, idx = table((B, n_prev, L)) if n_prev else (None, None)
    return state, conf0, idx0, conf, idx


def _check(state, conf0, idx0, tau, W, D, branch, full, leaf=None, conf=None, idx=None, branch_deep=1):
    B, L = state.shape
    k = conf0.shape[-1]
    tau32 = float(np.float32(tau))
    n_max = tsp.tree_max_nodes(B, L, k, W, D, branch, full, branch_deep)
    ref_t, ref_p, ref_n, ref_s = build_tree_batch(state, leaf, conf, idx, conf0, idx0, tau32, W, D, branch, full,
                                                  n_max, branch_deep)
    out = tsp.build_tree(cuda(state, torch.int32), cuda(conf0, torch.float32), cuda(idx0, torch.int32), tau, W, D,
                         branch, full, leaf=None if leaf is None else cuda(leaf, torch.int32),
                         conf=None if conf is None else cuda(conf, torch.float32),
                         idx=None if idx is None else cuda(idx, torch.int32), branch_deep=branch_deep)
    torch.cuda.synchronize()
    g = {key: v.cpu().numpy() for key, v in out.items()}
    assert np.array_equal(g["n_nodes"], ref_n)
    assert np.array_equal(g["parent"], ref_p)
    assert np.array_equal(g["tokens"], ref_t)
    fin = np.isfinite(ref_s)
    assert np.array_equal(np.isfinite(g["score"]), fin)
    assert (np.abs(g["score"][fin] - ref_s[fin]) <= 1e-5 * (1 + np.abs(ref_s[fin]))).all()
    for b in range(B):
        lf = -1 if leaf is None else int(leaf[b])
        C, I = (conf0[b], idx0[b]) if lf < 0 else (conf[b, lf], idx[b, lf])
        assert np.array_equal(g["conf_next"][b], C) and np.array_equal(g["idx_next"][b], I)
    return g


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_golden_trees(case):
    state = np.array([case["s0"]], dtype=np.int32)
    conf0 = np.array([case["conf"]], dtype=np.float32)
    idx0 = np.array([case["idx"]], dtype=np.int32)
    g = _check(state, conf0, idx0, case["tau"], case["width"], case["depth"], case["branch"], bool(case["full"]),
               branch_deep=case.get("branch_deep", 1))
    n = len(case["parent"])
    assert g["n_nodes"][0] == n and g["parent"][0, :n].tolist() == case["parent"]


@pytest.mark.parametrize("seed", range(36))
def test_random_parity(seed):
    """Random shapes and tables; several children per node below the first level only on tables
    without exact ties (pruning across parents compares fp32 sums of logf on the GPU with fp64
    sums in the oracle, so only clear score gaps decide identically)."""
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 40))
    L = int(rng.choice([1, 5, 17, 32, 63, 64]))
    k = int(rng.integers(1, 9))
    W, D = int(rng.integers(1, 6)), int(rng.integers(0, 7))
    branch = int(rng.integers(1, k + 1))
    full = bool(seed % 2)
    tau = float(rng.choice([0.3, 0.7, 0.9, 0.95]))
    n_prev = int(rng.integers(0, 5))
    state, conf0, idx0, conf, idx = _random_batch(rng, B, L, k, p_mask=float(rng.choice([0.0, 0.3, 0.9, 1.0])),
                                                  ties=seed % 3 == 0, n_prev=n_prev)
    leaf = rng.integers(-1, n_prev, B).astype(np.int32) if n_prev else None
    bd = 1 if seed % 3 == 0 else int(rng.integers(1, k + 1))
    if tsp.tree_max_nodes(B, L, k, W, D, branch, full, bd) > 64:
        bd = 1
    if tsp.tree_max_nodes(B, L, k, W, D, branch, full, bd) > 64:
        pytest.skip("tree larger than 64 nodes")
    _check(state, conf0, idx0, tau, W, D, branch, full, leaf, conf, idx, branch_deep=bd)


def test_workload_shapes():
    """The 8B-shaped blocks: L = 32, k = 3, W3D3 hybrid and full, 16 and 256 sequences."""
    rng = np.random.default_rng(5)
    for B, full, bd in ((16, False, 1), (256, True, 1), (64, True, 2)):
        state, conf0, idx0, _, _ = _random_batch(rng, B, 32, 3, p_mask=0.75)
        _check(state, conf0, idx0, 0.9, 3, 3, 3, full, branch_deep=bd)


def test_bad_leaf_is_reported_and_taken_as_minus_one():
    rng = np.random.default_rng(3)
    state, conf0, idx0, conf, idx = _random_batch(rng, 4, 16, 3, n_prev=2)
    tsp.device_status(reset=True)
    leaf = np.array([0, 5, -3, 1], dtype=np.int32)
    out = tsp.build_tree(cuda(state, torch.int32), cuda(conf0, torch.float32), cuda(idx0, torch.int32), 0.9, 3, 3, 3,
                         leaf=cuda(leaf, torch.int32), conf=cuda(conf, torch.float32), idx=cuda(idx, torch.int32))
    assert tsp.device_status(reset=True) & tsp.DEV_BAD_LEAF
    fixed = np.array([0, -1, -1, 1], dtype=np.int32)
    ref_t, ref_p, ref_n, _ = build_tree_batch(state, fixed, conf, idx, conf0, idx0, float(np.float32(0.9)), 3, 3, 3,
                                              False, out["parent"].shape[1])
    assert np.array_equal(out["tokens"].cpu().numpy(), ref_t) and np.array_equal(out["n_nodes"].cpu().numpy(), ref_n)


@pytest.mark.parametrize("full", [False, True])
def test_closed_loop_decode_of_a_block(full):
    """Build, accept (exact, greedy), build ... on the GPU until every block is complete; the
    candidate table is static (every node's own candidates are the block's table), so the oracle
    loop is exact and both must agree at every step."""
    rng = np.random.default_rng(11 + full)
    B, L, k, tau, W, D = 8, 32, 3, 0.9, 3, 3
    state, conf0, idx0, _, _ = _random_batch(rng, B, L, k, p_mask=1.0)
    n_max = tsp.tree_max_nodes(B, L, k, W, D, k, full)
    s_gpu = cuda(state, torch.int32)
    c0_gpu, i0_gpu = cuda(conf0, torch.float32), cuda(idx0, torch.int32)
    s_ref = state.copy()
    steps = 0
    while (s_ref == -1).any():
        steps += 1
        assert steps <= L
        tr = tsp.build_tree(s_gpu, c0_gpu, i0_gpu, tau, W, D, k, full)
        t_ref, p_ref, n_ref, _ = build_tree_batch(s_ref, None, None, None, conf0, idx0, float(np.float32(tau)), W,
                                                  D, k, full, n_max)
        torch.cuda.synchronize()
        assert np.array_equal(tr["tokens"].cpu().numpy(), t_ref) and np.array_equal(tr["parent"].cpu().numpy(), p_ref)
        conf_all = c0_gpu[:, None].expand(B, n_max, L, k).contiguous()
        idx_all = i0_gpu[:, None].expand(B, n_max, L, k).contiguous()
        acc = tsp.accept(conf_all, idx_all, tr["tokens"], tr["parent"], s_gpu, c0_gpu, i0_gpu, tau, "exact", "greedy")
        ref = oracle.accept_batch(t_ref, p_ref, s_ref, conf0, idx0, np.repeat(conf0[:, None], n_max, 1),
                                  np.repeat(idx0[:, None], n_max, 1), float(np.float32(tau)), "exact", "greedy")
        torch.cuda.synchronize()
        assert np.array_equal(acc["leaf"].cpu().numpy(), ref["leaf"])
        assert np.array_equal(acc["out_tokens"].cpu().numpy(), ref["out_tokens"])
        done = (s_ref != -1).all(axis=1)
        assert (ref["n_accepted"][~done] >= 1).all()  # every unfinished block advances
        s_gpu = acc["out_tokens"].clone()
        s_ref = ref["out_tokens"].astype(np.int32)
    assert steps >= 1 and (s_gpu.cpu().numpy() == s_ref).all()
