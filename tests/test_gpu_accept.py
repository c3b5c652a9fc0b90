"""GPU parity: traj_accept against the oracle.

With the oracle's own confidences fed to both sides there is nothing to
exclude: every output must be bit-exact, in every mode and traversal.
"""

import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from synthetic import WORKLOADS, decode_inputs, make_logits, seed_for
from helpers import cuda

pytestmark = pytest.mark.gpu

MODES = ["exact", "top1", "topk"]
TRAVS = ["greedy", "longest"]


def _run_both(tokens, parent, committed, conf0, idx0, conf, idx, tau, mode, trav):
    B, N, L = tokens.shape
    k = conf0.shape[-1]
    tau32 = float(np.float32(tau))  # the kernel compares fp32 values with fp32 tau
    ref = oracle.accept_batch(tokens, parent, committed, conf0.astype(np.float64), idx0,
                              conf.astype(np.float64), idx, tau32, mode, trav)
    out = tsp.accept(cuda(conf.reshape(-1, k), torch.float32), cuda(idx.reshape(-1, k), torch.int32),
                     cuda(tokens, torch.int32), cuda(parent, torch.int32), cuda(committed, torch.int32),
                     cuda(conf0, torch.float32), cuda(idx0, torch.int32), tau, mode, trav)
    torch.cuda.synchronize()
    g = {key: v.cpu().numpy() for key, v in out.items()}
    assert np.array_equal(g["leaf"], ref["leaf"]), (mode, trav, g["leaf"], ref["leaf"])
    assert np.array_equal(g["n_accepted"], ref["n_accepted"]), (mode, trav)
    assert np.array_equal(g["on_path"].astype(bool), ref["on_path"]), (mode, trav)
    assert np.array_equal(g["out_tokens"], ref["out_tokens"]), (mode, trav)
    assert np.array_equal(g["hi"].astype(bool), ref["hi"]), (mode, trav)
    return ref


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_oracle_fed_workloads_all_modes(cid):
    wl = WORKLOADS[cid]
    wl_small_v = wl.with_(V=min(wl.V, 2048))
    d = decode_inputs(wl_small_v, seed_for(cid))
    B, N, L, k = wl.B, wl.N, wl.L, wl.k
    lg = make_logits(d["row_margin"], d["row_top"], wl_small_v.V, torch.float32, seed_for(cid))
    c, i = oracle.confidence_topk(lg.numpy(), k)
    conf = c.astype(np.float32).reshape(B, N, L, k)
    idx = i.astype(np.int32).reshape(B, N, L, k)
    for mode, trav in itertools.product(MODES, TRAVS):
        ref = _run_both(d["tokens"], d["parent"], d["committed"], d["conf0"], d["idx0"], conf, idx,
                        wl.tau, mode, trav)
        if mode == "exact" and trav == "greedy":
            assert np.array_equal(ref["leaf"], d["planted_leaf"])


def test_random_small_trees_discrete_confidences():
    rng = np.random.default_rng(99)
    L, k = 5, 3
    for n in (1, 2, 3, 4):
        for par in itertools.product(*[range(-1, j) for j in range(n)]):
            B = 6
            parent = np.tile(np.array(par, dtype=np.int32), (B, 1))
            committed = rng.integers(0, 3, size=(B, L)).astype(np.int32)
            committed[rng.random((B, L)) < 0.7] = -1
            levels = np.array([0.25, 0.5, 0.75, 0.875, 0.9375], dtype=np.float32)
            conf0 = rng.choice(levels, size=(B, L, k)).astype(np.float32)
            idx0 = rng.integers(0, 3, size=(B, L, k)).astype(np.int32)
            conf = rng.choice(levels, size=(B, n, L, k)).astype(np.float32)
            idx = rng.integers(0, 3, size=(B, n, L, k)).astype(np.int32)
            tokens = rng.integers(0, 3, size=(B, n, L)).astype(np.int32)
            tokens[rng.random((B, n, L)) < 0.5] = -1
            for mode, trav in itertools.product(MODES, TRAVS):
                _run_both(tokens, parent, committed, conf0, idx0, conf, idx, 0.8, mode, trav)


@pytest.mark.parametrize("tau", [1.0, -0.5, 0.875])
def test_threshold_edges(tau):
    """tau >= 1: pure top-1 decoding; tau < 0: everything at once; tau equal to
    an fp32 confidence value: strict comparison."""
    wl = WORKLOADS[3].with_(V=512)
    d = decode_inputs(wl, 31, tau=tau)
    B, N, L, k = wl.B, wl.N, wl.L, wl.k
    lg = make_logits(d["row_margin"], d["row_top"], wl.V, torch.float32, 31)
    c, i = oracle.confidence_topk(lg.numpy(), k)
    conf = c.astype(np.float32).reshape(B, N, L, k)
    if tau == 0.875:
        conf[..., 0] = np.where(np.arange(L) % 3 == 0, np.float32(0.875), conf[..., 0])
    _run_both(d["tokens"], d["parent"], d["committed"], d["conf0"], d["idx0"], conf,
              i.astype(np.int32).reshape(B, N, L, k), tau, "exact", "greedy")


def test_largest_tree_and_block():
    rng = np.random.default_rng(5)
    B, N, L, k = 3, 64, 64, 8
    parent = np.array([[-1] + [int(rng.integers(-1, n)) for n in range(1, N)] for _ in range(B)], dtype=np.int32)
    parent[0] = np.arange(-1, N - 1)  # one deep chain
    committed = np.full((B, L), -1, dtype=np.int32)
    conf0 = rng.random((B, L, k)).astype(np.float32)
    idx0 = rng.integers(0, 50, size=(B, L, k)).astype(np.int32)
    conf = rng.random((B, N, L, k)).astype(np.float32)
    idx = rng.integers(0, 50, size=(B, N, L, k)).astype(np.int32)
    # plant exact steps along parents so long acceptances happen
    tokens = np.empty((B, N, L), dtype=np.int32)
    for b in range(B):
        for n in range(N):
            q = parent[b, n]
            s, C, I = (committed[b], conf0[b], idx0[b]) if q < 0 else (tokens[b, q], conf[b, q], idx[b, q])
            nxt = oracle.threshold_step(s, C.astype(np.float64), I, 0.7)
            tokens[b, n] = nxt if nxt is not None else s
            if rng.random() < 0.1:
                tokens[b, n, rng.integers(L)] = 7
    for mode, trav in itertools.product(MODES, TRAVS):
        _run_both(tokens, parent, committed, conf0, idx0, conf, idx, 0.7, mode, trav)


def test_invalid_parent_sets_device_status_and_is_treated_as_root():
    tsp.device_status(reset=True)
    B, N, L, k = 1, 3, 4, 3
    tokens = np.full((B, N, L), -1, dtype=np.int32)
    parent = np.array([[-1, 5, 1]], dtype=np.int32)   # parent 5 is out of range
    conf = np.full((B, N, L, k), 0.1, dtype=np.float32)
    idx = np.zeros((B, N, L, k), dtype=np.int32)
    out = tsp.accept(cuda(conf.reshape(-1, k)), cuda(idx.reshape(-1, k)), cuda(tokens), cuda(parent),
                     cuda(np.full((B, L), -1, dtype=np.int32)), cuda(np.full((B, L, k), 0.1, dtype=np.float32)),
                     cuda(np.zeros((B, L, k), dtype=np.int32)), 0.9)
    flags = tsp.device_status(reset=True)
    assert flags & tsp.DEV_BAD_PARENT
    assert out["leaf"].item() == -1
    assert tsp.device_status(reset=True) == 0
