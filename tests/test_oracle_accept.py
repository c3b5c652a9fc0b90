"""Pins for the acceptance oracle (CPU only)."""

import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from synthetic import WORKLOADS, decode_inputs, make_logits, seed_for, torch_dtype

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
M = oracle.MASK


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_golden_threshold_steps():
    g = _load("threshold_step.json")
    for case in g["cases"]:
        conf = [[c] for c in case["conf"]]
        idx = [[t] for t in case["top1"]]
        got = oracle.threshold_step(np.array(case["state"]), conf, idx, case["tau"])
        if case["expected"] is None:
            assert got is None, case["name"]
        else:
            assert got is not None and got.tolist() == case["expected"], case["name"]


def test_golden_consistency_modes():
    for g in _load("consistency.json")["groups"]:
        for case in g["cases"]:
            for mode in ("exact", "top1", "topk"):
                got = oracle.is_consistent(np.array(case["child"]), np.array(g["parent_state"]),
                                           g["conf"], g["idx"], g["tau"], mode)
                assert got == case[mode], (g["note"], case["child"], mode)
                # the path-enumeration pin carries its own consistency rule: it must agree too
                alt = brute.consistent_scalar(case["child"], g["parent_state"], g["conf"], g["idx"], g["tau"], mode)
                assert alt == case[mode], (g["note"], case["child"], mode, "brute")


def test_golden_tree_acceptance():
    g = _load("accept_tree.json")
    exp = g["expected"]
    for key in ("exact/greedy", "exact/longest", "top1/greedy", "top1/longest"):
        mode, trav = key.split("/")
        res = oracle.accept_sequence(np.array(g["tokens"]), np.array(g["parent"]), np.array(g["committed"]),
                                     np.array(g["conf0"]), np.array(g["idx0"]), np.array(g["conf"]),
                                     np.array(g["idx"]), g["tau"], mode, trav)
        e = exp[key]
        assert res["leaf"] == e["leaf"], key
        assert res["on_path"].astype(int).tolist() == e["on_path"], key
        assert res["n_accepted"] == e["n_accepted"], key
        assert res["out_tokens"].tolist() == e["out_tokens"], key
        assert res["hi"].astype(int).tolist() == exp["hi"], key


def _random_state(rng, L, p_mask=0.7):
    s = rng.integers(0, 50, size=L)
    s[rng.random(L) < p_mask] = M
    return s


def test_tau_at_least_one_is_pure_top1_decoding():
    """Theorem 1's setting: with tau >= 1 no confidence can exceed tau, so each
    step unmasks exactly the single most confident masked position."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        L = int(rng.integers(1, 9))
        s = _random_state(rng, L)
        conf = rng.random((L, 2))
        idx = rng.integers(100, 200, size=(L, 2))
        nxt = oracle.threshold_step(s, conf, idx, 1.0)
        masked = np.flatnonzero(s == M)
        if masked.size == 0:
            assert nxt is None
            continue
        changed = np.flatnonzero(nxt != s)
        assert changed.size == 1
        p = changed[0]
        assert conf[p, 0] == conf[masked, 0].max()
        assert nxt[p] == idx[p, 0]


def test_negative_tau_unmasks_everything_at_once():
    rng = np.random.default_rng(12)
    for _ in range(100):
        L = int(rng.integers(1, 9))
        s = _random_state(rng, L)
        conf = rng.random((L, 1))
        idx = rng.integers(100, 200, size=(L, 1))
        nxt = oracle.threshold_step(s, conf, idx, -0.1)
        if (s == M).sum() == 0:
            assert nxt is None
        else:
            assert np.all(nxt != M)
            assert np.array_equal(nxt[s != M], s[s != M])
            assert np.array_equal(nxt[s == M], idx[s == M, 0])


def test_chain_acceptance_is_sequential_threshold_decoding():
    """Invariant 3: on a one-candidate chain, acceptance is exactly sequential
    threshold decoding -- the accepted depth is the first planted step that
    departs from it.  The chain is planted by the generator; its intent is
    realised through logits and judged by the oracle's own confidences."""
    wl = WORKLOADS[1].with_(N=6, parents=(-1, 0, 1, 2, 3, 4), L=12, V=512, alpha=(1.0, 1.0))
    hits = 0
    for seed in range(40):
        d = decode_inputs(wl, seed)
        lg = make_logits(d["row_margin"], d["row_top"], wl.V, torch.float32, seed)
        conf, idx = oracle.confidence_topk(lg.numpy(), 3)
        B, N, L, k = wl.B, wl.N, wl.L, wl.k
        res = oracle.accept_batch(d["tokens"], d["parent"], d["committed"], d["conf0"], d["idx0"],
                                  conf.reshape(B, N, L, k), idx.reshape(B, N, L, k), wl.tau)
        assert res["leaf"][0] == d["planted_leaf"][0]
        hits += int(res["leaf"][0] == N - 1)
        # recompute by hand: walk the chain with threshold_step
        state, C, I = d["committed"][0], d["conf0"][0], d["idx0"][0]
        depth = 0
        for n in range(N):
            nxt = oracle.threshold_step(state, C, I, wl.tau)
            if nxt is None or not np.array_equal(nxt, d["tokens"][0, n]):
                break
            depth = n + 1
            state, C, I = d["tokens"][0, n], conf.reshape(N, L, k)[n], idx.reshape(N, L, k)[n]
        assert res["leaf"][0] == depth - 1
    assert hits > 0  # some chains are accepted to the end


def _all_parent_arrays(n):
    return list(itertools.product(*[range(-1, i) for i in range(n)]))


@pytest.mark.parametrize("mode", ["exact", "top1", "topk"])
def test_traversals_match_path_enumeration(mode):
    """Brute force: greedy leaf = lexicographically smallest maximal valid
    root path; longest leaf = valid endpoint of largest gain (lowest index)."""
    rng = np.random.default_rng({"exact": 21, "top1": 22, "topk": 23}[mode])
    L, k, tau = 3, 2, 0.6
    for n in range(1, 5):
        for par in _all_parent_arrays(n):
            for _ in range(6):
                committed = _random_state(rng, L, 0.9) % 3
                committed[rng.random(L) < 0.8] = M
                conf0 = rng.choice([0.3, 0.5, 0.7, 0.9], size=(L, k))
                idx0 = rng.integers(0, 3, size=(L, k))
                conf = rng.choice([0.3, 0.5, 0.7, 0.9], size=(n, L, k))
                idx = rng.integers(0, 3, size=(n, L, k))
                tokens = np.empty((n, L), dtype=np.int64)
                for c in range(n):
                    base = committed if par[c] == -1 else tokens[par[c]]
                    C, I = (conf0, idx0) if par[c] == -1 else (conf[par[c]], idx[par[c]])
                    nxt = oracle.threshold_step(base, C, I, tau)
                    if nxt is not None and rng.random() < 0.6:
                        tokens[c] = nxt
                    else:
                        t = base.copy()
                        pos = rng.integers(0, L)
                        t[pos] = rng.integers(0, 3) if rng.random() < 0.8 else M
                        tokens[c] = t
                parent = np.array(par)
                g_leaf, l_leaf = brute.accept_by_paths(tokens, parent, committed, conf0, idx0, conf, idx,
                                                       tau, mode)
                rg = oracle.accept_sequence(tokens, parent, committed, conf0, idx0, conf, idx, tau,
                                            mode, "greedy")
                rl = oracle.accept_sequence(tokens, parent, committed, conf0, idx0, conf, idx, tau,
                                            mode, "longest")
                assert rg["leaf"] == g_leaf, (par, mode)
                assert rl["leaf"] == l_leaf, (par, mode)


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_planted_trees_are_accepted_as_planted(cid):
    """The generator plants an intended trajectory (decide-first, from its own
    margins); realised through logits and scored by the oracle's own
    confidences, the oracle must accept exactly the planted leaf."""
    wl = WORKLOADS[cid]
    if wl.V > 4096:
        wl = wl.with_(V=4096)
    for salt in range(3):
        seed = seed_for(cid, salt)
        d = decode_inputs(wl, seed)
        lg = make_logits(d["row_margin"], d["row_top"], wl.V, torch_dtype(wl.logits_dtype), seed)
        conf, idx = oracle.confidence_topk(lg.float().numpy(), wl.k)
        B, N, L, k = wl.B, wl.N, wl.L, wl.k
        res = oracle.accept_batch(d["tokens"], d["parent"], d["committed"], d["conf0"], d["idx0"],
                                  conf.reshape(B, N, L, k), idx.reshape(B, N, L, k), wl.tau)
        assert np.array_equal(res["leaf"], d["planted_leaf"])
        fr = oracle.fragile_states(d["tokens"][0], d["committed"][0], d["conf0"][0],
                                   conf.reshape(B, N, L, k)[0], wl.tau)
        assert not fr.any()


def test_acceptance_depth_matches_planted_level_probabilities():
    """Prop. 1 sanity check: with per-level agreement alpha = (0.85, 0.68) and
    no pruning of rank-0 chains, E[accepted depth] = a1 + a1*a2."""
    wl = WORKLOADS[3].with_(B=1, N=12, level_sizes=(3, 9), V=256)
    depths = []
    for seed in range(300):
        d = decode_inputs(wl, 50000 + seed)
        # intended rank-0 chains are complete in a (3, 9) tree
        leaf = d["planted_leaf"][0]
        depths.append(0 if leaf == -1 else int(d["level"][0, leaf]))
    expect = 0.85 + 0.85 * 0.68
    mean = float(np.mean(depths))
    sd = float(np.std(depths)) / np.sqrt(len(depths))
    assert abs(mean - expect) < 4 * sd + 1e-9


def test_hi_set_is_strict_and_masked_only():
    tokens = np.array([[M, 3, M, M]])
    conf = np.array([[[0.95], [0.99], [0.9], [0.2]]])
    idx = np.zeros((1, 4, 1), dtype=np.int64)
    res = oracle.accept_sequence(tokens, np.array([-1]), np.array([M, M, M, M]), np.full((4, 1), 0.1),
                                 np.zeros((4, 1), dtype=np.int64), conf, idx, 0.9)
    assert res["hi"].astype(int).tolist() == [[1, 0, 0, 0]]


def test_nothing_accepted_falls_back_to_committed_state():
    committed = np.array([M, 7, M])
    tokens = np.array([[1, 7, 2]])
    res = oracle.accept_sequence(tokens, np.array([-1]), committed, np.array([[0.1], [0.1], [0.2]]),
                                 np.array([[9], [9], [9]]), np.zeros((1, 3, 1)),
                                 np.zeros((1, 3, 1), dtype=np.int64), 0.9)
    assert res["leaf"] == -1 and res["n_accepted"] == 0
    assert res["out_tokens"].tolist() == committed.tolist()
    assert not res["on_path"].any()


def test_fragile_state_rule():
    tau = 0.9
    committed = np.array([M, M, 4])
    conf0 = np.array([[0.90005], [0.1], [0.9]])  # masked position within 1e-4 of tau
    tokens = np.array([[M, M, 4], [5, 5, 4]])
    conf = np.array([[[0.5], [0.50005], [0.1]], [[0.1], [0.2], [0.3]]])  # fallback near-tie
    f = oracle.fragile_states(tokens, committed, conf0, conf, tau)
    assert f.tolist() == [True, True, False]


def test_invalid_parent_is_rejected():
    with pytest.raises(ValueError):
        oracle.accept_sequence(np.zeros((2, 2), dtype=int), np.array([-1, 1]), np.array([M, M]),
                               np.zeros((2, 1)), np.zeros((2, 1), dtype=int), np.zeros((2, 2, 1)),
                               np.zeros((2, 2, 1), dtype=int), 0.9)
