"""Pins of the tree-construction oracle (Alg. 1) against hand-worked trees, an independently
written closed form, the threshold-decoding step and the acceptance oracle (CPU only)."""

import json
import math
import os

import numpy as np
import pytest

from oracle.accept import accept_sequence, is_consistent, threshold_step
from oracle.tree import MASK, build_tree, build_tree_batch, level_widths

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_build.json")


def _cases():
    return json.load(open(GOLDEN))["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_golden_trees(case):
    conf = np.array(case["conf"], dtype=np.float32)
    idx = np.array(case["idx"])
    tokens, parent, score = build_tree(case["s0"], conf, idx, case["tau"], case["width"], case["depth"],
                                       case["branch"], bool(case["full"]), case.get("branch_deep", 1))
    L = len(case["s0"])
    assert tokens.tolist() == [list(r) for r in np.array(case["tokens"], dtype=np.int64).reshape(-1, L)]
    assert parent.tolist() == case["parent"]
    expect = [sum(math.log(float(conf[p][j])) for p, j in terms) for terms in case["score_terms"]]
    assert np.allclose(score, expect, rtol=0, atol=1e-12)


def random_state(rng, L, k, p_mask=0.7, tau=0.9, ties=False):
    s0 = np.where(rng.random(L) < p_mask, MASK, rng.integers(0, 1000, L))
    top = rng.random(L) ** 0.5
    if ties:
        top = np.round(top * 4) / 4  # many equal confidences
    conf = np.zeros((L, k), dtype=np.float32)
    for p in range(L):
        rest = np.minimum(np.sort(rng.random(k - 1))[::-1] * (1 - top[p]) / max(k - 1, 1), top[p])
        conf[p] = np.concatenate([[top[p]], rest]).astype(np.float32)
    idx = np.stack([rng.permutation(1000)[:k] for _ in range(L)])
    return s0, conf, idx


def closed_form(s0, conf, idx, tau, width, depth, branch, full):
    """The same tree derived directly: rank the low-confidence positions once; level 1 takes
    the first-ranked position's top `branch` candidates (kept: the first w_1), level l >= 2
    extends the first w_l nodes of level l-1 at the l-th ranked position with its top-1."""
    L = len(s0)
    masked = [p for p in range(L) if s0[p] == MASK]
    high = [p for p in masked if conf[p][0] > tau]
    ranked = sorted([p for p in masked if conf[p][0] <= tau], key=lambda p: (-float(conf[p][0]), p))
    root = np.array(s0, dtype=np.int64)
    for p in high:
        root[p] = idx[p][0]
    tokens, parent = [], []
    if high:
        tokens.append(root.copy())
        parent.append(-1)
    if not masked:
        return tokens, parent
    prev = []  # node indices of the previous level
    for level in range(1, depth + 1):
        if level > len(ranked):
            break
        p = ranked[level - 1]
        w = width if full else max(width - level + 1, 1)
        if level == 1:
            base = 0 if high else -1
            for j in range(min(branch, w)):
                t = root.copy()
                t[p] = idx[p][j]
                tokens.append(t)
                parent.append(base)
                prev.append(len(tokens) - 1)
        else:
            cur = []
            for node in prev[:w]:
                t = tokens[node].copy()
                t[p] = idx[p][0]
                tokens.append(t)
                parent.append(node)
                cur.append(len(tokens) - 1)
            prev = cur
    return tokens, parent


@pytest.mark.parametrize("seed", range(40))
def test_matches_closed_form(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 20))
    k = int(rng.integers(1, 5))
    tau = float(rng.choice([0.5, 0.8, 0.9, 0.99]))
    width, depth = int(rng.integers(1, 5)), int(rng.integers(0, 6))
    branch = int(rng.integers(1, k + 1))
    full = bool(rng.integers(0, 2))
    s0, conf, idx = random_state(rng, L, k, tau=tau, ties=seed % 3 == 0)
    tokens, parent, _ = build_tree(s0, conf, idx, tau, width, depth, branch, full)
    t2, p2 = closed_form(s0, conf, idx, tau, width, depth, branch, full)
    assert parent.tolist() == p2
    assert tokens.tolist() == [list(t) for t in t2]


@pytest.mark.parametrize("seed", range(20))
def test_structure_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    L, k, tau = 16, 3, 0.9
    s0, conf, idx = random_state(rng, L, k, tau=tau)
    tokens, parent, score = build_tree(s0, conf, idx, tau, 3, 4, 3, False)
    if not (s0 == MASK).any():
        assert len(parent) == 0
        return
    # the first node is one threshold-decoding step of s0
    assert np.array_equal(tokens[0], threshold_step(s0, conf, idx, tau))
    high = (s0 == MASK) & (conf[:, 0] > tau)
    for n in range(len(parent)):
        q = int(parent[n])
        assert -1 <= q < n
        if q == -1 and n == 0 and high.any():
            continue  # the root node
        base = s0.copy() if q == -1 else tokens[q]
        if q == -1:
            base[high] = idx[high, 0]
        diff = np.flatnonzero(tokens[n] != base)
        assert len(diff) == 1 and base[diff[0]] == MASK  # one masked position filled per edge
        p = diff[0]
        j = list(idx[p]).index(tokens[n][p])
        base_score = 0.0 if q == -1 else score[q]
        assert score[n] == pytest.approx(base_score + math.log(float(conf[p][j])), abs=1e-12)
    assert len(parent) <= int(high.any()) + sum(level_widths(3, 4, False))


@pytest.mark.parametrize("seed", range(20))
def test_static_model_acceptance_follows_top1_chain(seed):
    """If every node's own logits equal those the tree was built from, exact greedy acceptance
    walks the top-1 chain: |H| positions at the root plus one position per level."""
    rng = np.random.default_rng(200 + seed)
    L, k, tau = 12, 3, 0.9
    s0, conf, idx = random_state(rng, L, k, tau=tau)
    depth = int(rng.integers(1, 5))
    tokens, parent, _ = build_tree(s0, conf, idx, tau, 3, depth, 3, bool(seed % 2))
    N = len(parent)
    if N == 0:
        return
    res = accept_sequence(tokens, parent, s0, conf, idx, np.repeat(conf[None], N, 0), np.repeat(idx[None], N, 0),
                          tau, "exact", "greedy")
    masked = s0 == MASK
    n_high = int((masked & (conf[:, 0] > tau)).sum())
    n_low = int((masked & (conf[:, 0] <= tau)).sum())
    assert res["n_accepted"] == n_high + min(depth, n_low)
    # the accepted leaf sits on the first-generated chain (candidate 0 everywhere)
    leaf = res["leaf"]
    assert leaf >= 0
    j = leaf
    while j != -1:
        q = int(parent[j])
        siblings = [c for c in range(N) if int(parent[c]) == q]
        assert j == siblings[0]
        j = q


def test_batch_padding_is_never_consistent():
    rng = np.random.default_rng(7)
    B, L, k, n_max = 3, 8, 3, 12
    states, confs, idxs = zip(*[random_state(rng, L, k) for _ in range(B)])
    state = np.stack(states)
    state[2] = np.arange(L)  # complete block: empty tree
    conf0, idx0 = np.stack(confs), np.stack(idxs)
    tokens, parent, n_nodes, score = build_tree_batch(state, None, None, None, conf0, idx0, 0.9, 3, 3, 3, False, n_max)
    assert n_nodes[2] == 0
    for b in range(B):
        for n in range(int(n_nodes[b]), n_max):
            assert np.array_equal(tokens[b, n], state[b]) and parent[b, n] == -1 and score[b, n] == -np.inf
            for mode in ("exact", "top1", "topk"):
                assert not is_consistent(tokens[b, n], state[b], conf0[b], idx0[b], 0.9, mode)


def test_gather_uses_leaf_rows():
    rng = np.random.default_rng(9)
    L, k, N = 6, 2, 4
    s0, c, i = random_state(rng, L, k)
    conf = np.stack([random_state(rng, L, k)[1] for _ in range(N)])[None]
    idx = np.stack([random_state(rng, L, k)[2] for _ in range(N)])[None]
    t_leaf, p_leaf, n_leaf, _ = build_tree_batch(s0[None], np.array([2]), conf, idx, c[None], i[None],
                                                 0.9, 2, 2, 2, False, 8)
    t_ref, p_ref, _ = build_tree(s0, conf[0, 2], idx[0, 2], 0.9, 2, 2, 2, False)
    assert n_leaf[0] == len(p_ref) and np.array_equal(t_leaf[0, :len(p_ref)], t_ref)
    t_c, _, n_c, _ = build_tree_batch(s0[None], np.array([-1]), conf, idx, c[None], i[None], 0.9, 2, 2, 2, False, 8)
    t_ref, p_ref, _ = build_tree(s0, c, i, 0.9, 2, 2, 2, False)
    assert n_c[0] == len(p_ref) and np.array_equal(t_c[0, :len(p_ref)], t_ref)


@pytest.mark.parametrize("seed", range(20))
def test_deeper_branching_prunes_to_the_best(seed):
    """With several children per node below the first level (the ablation's top-2 policy), each
    level holds the w_l best children of the kept nodes of the level above: none of the
    children left out scores higher than a kept one, and kept nodes come best first."""
    rng = np.random.default_rng(300 + seed)
    L, k, tau = 10, 4, 0.9
    s0, conf, idx = random_state(rng, L, k, tau=tau, ties=seed % 4 == 0)
    W, D, bd = int(rng.integers(1, 5)), int(rng.integers(1, 5)), int(rng.integers(2, k + 1))
    full = bool(seed % 2)
    tokens, parent, score = build_tree(s0, conf, idx, tau, W, D, int(rng.integers(1, k + 1)), full, bd)
    high = (s0 == MASK) & (conf[:, 0] > tau)
    depth_of = {}
    for n in range(len(parent)):
        q = int(parent[n])
        depth_of[n] = 0 if (q == -1 and n == 0 and high.any()) else (1 if q == -1 else depth_of[q] + 1)
    widths = level_widths(W, D, full)
    for level in range(2, D + 1):
        kept = [n for n in depth_of if depth_of[n] == level]
        parents = [n for n in depth_of if depth_of[n] == level - 1]
        if not kept:
            continue
        assert len(kept) <= widths[level - 1]
        assert all(score[a] >= score[b] for a, b in zip(kept, kept[1:]))
        # every child the parents could generate, scored like the oracle
        cands = []
        for q in parents:
            masked_low = [p for p in range(L) if tokens[q][p] == MASK and conf[p][0] <= tau]
            p = min(masked_low, key=lambda x: (-float(conf[x][0]), x))
            for j in range(bd):
                cands.append(score[q] + math.log(float(conf[p][j])))
        worst_kept = min(score[n] for n in kept)
        assert sum(1 for c in cands if c > worst_kept) <= len(kept) - 1
