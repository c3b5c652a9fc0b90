"""Pins for the attention oracle (CPU only).

Each test ties ``oracle.verify_attention`` to something other than itself:
a library routine (torch SDPA), an invariant, a closed form, a hand-worked
fixture, or the scalar-loop brute force over every small parent array.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from synthetic import WORKLOADS, attention_inputs, decode_inputs, seed_for

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_inputs(rng, B, N, L, Hq, Hkv, D, S, std=1.0):
    q = rng.standard_normal((B, N, L, Hq, D)) * std
    kc = rng.standard_normal((B, S, Hkv, D))
    vc = rng.standard_normal((B, S, Hkv, D))
    kd = rng.standard_normal((B, N, L, Hkv, D))
    vd = rng.standard_normal((B, N, L, Hkv, D))
    return q, kc, vc, kd, vd


def _all_parent_arrays(n):
    """Every topologically labelled forest on n nodes: parent[i] in {-1..i-1}."""
    return list(itertools.product(*[range(-1, i) for i in range(n)]))


def test_forest_count_matches_enumeration():
    # 1 + 2 + 6 + 24 labelled forests with n <= 4 nodes
    assert sum(len(_all_parent_arrays(n)) for n in range(1, 5)) == 33


@pytest.mark.parametrize("Hq,Hkv,D,S,L", [(2, 2, 8, 5, 3), (4, 2, 16, 7, 4), (3, 1, 8, 0, 5)])
def test_single_draft_equals_plain_bidirectional_attention(Hq, Hkv, D, S, L):
    """Invariant 1: one draft under the committed state is ordinary
    bidirectional attention over [cache ; block] (torch SDPA, fp64, no mask)."""
    rng = np.random.default_rng(1)
    q, kc, vc, kd, vd = _rand_inputs(rng, 2, 1, L, Hq, Hkv, D, S)
    par = np.full((2, 1), -1)
    got = oracle.verify_attention(q, kc, vc, kd, vd, par)
    for b in range(2):
        k_all = np.concatenate([kc[b], kd[b, 0]], axis=0)  # [S+L, Hkv, D]
        v_all = np.concatenate([vc[b], vd[b, 0]], axis=0)
        qt = torch.from_numpy(q[b, 0]).permute(1, 0, 2)            # [Hq, L, D]
        kt = torch.from_numpy(k_all).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
        vt = torch.from_numpy(v_all).permute(1, 0, 2).repeat_interleave(Hq // Hkv, dim=0)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)  # [Hq, L, D]
        np.testing.assert_allclose(got[b, 0], ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_perturbing_non_ancestors_leaves_output_bitwise_unchanged():
    """Invariant 2: a draft's output ignores every non-ancestor draft exactly,
    and changes when an ancestor is perturbed."""
    rng = np.random.default_rng(2)
    B, N, L, Hq, Hkv, D, S = 1, 7, 4, 2, 1, 8, 6
    parent = np.array([[-1, -1, 0, 0, 2, 1, -1]])
    q, kc, vc, kd, vd = _rand_inputs(rng, B, N, L, Hq, Hkv, D, S)
    base = oracle.verify_attention(q, kc, vc, kd, vd, parent)
    anc = oracle.ancestor_sets(parent[0])
    for i in range(N):
        for j in range(N):
            kd2, vd2, q2 = kd.copy(), vd.copy(), q.copy()
            kd2[0, j] += rng.standard_normal(kd2[0, j].shape)
            vd2[0, j] += rng.standard_normal(vd2[0, j].shape)
            if j != i:
                q2[0, j] += 1.0  # another draft's queries never matter either
            out = oracle.verify_attention(q2, kc, vc, kd2, vd2, parent)
            if j in anc[i]:
                assert not np.array_equal(out[0, i], base[0, i]), (i, j)
            else:
                assert np.array_equal(out[0, i], base[0, i]), (i, j)


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_dense_mask_equals_scalar_bruteforce_over_all_small_forests(n):
    """Invariant 4: for every parent array on n <= 4 drafts (L up to 4), the
    dense-mask oracle equals nested-loop attention that walks parent chains."""
    rng = np.random.default_rng(10 + n)
    L = {1: 4, 2: 3, 3: 2, 4: 2}[n]
    Hq, Hkv, D, S = 2, 1, 3, 2
    for par in _all_parent_arrays(n):
        q, kc, vc, kd, vd = _rand_inputs(rng, 1, n, L, Hq, Hkv, D, S, std=2.0)
        parent = np.array([par])
        got = oracle.verify_attention(q, kc, vc, kd, vd, parent)
        ref = np.array(brute.attention_scalar(q, kc, vc, kd, vd, parent))
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12, err_msg=str(par))


def test_zero_query_gives_mean_of_visible_values():
    """Closed form: with q = 0 every visible key gets the same weight, so the
    output is the mean of the visible values (cache + root-path blocks)."""
    rng = np.random.default_rng(3)
    B, N, L, Hq, Hkv, D, S = 1, 5, 3, 2, 2, 4, 4
    parent = np.array([[-1, 0, 1, -1, 3]])
    _, kc, vc, kd, vd = _rand_inputs(rng, B, N, L, Hq, Hkv, D, S)
    q = np.zeros((B, N, L, Hq, D))
    got = oracle.verify_attention(q, kc, vc, kd, vd, parent)
    depth_sets = {0: [0], 1: [0, 1], 2: [0, 1, 2], 3: [3], 4: [3, 4]}
    for i, anc in depth_sets.items():
        for h in range(Hq):
            vals = [vc[0, :, h, :]] + [vd[0, j, :, h, :] for j in anc]
            expect = np.concatenate(vals).mean(axis=0)
            for p in range(L):
                np.testing.assert_allclose(got[0, i, p, h], expect, rtol=1e-13, atol=1e-14)


def test_golden_worked_example():
    with open(os.path.join(GOLDEN, "attention_worked.json")) as f:
        g = json.load(f)
    q = np.array(g["q"]).reshape(1, 2, 1, 1, 1)
    kc = np.array(g["k_cache"]).reshape(1, 1, 1, 1)
    vc = np.array(g["v_cache"]).reshape(1, 1, 1, 1)
    kd = np.array(g["k_draft"]).reshape(1, 2, 1, 1, 1)
    vd = np.array(g["v_draft"]).reshape(1, 2, 1, 1, 1)
    for case in g["cases"]:
        out = oracle.verify_attention(q, kc, vc, kd, vd, np.array([case["parent"]]), scale=g["scale"])
        np.testing.assert_allclose(out.reshape(-1), case["expected"], rtol=1e-13)


def test_all_siblings_mask_is_the_papers_isolation_mask():
    """With every parent -1 a block sees the cache and itself only."""
    m = oracle.trajectory_mask([-1, -1, -1], L=2, S=2)
    expect = np.array([
        [1, 1, 1, 1, 0, 0, 0, 0],
        [1, 1, 1, 1, 0, 0, 0, 0],
        [1, 1, 0, 0, 1, 1, 0, 0],
        [1, 1, 0, 0, 1, 1, 0, 0],
        [1, 1, 0, 0, 0, 0, 1, 1],
        [1, 1, 0, 0, 0, 0, 1, 1],
    ], dtype=bool)
    assert np.array_equal(m, expect)
    m2 = oracle.trajectory_mask([-1, 0, 1], L=1, S=1)
    assert np.array_equal(m2, np.array([[1, 1, 0, 0], [1, 1, 1, 0], [1, 1, 1, 1]], dtype=bool))


def test_gqa_grouping_is_contiguous():
    """Query head h reads K/V head h // (Hq/Hkv): equal to MHA on K/V heads
    repeated contiguously (torch.repeat_interleave)."""
    rng = np.random.default_rng(4)
    B, N, L, Hq, Hkv, D, S = 1, 3, 2, 6, 2, 4, 3
    parent = np.array([[-1, 0, -1]])
    q, kc, vc, kd, vd = _rand_inputs(rng, B, N, L, Hq, Hkv, D, S)
    got = oracle.verify_attention(q, kc, vc, kd, vd, parent)
    rep = lambda a, ax: np.repeat(a, Hq // Hkv, axis=ax)  # noqa: E731
    mha = oracle.verify_attention(q, rep(kc, 2), rep(vc, 2), rep(kd, 3), rep(vd, 3), parent)
    np.testing.assert_array_equal(got, mha)


def test_default_scale_is_inverse_sqrt_head_dim():
    rng = np.random.default_rng(5)
    q, kc, vc, kd, vd = _rand_inputs(rng, 1, 2, 2, 1, 1, 16, 3)
    parent = np.array([[-1, 0]])
    a = oracle.verify_attention(q, kc, vc, kd, vd, parent)
    b = oracle.verify_attention(q, kc, vc, kd, vd, parent, scale=1.0 / math.sqrt(16))
    c = oracle.verify_attention(q, kc, vc, kd, vd, parent, scale=1.0)
    assert np.array_equal(a, b)
    assert not np.allclose(a, c)


def test_bad_parent_arrays_are_rejected():
    with pytest.raises(ValueError):
        oracle.ancestor_sets([0])
    with pytest.raises(ValueError):
        oracle.ancestor_sets([-1, 2, 0])
    with pytest.raises(ValueError):
        oracle.ancestor_sets([-2])


@pytest.mark.parametrize("cid", [3, 4, 5])
def test_full_shape_sharp_inputs_tell_masks_apart(cid):
    """Discriminating power of the full-size GPU check: on one (sequence, head) slice of the
    workload's real shape (cache length, drafts, tree) with sharp inputs, an oracle with a wrong
    mask (ancestors dropped; siblings chained) differs from the right one by more than the
    sharp-input bound on a sizeable share of the elements."""
    from helpers import attn_close
    wl = WORKLOADS[cid]
    parent = decode_inputs(wl.with_(V=64), seed_for(cid))["parent"][:1]
    one = wl.with_(B=1, Hq=wl.Hq // wl.Hkv, Hkv=1)
    q, kc, vc, kd, vd = [t.float().numpy().astype(np.float64) for t in attention_inputs(one, 500 + cid, "sharp")]
    q = q[:, :, :, :1]
    ref = oracle.verify_attention(q, kc, vc, kd, vd, parent)
    wrong = {"siblings_chained": np.arange(-1, wl.N - 1, dtype=np.int32)[None]}
    if (parent >= 0).any():
        wrong["ancestors_dropped"] = np.full_like(parent, -1)
    for name, wp in wrong.items():
        bad = oracle.verify_attention(q, kc, vc, kd, vd, wp)
        aw = oracle.verify_attention(q, kc, np.abs(vc), kd, np.abs(vd), wp)
        ok, _, frac = attn_close(ref, bad, aw)
        assert not ok and frac > 0.05, (name, frac)
