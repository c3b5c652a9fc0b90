"""Pins of the inter-block oracle (trigger, joint-tree peers) and of the attention oracle's
peer visibility, on CPU."""

import json
import os

import numpy as np
import pytest
import torch

from oracle.attention import trajectory_mask, verify_attention, visible_sets
from oracle.brute import attention_scalar
from oracle.interblock import interblock_trigger, interblock_trigger_batch, joint_peers

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "interblock_trigger.json")


def _golden():
    return json.load(open(GOLDEN))


@pytest.mark.parametrize("case", _golden()["cases"], ids=lambda c: c["name"])
def test_trigger_golden(case):
    g = _golden()
    trig, c_t, c_t1 = interblock_trigger(case["state"], case["conf"], g["L"], g["tau"])
    assert trig == case["trigger"] and c_t == pytest.approx(case["c_t"]) and c_t1 == pytest.approx(case["c_t1"])


def test_trigger_batch_matches_single():
    rng = np.random.default_rng(0)
    B, L, k = 20, 8, 3
    state = np.where(rng.random((B, 2 * L)) < 0.5, -1, 3)
    conf = rng.random((B, 2 * L, k)).astype(np.float32)
    trig, c_t, c_t1 = interblock_trigger_batch(state, conf, L, 0.9)
    for b in range(B):
        assert (trig[b], c_t[b], c_t1[b]) == interblock_trigger(state[b], conf[b], L, 0.9)


def test_joint_peers_by_hand():
    # current tree: drafts 0 (root), 1, 2; next tree: drafts 3 (root), 4
    peers = joint_peers(3, 2, 0, 0)
    assert peers == [1 << 3, 1 << 3, 1 << 3, 1 << 0, 1 << 0]
    vis = visible_sets([-1, 0, 0, -1, 3], peers)
    assert vis == [{0, 3}, {0, 1, 3}, {0, 2, 3}, {3, 0}, {3, 4, 0}]


def _inputs(rng, B, N, L, Hq, Hkv, D, S):
    f = lambda *s: rng.standard_normal(s)  # noqa: E731
    return f(B, N, L, Hq, D), f(B, S, Hkv, D), f(B, S, Hkv, D), f(B, N, L, Hkv, D), f(B, N, L, Hkv, D)


def test_zero_peers_change_nothing():
    rng = np.random.default_rng(1)
    x = _inputs(rng, 2, 4, 3, 2, 1, 8, 5)
    parent = np.array([[-1, 0, 0, 1], [-1, -1, 1, 2]])
    a = verify_attention(*x, parent)
    b = verify_attention(*x, parent, peers=np.zeros((2, 4), dtype=np.int64))
    assert np.array_equal(a, b)


def test_all_peers_is_unmasked_attention():
    """Every draft sees every draft: plain softmax attention over all S + N L keys (torch SDPA)."""
    rng = np.random.default_rng(2)
    B, N, L, Hq, Hkv, D, S = 1, 3, 4, 2, 2, 8, 6
    q, kc, vc, kd, vd = _inputs(rng, B, N, L, Hq, Hkv, D, S)
    parent = np.array([[-1, 0, -1]])
    peers = np.full((B, N), (1 << N) - 1, dtype=np.int64)
    out = verify_attention(q, kc, vc, kd, vd, parent, peers=peers)
    for h in range(Hq):
        qq = torch.tensor(q[0, :, :, h, :].reshape(N * L, D))
        kk = torch.tensor(np.concatenate([kc[0, :, h], kd[0, :, :, h].reshape(N * L, D)]))
        vv = torch.tensor(np.concatenate([vc[0, :, h], vd[0, :, :, h].reshape(N * L, D)]))
        ref = torch.nn.functional.scaled_dot_product_attention(qq[None], kk[None], vv[None])[0].numpy()
        assert np.allclose(out[0, :, :, h, :].reshape(N * L, D), ref, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_peers_against_scalar_brute_force(seed):
    rng = np.random.default_rng(10 + seed)
    B, N, L, Hq, Hkv, D, S = 1, 4, 2, 2, 1, 4, 3
    x = _inputs(rng, B, N, L, Hq, Hkv, D, S)
    parent = np.array([[-1, 0, -1, 1]])
    peers = rng.integers(0, 1 << N, (B, N))
    a = verify_attention(*x, parent, peers=peers)
    b = np.array(attention_scalar(*x, parent, peers=peers))
    assert np.allclose(a, b, atol=1e-12)


def test_peer_visibility_is_one_directional_and_exact():
    rng = np.random.default_rng(3)
    B, N, L, Hq, Hkv, D, S = 1, 3, 2, 1, 1, 4, 2
    q, kc, vc, kd, vd = _inputs(rng, B, N, L, Hq, Hkv, D, S)
    parent = np.array([[-1, -1, -1]])
    peers = np.array([[1 << 2, 0, 0]])  # draft 0 sees draft 2, not the other way
    base = verify_attention(q, kc, vc, kd, vd, parent, peers=peers)
    kd2, vd2 = kd.copy(), vd.copy()
    kd2[0, 0] += 1.0
    vd2[0, 0] += 1.0
    moved = verify_attention(q, kc, vc, kd2, vd2, parent, peers=peers)
    assert np.array_equal(base[0, 2], moved[0, 2])   # draft 2 does not see draft 0
    assert np.array_equal(base[0, 1], moved[0, 1])
    kd3 = kd.copy()
    kd3[0, 2] += 1.0
    moved = verify_attention(q, kc, vc, kd3, vd, parent, peers=peers)
    assert not np.allclose(base[0, 0], moved[0, 0])  # draft 0 sees draft 2
    assert trajectory_mask([-1, -1, -1], L, S, [1 << 2, 0, 0])[0, S + 2 * L]
