"""Pins of the verification-layer oracle: bf16 rounding against torch, RMSNorm and rotary
closed forms and invariants, SwiGLU against torch, the residual identity, and the whole layer
against the nested-loop re-derivation; of the refresh layer: full attention against torch's
SDPA, the cache's dependence on its own positions only, and agreement with the verification
layer for the block's root state (CPU only)."""

import math

import numpy as np
import pytest
import torch

from oracle.brute import layer_scalar
from oracle.layer import bf16_round, full_attention, linear, refresh_layer, rmsnorm, rope, silu, verify_layer


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000) * 10 ** rng.uniform(-5, 5, 10000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.0078125, 1.005859375, 65504.0]])
    ref = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_round(x), ref)


def test_rmsnorm_closed_form():
    for c in (0.5, -3.0, 10.0):
        x = np.full((1, 64), c)
        w = np.linspace(0.5, 1.5, 64)
        out = rmsnorm(x, w, 1e-5)
        assert np.allclose(out[0], np.sign(c) / math.sqrt(1 + 1e-5 / c ** 2) * w, rtol=1e-14)


def test_rope_invariants():
    rng = np.random.default_rng(1)
    T, H, D, theta = 6, 2, 16, 10000.0
    q = rng.standard_normal((T, H, D))
    assert np.allclose(rope(q, np.zeros(T), theta), q, atol=0)            # position 0: identity
    pos = rng.integers(0, 5000, T)
    r = rope(q, pos, theta)
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(q, axis=-1))  # rotations
    # relative positions: <rope(q, m), rope(k, n)> depends on m - n only
    k = rng.standard_normal((1, H, D))
    qq = q[:1]
    a = (rope(qq, np.array([700]), theta) * rope(k, np.array([500]), theta)).sum(-1)
    b = (rope(qq, np.array([1200]), theta) * rope(k, np.array([1000]), theta)).sum(-1)
    assert np.allclose(a, b, atol=1e-9)


def test_silu_matches_torch():
    g = np.linspace(-20, 20, 401)
    assert np.allclose(silu(g), torch.nn.functional.silu(torch.tensor(g)).numpy(), rtol=1e-14, atol=1e-300)


def test_linear_against_loops_and_identity():
    rng = np.random.default_rng(3)
    x, w, y = rng.standard_normal((3, 5)), rng.standard_normal((5, 4)), rng.standard_normal((3, 4))
    loops = [[sum(x[i][k] * w[k][j] for k in range(5)) + y[i][j] for j in range(4)] for i in range(3)]
    assert np.allclose(linear(x, w, y), loops, rtol=1e-14, atol=1e-14)
    assert np.array_equal(linear(x, np.eye(5)), x)
    assert np.array_equal(linear(x, np.zeros((5, 4)), y), y)


def _weights(rng, hidden, Hq, Hkv, D, inter, zero_out=False):
    f = lambda *s: bf16_round(rng.standard_normal(s) / math.sqrt(s[0]))  # noqa: E731
    w = {"attn_norm": bf16_round(1 + 0.1 * rng.standard_normal(hidden)), "w_qkv": f(hidden, (Hq + 2 * Hkv) * D),
         "w_o": f(Hq * D, hidden), "mlp_norm": bf16_round(1 + 0.1 * rng.standard_normal(hidden)),
         "w_gate_up": f(hidden, 2 * inter), "w_down": f(inter, hidden)}
    if zero_out:
        w["w_o"] = np.zeros_like(w["w_o"])
        w["w_down"] = np.zeros_like(w["w_down"])
    return w


def test_residual_identity():
    rng = np.random.default_rng(2)
    B, N, L, Hq, Hkv, D, S, inter = 1, 3, 4, 2, 1, 8, 5, 32
    x = bf16_round(rng.standard_normal((B, N, L, Hq * D)))
    w = _weights(rng, Hq * D, Hq, Hkv, D, inter, zero_out=True)
    kc, vc = bf16_round(rng.standard_normal((B, S, Hkv, D))), bf16_round(rng.standard_normal((B, S, Hkv, D)))
    out = verify_layer(x, w, kc, vc, np.array([[-1, 0, 0]]), Hq, pos0=np.array([9]))
    assert np.array_equal(out, x)


@pytest.mark.parametrize("seed", range(3))
def test_layer_against_scalar_loops(seed):
    rng = np.random.default_rng(10 + seed)
    B, N, L, Hq, Hkv, D, S, inter = 1, 3, 2, 2, 1, 4, 3, 8
    x = bf16_round(rng.standard_normal((B, N, L, Hq * D)))
    w = _weights(rng, Hq * D, Hq, Hkv, D, inter)
    kc, vc = bf16_round(rng.standard_normal((B, S, Hkv, D))), bf16_round(rng.standard_normal((B, S, Hkv, D)))
    parent = np.array([[-1, 0, -1]])
    pos0 = np.array([int(rng.integers(0, 100))])
    a = verify_layer(x, w, kc, vc, parent, Hq, pos0=pos0, rms_eps=1e-5, rope_theta=10000.0)
    b = np.array(layer_scalar(x, w, kc, vc, parent, Hq, pos0, 1e-5, 10000.0))
    # identical rounding points; the two differ only in summation order (fp64), so they agree
    # except where a value lands within an ulp of a bf16 rounding boundary
    frac_equal = float(np.mean(a == b))
    assert frac_equal > 0.95, frac_equal
    assert np.allclose(a, b, rtol=2e-2, atol=2e-2)


def test_full_attention_matches_torch_sdpa():
    rng = np.random.default_rng(20)
    T, Hq, Hkv, D = 11, 4, 2, 16
    q, k, v = rng.standard_normal((T, Hq, D)), rng.standard_normal((T, Hkv, D)), rng.standard_normal((T, Hkv, D))
    got = full_attention(q, k, v, scale=0.3)
    tq = torch.tensor(q).permute(1, 0, 2)
    tk = torch.tensor(np.repeat(k, 2, axis=1)).permute(1, 0, 2)
    tv = torch.tensor(np.repeat(v, 2, axis=1)).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=0.3).permute(1, 0, 2).numpy()
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


def _refresh_case(seed, B=1, S=9, L=4, Hq=2, Hkv=1, D=8, inter=16):
    rng = np.random.default_rng(seed)
    x = bf16_round(rng.standard_normal((B, S + L, Hq * D)))
    return rng, x, _weights(rng, Hq * D, Hq, Hkv, D, inter)


def test_refresh_cache_depends_on_its_own_positions_only():
    rng, x, w = _refresh_case(21)
    L, Hq, Hkv = 4, 2, 1
    _, kc, vc = refresh_layer(x, w, [3], L, Hq, Hkv)
    # the block's own rows do not reach the cache
    x2 = x.copy()
    x2[0, 3:7] = bf16_round(rng.standard_normal((4, x.shape[2])))
    _, kc2, vc2 = refresh_layer(x2, w, [3], L, Hq, Hkv)
    assert np.array_equal(kc, kc2) and np.array_equal(vc, vc2)
    # a prefix row changes its own cache row only; the suffix starts after the block
    x3 = x.copy()
    x3[0, 1] = bf16_round(rng.standard_normal(x.shape[2]))
    _, kc3, vc3 = refresh_layer(x3, w, [3], L, Hq, Hkv)
    changed = np.any(kc3 != kc, axis=(0, 2, 3)) | np.any(vc3 != vc, axis=(0, 2, 3))
    assert changed.tolist() == [s == 1 for s in range(9)]
    x4 = x.copy()
    x4[0, 10] = bf16_round(rng.standard_normal(x.shape[2]))  # position 10 = cache row 6
    _, kc4, _ = refresh_layer(x4, w, [3], L, Hq, Hkv)
    assert np.any(kc4 != kc, axis=(0, 2, 3)).tolist() == [s == 6 for s in range(9)]


def test_refresh_positions_rotate_identical_rows():
    """Identical token rows at every position: V rows are identical, K rows are rotations of one
    vector (same norm per head, different values), so the positions are applied."""
    rng, x, w = _refresh_case(22)
    x[0, :] = x[0, 0]
    _, kc, vc = refresh_layer(x, w, [0], 4, 2, 1)
    assert np.all(vc == vc[:, :1])
    norms = np.linalg.norm(kc, axis=-1)
    assert np.allclose(norms, norms[:, :1], rtol=2e-2)
    assert len({kc[0, s].tobytes() for s in range(kc.shape[1])}) == kc.shape[1]


def test_refresh_then_verify_root_state_agrees():
    """The dual cache's contract: verifying the block's current state (one draft, no parent)
    against the refreshed cache, at positions block_start + p, gives the refresh layer's own
    output for the block rows -- two different attention paths over the same visible keys."""
    rng, x, w = _refresh_case(23, B=2, S=10, L=5, Hq=2, Hkv=2, D=8, inter=16)
    bs = [4, 10]
    out, kc, vc = refresh_layer(x, w, bs, 5, 2, 2)
    for b in range(2):
        xb = x[b:b + 1, bs[b]:bs[b] + 5][:, None]  # [1, 1, L, hidden]
        ver = verify_layer(xb, w, kc[b:b + 1], vc[b:b + 1], np.array([[-1]]), 2, pos0=np.array([bs[b]]))
        ref = out[b, bs[b]:bs[b] + 5]
        assert np.allclose(ver[0, 0], ref, rtol=2 ** -7, atol=2 ** -7 * np.abs(ref).max())
        assert np.mean(ver[0, 0] == ref) > 0.95
