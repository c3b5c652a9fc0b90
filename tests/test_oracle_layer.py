"""Pins of the verification-layer oracle: bf16 rounding against torch, RMSNorm and rotary
closed forms and invariants, SwiGLU against torch, the residual identity, and the whole layer
against the nested-loop re-derivation (CPU only)."""

import math

import numpy as np
import pytest
import torch

from oracle.brute import layer_scalar
from oracle.layer import bf16_round, linear, rmsnorm, rope, silu, verify_layer


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
