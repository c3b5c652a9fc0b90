"""Oracle: one verification decoder layer around the trajectory-masked attention, and the
dual-cache refresh layer.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The verification step runs every draft block through the model in one concatenated forward
pass (Sec. 3.2 "Complexity analysis"; App. A: only block K/V is recomputed, the dual cache
supplies the rest).  One pre-norm decoder layer of the 8B-shaped diffusion LMs the paper runs
(LLaMA-style blocks: RMSNorm, rotary positions, SwiGLU MLP), over the packed draft tokens:

    xn = rmsnorm(x) * attn_norm;     [q | k | v] = xn @ w_qkv;     q, k rotated;
    x  = x + attention(q, k_cache, v_cache, k, v, parent) @ w_o;
    xn = rmsnorm(x) * mlp_norm;      [g | u] = xn @ w_gate_up;
    x  = x + (silu(g) * u) @ w_down

* rmsnorm(x) = x / sqrt(mean(x^2) + eps) per token.
* Rotary positions: pairs (d, d + D/2) of each q / k head rotate by pos * theta^(-2d/D); token
  p of every draft of a block sits at position pos0[b] + p (the drafts are alternative states
  of the same block, Sec. 3.2 "Tree construction").
* Arithmetic in fp64; values are rounded to bf16 (round to nearest even, through fp32) wherever
  the library stores an activation, so that both sides see the same stored intermediates.

Dual-cache refresh (App. A): at a block boundary the model runs over the whole sequence
(prefix, the block, suffix: T = S + L tokens at positions 0 .. T-1) with bidirectional
attention, and the K / V of the prefix and suffix positions are kept as the cache for the
block's speculation.  :func:`refresh_layer` is the same decoder layer as above over whole
sequences, with full attention in place of the trajectory mask, returning that cache (the
rotated K, as the verification layer expects it).
"""

import numpy as np

from .attention import verify_attention


def bf16_round(a):
    """Round to bf16 (nearest even) through fp32; returns float64."""
    a32 = np.asarray(a, dtype=np.float64).astype(np.float32)
    bits = a32.view(np.uint32).astype(np.uint64)
    rounded = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32).astype(np.float64)


def rmsnorm(x, w, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(w, dtype=np.float64)


def rope(x, pos, theta):
    """x [T, H, D], pos [T]: rotate pairs (d, d + D/2) by pos * theta^(-2d/D)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    inv_freq = theta ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]  # [T, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def linear(x, w, y=None):
    """A projection: x @ w in fp64, plus y when given (the residual add of the O and down
    projections).  The library stores the result rounded once to bf16; this is the exact value."""
    out = np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64)
    return out if y is None else out + np.asarray(y, dtype=np.float64)


def silu(g):
    return g / (1.0 + np.exp(-g))


def verify_layer(x, weights, k_cache, v_cache, parent, Hq, pos0=None, rms_eps=1e-5, rope_theta=500000.0,
                 scale=None):
    """x [B,N,L,hidden] (bf16 values); weights: attn_norm [hidden], w_qkv [hidden, (Hq+2Hkv)D],
    w_o [Hq D, hidden], mlp_norm [hidden], w_gate_up [hidden, 2I], w_down [I, hidden].
    Returns the updated x (float64 holding bf16 values)."""
    r = bf16_round
    x = np.asarray(x, dtype=np.float64)
    B, N, L, hidden = x.shape
    D = hidden // Hq
    Hkv = k_cache.shape[2]
    T = B * N * L
    W = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    inter = W["w_down"].shape[0]
    pos = np.array([(0 if pos0 is None else int(pos0[b])) + p for b in range(B) for _ in range(N) for p in range(L)])

    h = x.reshape(T, hidden)
    xn = r(rmsnorm(h, W["attn_norm"], rms_eps))
    qkv = r(linear(xn, W["w_qkv"]))
    q = qkv[:, :Hq * D].reshape(T, Hq, D)
    k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
    v = qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D)
    q, k = r(rope(q, pos, rope_theta)), r(rope(k, pos, rope_theta))
    a = verify_attention(q.reshape(B, N, L, Hq, D), k_cache, v_cache, k.reshape(B, N, L, Hkv, D),
                         v.reshape(B, N, L, Hkv, D), parent, scale=scale)
    a = r(a).reshape(T, Hq * D)
    h = r(linear(a, W["w_o"], h))
    xn = r(rmsnorm(h, W["mlp_norm"], rms_eps))
    gu = r(linear(xn, W["w_gate_up"]))
    act = r(silu(gu[:, :inter]) * gu[:, inter:])
    h = r(linear(act, W["w_down"], h))
    return h.reshape(B, N, L, hidden)


def full_attention(q, k, v, scale=None):
    """Bidirectional attention of one sequence: q [T, Hq, D], k / v [T2, Hkv, D]; query head h
    reads K / V head h // (Hq / Hkv).  softmax(q k^T * scale) v per head, fp64."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    T, Hq, D = q.shape
    G = Hq // k.shape[1]
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    out = np.empty((T, Hq, D))
    for h in range(Hq):
        s = q[:, h] @ k[:, h // G].T * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        out[:, h] = (p / p.sum(axis=1, keepdims=True)) @ v[:, h // G]
    return out


def refresh_layer(x, weights, block_start, L, Hq, Hkv, rms_eps=1e-5, rope_theta=500000.0, scale=None):
    """x [B, T, hidden] (bf16 values), block_start [B] in [0, T - L].  Returns the updated x and
    the cache (k_cache, v_cache) [B, S, Hkv, D] of the positions outside each block (prefix
    rows, then suffix rows), all float64 holding bf16 values."""
    r = bf16_round
    x = np.asarray(x, dtype=np.float64)
    B, T, hidden = x.shape
    D = hidden // Hq
    S = T - L
    W = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    inter = W["w_down"].shape[0]
    out = np.empty_like(x)
    k_cache = np.empty((B, S, Hkv, D))
    v_cache = np.empty((B, S, Hkv, D))
    pos = np.arange(T)
    for b in range(B):
        h = x[b]
        xn = r(rmsnorm(h, W["attn_norm"], rms_eps))
        qkv = r(linear(xn, W["w_qkv"]))
        q = qkv[:, :Hq * D].reshape(T, Hq, D)
        k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
        v = qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D)
        q, k = r(rope(q, pos, rope_theta)), r(rope(k, pos, rope_theta))
        bs = int(block_start[b])
        keep = np.r_[0:bs, bs + L:T]  # prefix then suffix
        k_cache[b], v_cache[b] = k[keep], v[keep]
        a = r(full_attention(q, k, v, scale)).reshape(T, Hq * D)
        h = r(linear(a, W["w_o"], h))
        xn = r(rmsnorm(h, W["mlp_norm"], rms_eps))
        gu = r(linear(xn, W["w_gate_up"]))
        act = r(silu(gu[:, :inter]) * gu[:, inter:])
        out[b] = r(linear(act, W["w_down"], h))
    return out, k_cache, v_cache
