"""Scalar-loop re-derivations used only to pin the oracle on tiny inputs.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

These are deliberately written in a different shape from the vectorised
oracle so that a mistake in one does not repeat in the other:

* ``attention_scalar`` enumerates, for every single query token, the keys it
  may see by walking the parent chain of its own draft (Sec. 3.3 mask rules
  plus tree ancestors), and forms the softmax with ``math.fsum``.
* ``accept_by_paths`` enumerates every root path of the draft tree, keeps the
  paths whose every edge is consistent, and then picks the greedy leaf as the
  lexicographically smallest *maximal* valid path (the walk that always takes
  the lowest-index consistent child ends exactly there) and the longest leaf
  as the valid endpoint with the largest gain (Sec. 3.3 traversal).  Edge
  consistency comes from ``consistent_scalar``, written here from the
  definitions as set comparisons (it imports nothing from the oracle).
"""

import math

MASK = -1


def _is_on_root_path(j, i, parent_row):
    """True when draft j is draft i itself or one of i's ancestors."""
    cur = i
    while cur != -1:
        if cur == j:
            return True
        cur = int(parent_row[cur])
    return False


def attention_scalar(q, k_cache, v_cache, k_draft, v_draft, parent, scale=None, peers=None):
    """Nested-loop attention.  Arrays are nested sequences or numpy arrays with
    the layouts of :func:`oracle.attention.verify_attention`."""
    B = len(q)
    N = len(q[0])
    L = len(q[0][0])
    Hq = len(q[0][0][0])
    D = len(q[0][0][0][0])
    S = len(k_cache[0])
    Hkv = len(k_cache[0][0]) if S > 0 else len(k_draft[0][0][0])
    group = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = [[[[[0.0] * D for _ in range(Hq)] for _ in range(L)] for _ in range(N)] for _ in range(B)]
    for b in range(B):
        for i in range(N):
            for p in range(L):
                for h in range(Hq):
                    g = h // group
                    qv = [float(x) for x in q[b][i][p][h]]
                    keys = []
                    vals = []
                    for s in range(S):
                        keys.append(k_cache[b][s][g])
                        vals.append(v_cache[b][s][g])
                    for j in range(N):
                        extra = peers is not None and (int(peers[b][i]) >> j) & 1
                        if _is_on_root_path(j, i, parent[b]) or extra:
                            for pp in range(L):
                                keys.append(k_draft[b][j][pp][g])
                                vals.append(v_draft[b][j][pp][g])
                    logits = [scale * math.fsum(qv[d] * float(kk[d]) for d in range(D)) for kk in keys]
                    top = max(logits)
                    w = [math.exp(x - top) for x in logits]
                    z = math.fsum(w)
                    for d in range(D):
                        out[b][i][p][h][d] = math.fsum(w[t] * float(vals[t][d]) for t in range(len(w))) / z
    return out


def consistent_scalar(child, parent_state, conf, idx, tau, mode="exact"):
    """Is ``child`` an acceptable next step of ``parent_state`` (Sec. 3.3 verification; Sec. 2.1
    threshold decoding)?  Written as set comparisons over positions:

    * exact: the positions the child unmasks are exactly the threshold step's set (every masked
      position whose top-1 confidence is above tau, or, when there is none, the masked position
      with the largest top-1 confidence, the smaller position on ties), each set to its top-1
      candidate, and every other position is unchanged;
    * top1 / topk: no previously unmasked position changes, at least one masked position is
      unmasked, and each such token is among the first 1 / k candidates of its position.
    """
    L = len(parent_state)
    masked = {p for p in range(L) if parent_state[p] == MASK}
    unchanged_outside = all(child[p] == parent_state[p] for p in range(L) if p not in masked)
    newly = {p for p in masked if child[p] != MASK}
    if not unchanged_outside:
        return False
    if mode == "exact":
        if not masked:
            return False  # a complete block has no next step
        chosen = {p for p in masked if conf[p][0] > tau}
        if not chosen:
            best = max(float(conf[p][0]) for p in masked)
            chosen = {min(p for p in masked if float(conf[p][0]) == best)}
        return newly == chosen and all(child[p] == idx[p][0] for p in chosen)
    width = {"top1": 1, "topk": len(idx[0])}[mode]
    return len(newly) >= 1 and all(child[p] in [idx[p][j] for j in range(width)] for p in newly)


def _gain(state, committed):
    return sum(1 for p in range(len(committed)) if committed[p] == MASK and state[p] != MASK)


def accept_by_paths(tokens, parent, committed, conf0, idx0, conf, idx, tau, mode="exact"):
    """Return (greedy_leaf, longest_leaf) by explicit path enumeration."""
    N = len(tokens)

    def state(q):
        return committed if q == -1 else tokens[q]

    def scores(q):
        return (conf0, idx0) if q == -1 else (conf[q], idx[q])

    def children(q):
        return [c for c in range(N) if int(parent[c]) == q]

    def edge_ok(c):
        q = int(parent[c])
        C, I = scores(q)
        return consistent_scalar([int(t) for t in tokens[c]], [int(t) for t in state(q)], C, I, tau, mode)

    # all root paths (sequences of drafts starting at a child of -1)
    paths = []
    stack = [[c] for c in children(-1)]
    while stack:
        path = stack.pop()
        paths.append(path)
        for c in children(path[-1]):
            stack.append(path + [c])
    valid = [pth for pth in paths if all(edge_ok(c) for c in pth)]
    valid_set = {tuple(pth) for pth in valid}
    maximal = [pth for pth in valid
               if not any(tuple(pth + [c]) in valid_set for c in children(pth[-1]))]
    greedy_leaf = min(maximal)[-1] if maximal else -1

    longest_leaf = -1
    best = -1
    for end in sorted({pth[-1] for pth in valid}):
        g = _gain(tokens[end], committed)
        if g > best:
            best = g
            longest_leaf = end
    return greedy_leaf, longest_leaf


def _bf16(x):
    """Nearest-even bf16 of a float, through fp32 (struct-level bit manipulation)."""
    import struct
    b = struct.unpack("<I", struct.pack("<f", float(x)))[0]
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return struct.unpack("<f", struct.pack("<I", b & 0xFFFFFFFF))[0]


def layer_scalar(x, weights, k_cache, v_cache, parent, Hq, pos0, rms_eps, rope_theta):
    """Nested-loop verification layer (one token, one feature at a time) with the same bf16
    rounding points as :func:`oracle.layer.verify_layer`."""
    B, N, L, hidden = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    D = hidden // Hq
    Hkv = len(k_cache[0][0]) if len(k_cache[0]) else Hq
    inter = len(weights["w_down"])
    W = weights
    out = [[[list(map(float, x[b][n][p])) for p in range(L)] for n in range(N)] for b in range(B)]

    def norm(v, g):
        ms = math.fsum(t * t for t in v) / len(v)
        inv = 1.0 / math.sqrt(ms + rms_eps)
        return [_bf16(v[i] * inv * float(g[i])) for i in range(len(v))]

    def matvec(v, m, cols):
        return [math.fsum(v[i] * float(m[i][j]) for i in range(len(v))) for j in range(cols)]

    qs = [[[None] * L for _ in range(N)] for _ in range(B)]
    ks = [[[None] * L for _ in range(N)] for _ in range(B)]
    vs = [[[None] * L for _ in range(N)] for _ in range(B)]
    for b in range(B):
        for n in range(N):
            for p in range(L):
                xn = norm(out[b][n][p], W["attn_norm"])
                qkv = [_bf16(t) for t in matvec(xn, W["w_qkv"], (Hq + 2 * Hkv) * D)]
                pos = (0 if pos0 is None else int(pos0[b])) + p
                heads = []
                for hh in range(Hq + Hkv):
                    seg = qkv[hh * D:(hh + 1) * D]
                    rot = [0.0] * D
                    for d in range(D // 2):
                        a = pos * rope_theta ** (-2.0 * d / D)
                        rot[d] = _bf16(seg[d] * math.cos(a) - seg[d + D // 2] * math.sin(a))
                        rot[d + D // 2] = _bf16(seg[d + D // 2] * math.cos(a) + seg[d] * math.sin(a))
                    heads.append(rot)
                qs[b][n][p] = heads[:Hq]
                ks[b][n][p] = heads[Hq:]
                vs[b][n][p] = [qkv[(Hq + Hkv + hh) * D:(Hq + Hkv + hh + 1) * D] for hh in range(Hkv)]
    att = attention_scalar(qs, k_cache, v_cache, ks, vs, parent)
    for b in range(B):
        for n in range(N):
            for p in range(L):
                a = [_bf16(t) for hh in range(Hq) for t in att[b][n][p][hh]]
                h = [_bf16(out[b][n][p][i] + t) for i, t in enumerate(matvec(a, W["w_o"], hidden))]
                xn = norm(h, W["mlp_norm"])
                gu = [_bf16(t) for t in matvec(xn, W["w_gate_up"], 2 * inter)]
                act = [_bf16(gu[i] / (1.0 + math.exp(-gu[i])) * gu[inter + i]) for i in range(inter)]
                out[b][n][p] = [_bf16(h[i] + t) for i, t in enumerate(matvec(act, W["w_down"], hidden))]
    return out
