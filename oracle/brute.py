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
  as the valid endpoint with the largest gain (Sec. 3.3 traversal).
"""

import math

from .accept import MASK, is_consistent


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
        return is_consistent(tokens[c], state(q), C, I, tau, mode)

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
