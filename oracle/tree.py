"""Oracle: confidence-stratified trajectory tree construction (Alg. 1).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Follows Alg. 1 (Sec. 3.2, "Tree construction" and "Algorithm") step by step: phase 1
stratifies the masked positions of a block state by confidence, phase 2 expands the tree level
by level (top-k at the first level, top-1 deeper, each level pruned to a width).  The paper
names GenerateTopK, GenerateTop1 and PruneByConfidence without defining them; the readings
taken here are:

* Inputs: the block state ``s0`` to extend and the [L,k] confidences / candidates of the
  logits produced at that state (logit reuse, Sec. 3.1: the verification pass that accepted
  the state also scored it).
* Phase 1: H = masked positions with conf > tau (strict), Low = masked positions with
  conf <= tau.  The root is s0 with every position of H set to its top-1 token.  When H is
  empty the root equals s0 and is not emitted as a node: the first level then hangs off the
  committed state (parent -1).  When H is not empty the root is node 0 with parent -1.
* A node's candidate position: its highest-confidence masked position of Low (ties to the
  smaller position).
* GenerateTopK(n, Low, k): ``branch`` children; child j sets the candidate position to its
  j-th candidate token.  With H empty, child 0 is exactly one threshold-decoding step of s0
  (the top-1 fallback), so an exact-mode acceptance can always advance.
* GenerateTop1(n, Low): one child setting the candidate position to its top-1 token.  The
  expansion ablation (App. C, "full top-2") expands every level with the top 2: ``branch_deep``
  children per node below the first level (1 = the hybrid policy).
* A node's score: the sum of log conf of the candidates chosen on its path below the root
  (root 0).  PruneByConfidence(frontier, w) keeps the w highest scores, ties to generation
  order.
* Widths: hybrid w_l = max(W - l + 1, 1) for l = 1..D (W2D2 -> 2+1 = 3 children blocks,
  W3D3 -> 3+2+1 = 6: the n of the paper's W x D(n) notation); full w_l = W (W3D3(9)).
* Node order: breadth first, each level in kept order; parent = index of the generating node.
"""

import math

import numpy as np

MASK = -1


def level_widths(width, depth, full):
    """Kept nodes per expansion level l = 1..depth (before running out of positions)."""
    return [width if full else max(width - l + 1, 1) for l in range(1, depth + 1)]


def _rank_key(p, conf):
    return (-float(conf[p][0]), p)


def _candidate_position(state, low, conf):
    """Highest-confidence still-masked position of the low set (ties: smaller position)."""
    cands = [p for p in low if state[p] == MASK]
    if not cands:
        return None
    return min(cands, key=lambda p: _rank_key(p, conf))


def build_tree(s0, conf, idx, tau, width, depth, branch, full=False, branch_deep=1):
    """Builds the draft tree for one sequence.

    s0: [L] block state (MASK = -1); conf/idx: [L,k] top-k confidences / candidates at s0.
    Returns (tokens [N,L] int64, parent [N] int64, score [N] float64).
    """
    s0 = np.asarray(s0)
    L = len(s0)
    k = len(idx[0]) if L else 0
    if not 1 <= branch <= max(k, 1) or not 1 <= branch_deep <= max(k, 1):
        raise ValueError("branch and branch_deep must be in 1..k")
    # Phase 1: confidence stratification
    masked = [p for p in range(L) if s0[p] == MASK]
    high = [p for p in masked if conf[p][0] > tau]
    low = [p for p in masked if conf[p][0] <= tau]
    root = s0.copy()
    for p in high:
        root[p] = idx[p][0]

    tokens, parent, score = [], [], []
    if high:
        tokens.append(root.copy())
        parent.append(-1)
        score.append(0.0)
        frontier = [(0, root, 0.0)]  # (node index, state, score)
    else:
        frontier = [(-1, root, 0.0)]  # the root is the committed state itself
    if not masked:
        return _pack(tokens, parent, score, L)

    # Phase 2: speculative expansion
    widths = level_widths(width, depth, full)
    for level in range(1, depth + 1):
        next_frontier = []
        for node, state, sc in frontier:
            p = _candidate_position(state, low, conf)
            if p is None:
                continue
            n_children = branch if level == 1 else branch_deep  # GenerateTopK at the root, GenerateTop1 deeper
            for j in range(n_children):
                child = state.copy()
                child[p] = idx[p][j]
                next_frontier.append((node, child, sc + math.log(conf[p][j]) if conf[p][j] > 0 else -math.inf))
        # PruneByConfidence: highest scores first, ties in generation order
        order = sorted(range(len(next_frontier)), key=lambda i: (-next_frontier[i][2], i))
        kept = [next_frontier[i] for i in order[:widths[level - 1]]]
        frontier = []
        for par, state, sc in kept:
            tokens.append(state)
            parent.append(par)
            score.append(sc)
            frontier.append((len(tokens) - 1, state, sc))
        if not frontier:
            break
    return _pack(tokens, parent, score, L)


def _pack(tokens, parent, score, L):
    t = np.array(tokens, dtype=np.int64).reshape(len(tokens), L)
    return t, np.array(parent, dtype=np.int64), np.array(score, dtype=np.float64)


def gather_state_scores(leaf, conf, idx, conf0, idx0):
    """conf/idx of the state a tree is built from: the accepted leaf's rows of the verified
    tree (conf/idx [N,L,k]), or the committed state's conf0/idx0 when nothing was accepted."""
    if leaf >= 0:
        return np.asarray(conf)[leaf], np.asarray(idx)[leaf]
    return np.asarray(conf0), np.asarray(idx0)


def build_tree_batch(state, leaf, conf, idx, conf0, idx0, tau, width, depth, branch, full, n_max, branch_deep=1):
    """Batched form with the library's output layout: tokens [B,n_max,L], parent [B,n_max],
    n_nodes [B], score [B,n_max]; slots past n_nodes hold the state itself, parent -1,
    score -inf (a copy of the state is never a consistent child)."""
    state = np.asarray(state)
    B, L = state.shape
    tokens = np.repeat(state[:, None, :], n_max, axis=1).astype(np.int64)
    parent = np.full((B, n_max), -1, dtype=np.int64)
    score = np.full((B, n_max), -np.inf)
    n_nodes = np.zeros(B, dtype=np.int64)
    for b in range(B):
        lf = int(leaf[b]) if leaf is not None else -1
        C, I = gather_state_scores(lf, None if conf is None else conf[b], None if idx is None else idx[b],
                                   conf0[b], idx0[b])
        t, p, s = build_tree(state[b], C, I, tau, width, depth, branch, full, branch_deep)
        n = len(p)
        if n > n_max:
            raise ValueError("tree larger than n_max")
        tokens[b, :n] = t
        parent[b, :n] = p
        score[b, :n] = s
        n_nodes[b] = n
    return tokens, parent, n_nodes, score
