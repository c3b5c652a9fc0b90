"""Oracle: threshold decoding step, draft consistency and trajectory acceptance.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Definitions followed:

* Threshold decoding with top-1 fallback (Sec. 2.1, "Parallel decoding
  strategies", strategy 2; the same rule drives Fast-dLLM, the baseline of
  Theorem 1): every masked position whose confidence exceeds tau is unmasked
  with its most likely token; when no position exceeds tau, the single most
  confident masked position is unmasked.  "Exceeds" is strict: Alg. 1 phase 1
  puts confidence > tau in the high set H and confidence <= tau in the low set.
  Equal fallback confidences go to the smallest position (not stated in the
  paper).
* Logit reuse (Sec. 3.1): the confidences that decide a node's next step are
  the ones produced by verifying that node.  The children of the committed
  state (parent -1) are checked against the committed state's own conf/idx,
  i.e. the previous step's logits.
* Verification (Sec. 3.3, "Verification procedure"): a draft block passes
  when its tokens agree with the model's best predictions; the section also
  admits looser checks based on the top-k candidates or on the threshold.
  Three readings:
    - ``exact`` (default): the child equals step_tau(parent) at every
      position.  A chain of exact acceptances reproduces sequential threshold
      decoding, which is the exactness setting of Theorem 1.
    - ``top1``: the child keeps every unmasked token of its parent, unmasks at
      least one new position, and each new token is the parent's top-1
      candidate there.
    - ``topk``: as ``top1`` but each new token may be any of the parent's k
      candidates there.
* Traversal (Sec. 3.3): ``greedy`` walks from the committed state and takes
  the first (lowest-index) consistent child at each level; ``longest`` picks,
  among nodes whose whole root path is consistent, the one that unmasks the
  most positions of the committed state (ties: lowest index).
* Outputs: accepted leaf (-1 if none), on-path flags, number of positions the
  leaf unmasks relative to the committed state, the accepted block state (the
  committed state when nothing is accepted), and hi[n,p] = (position p of draft
  n is still masked and its confidence exceeds tau) -- the high-confidence set
  H of Alg. 1 phase 1 that seeds the next root.

Shapes for one sequence: tokens [N,L] (MASK = -1), parent [N], committed [L],
conf0/idx0 [L,k], conf/idx [N,L,k].
"""

import numpy as np

MASK = -1
MODES = ("exact", "top1", "topk")
TRAVERSALS = ("greedy", "longest")


def threshold_step(state, conf, idx, tau):
    """One threshold-decoding step from block ``state``.

    Returns the new state (a copy), or None when the state has no masked
    position left (the block is complete and cannot be stepped).
    """
    state = np.asarray(state)
    masked = [p for p in range(len(state)) if state[p] == MASK]
    if not masked:
        return None
    chosen = [p for p in masked if conf[p][0] > tau]
    if not chosen:
        best = masked[0]
        for p in masked[1:]:
            if conf[p][0] > conf[best][0]:
                best = p
        chosen = [best]
    new_state = state.copy()
    for p in chosen:
        new_state[p] = idx[p][0]
    return new_state


def is_consistent(child, parent_state, conf, idx, tau, mode="exact"):
    """Is block state ``child`` an acceptable next step of ``parent_state``?

    ``conf``/``idx`` are the parent's [L,k] confidences and candidates.
    """
    child = np.asarray(child)
    parent_state = np.asarray(parent_state)
    if mode == "exact":
        expected = threshold_step(parent_state, conf, idx, tau)
        return expected is not None and bool(np.array_equal(child, expected))
    if mode not in ("top1", "topk"):
        raise ValueError(f"unknown mode {mode!r}")
    k_allowed = 1 if mode == "top1" else len(idx[0])
    unmasked_new = 0
    for p in range(len(child)):
        if parent_state[p] != MASK:
            if child[p] != parent_state[p]:
                return False
        elif child[p] != MASK:
            if child[p] not in list(idx[p][:k_allowed]):
                return False
            unmasked_new += 1
    return unmasked_new >= 1


def _state_and_scores(q, tokens, committed, conf0, idx0, conf, idx):
    if q == -1:
        return committed, conf0, idx0
    return tokens[q], conf[q], idx[q]


def _gain(tokens_n, committed):
    return int(sum(1 for p in range(len(committed)) if committed[p] == MASK and tokens_n[p] != MASK))


def accept_sequence(tokens, parent, committed, conf0, idx0, conf, idx, tau,
                    mode="exact", traversal="greedy"):
    """Acceptance for one sequence; returns a dict of outputs."""
    tokens = np.asarray(tokens)
    parent = np.asarray(parent)
    committed = np.asarray(committed)
    N, L = tokens.shape
    for n in range(N):
        if not (-1 <= int(parent[n]) < n):
            raise ValueError(f"draft {n}: parent {int(parent[n])} breaks -1 <= parent[n] < n")
    if mode not in MODES:
        raise ValueError(f"unknown mode {mode!r}")
    if traversal not in TRAVERSALS:
        raise ValueError(f"unknown traversal {traversal!r}")

    def consistent(c):
        q = int(parent[c])
        s, C, I = _state_and_scores(q, tokens, committed, conf0, idx0, conf, idx)
        return is_consistent(tokens[c], s, C, I, tau, mode)

    leaf = -1
    if traversal == "greedy":
        cur = -1
        while True:
            nxt = -1
            for c in range(N):
                if int(parent[c]) == cur and consistent(c):
                    nxt = c
                    break
            if nxt == -1:
                break
            leaf = nxt
            cur = nxt
    else:
        valid = [False] * N
        for c in range(N):  # parents precede children
            q = int(parent[c])
            valid[c] = consistent(c) and (q == -1 or valid[q])
        best_gain = -1
        for c in range(N):
            if valid[c]:
                g = _gain(tokens[c], committed)
                if g > best_gain:
                    best_gain = g
                    leaf = c

    on_path = np.zeros(N, dtype=bool)
    j = leaf
    while j != -1:
        on_path[j] = True
        j = int(parent[j])
    if leaf == -1:
        n_acc = 0
        out_tokens = committed.copy()
    else:
        n_acc = _gain(tokens[leaf], committed)
        out_tokens = tokens[leaf].copy()
    hi = np.zeros((N, L), dtype=bool)
    for n in range(N):
        for p in range(L):
            hi[n, p] = tokens[n][p] == MASK and conf[n][p][0] > tau
    return {"leaf": leaf, "on_path": on_path, "n_accepted": n_acc,
            "out_tokens": out_tokens, "hi": hi}


def accept_batch(tokens, parent, committed, conf0, idx0, conf, idx, tau,
                 mode="exact", traversal="greedy"):
    """Acceptance for a batch: tokens [B,N,L], parent [B,N], committed [B,L],
    conf0/idx0 [B,L,k], conf/idx [B,N,L,k].  Returns stacked outputs."""
    B = len(tokens)
    res = [accept_sequence(tokens[b], parent[b], committed[b], conf0[b], idx0[b],
                           conf[b], idx[b], tau, mode, traversal) for b in range(B)]
    return {
        "leaf": np.array([r["leaf"] for r in res], dtype=np.int64),
        "on_path": np.stack([r["on_path"] for r in res]),
        "n_accepted": np.array([r["n_accepted"] for r in res], dtype=np.int64),
        "out_tokens": np.stack([r["out_tokens"] for r in res]),
        "hi": np.stack([r["hi"] for r in res]),
    }


def fragile_states(tokens, committed, conf0, conf, tau, eps=1e-4):
    """Flags the block states whose next step is numerically fragile.

    Returns a bool array of length N+1: entry 0 is the committed state, entry
    n+1 is draft n.  A state is fragile when some masked position has
    |conf - tau| < eps (the strict threshold could go either way), or when no
    masked position exceeds tau and the two largest masked confidences are
    within eps (the top-1 fallback could pick either).  Child decisions below a
    fragile state are excluded from bit-exact comparison between
    implementations that compute confidences in different precisions.
    """
    tokens = np.asarray(tokens)
    N = tokens.shape[0]
    flags = np.zeros(N + 1, dtype=bool)
    for q in range(-1, N):
        s = committed if q == -1 else tokens[q]
        C = conf0 if q == -1 else conf[q]
        cm = [float(C[p][0]) for p in range(len(s)) if s[p] == MASK]
        if not cm:
            continue
        if any(abs(c - tau) < eps for c in cm):
            flags[q + 1] = True
            continue
        if not any(c > tau for c in cm) and len(cm) >= 2:
            top = sorted(cm, reverse=True)
            if top[0] - top[1] < eps:
                flags[q + 1] = True
    return flags
