"""Seeded synthetic workloads for the trajectory-verification step.

This module builds inputs only.  It holds none of the step's arithmetic (no
attention, no softmax confidence, no top-k selection, no acceptance): it
*plants* an intended outcome with its own random draws and then constructs
tensors that realise it.  Both the GPU path and the CPU oracle consume the
exact same bits it returns.

Workloads (shapes of an 8B-class bidirectional diffusion LM, one layer):

  id  name            B   N   L  Hq Hkv   D  cache (prefix+suffix)  vocab   logits  tree
  1   tiny-fp32       1   4   8   4   4  64  128+64                 1000    fp32    root + 3 children
  2   8b-siblings     1   8  32  32  32 128  512+224                126464  bf16    8 siblings
  3   8b-tree         1  32  32  32  32 128  1024+480               126464  bf16    3-ary, levels 3+9+20
  4   gqa-lookahead   1  16  64  28   4 128  1536+512               152064  bf16    16 siblings
  5   8b-batched     16  64  32  32  32 128  3584+512               126464  bf16    3-ary, levels 3+9+27+25

Recipe:
* Attention tensors q, k_cache, v_cache, k_draft, v_draft ~ N(0,1)/sqrt(D),
  rounded to bf16 (round-to-nearest-even).  Variant "sharp": q ~ 3 N(0,1),
  k, v ~ N(0,1), so attention weights are far from uniform.
* Draft trees: BFS order (parent[n] < n).  3-ary trees keep, per level, the
  children with the largest planted path weight (rank weights 0.6/0.25/0.15
  times log-normal noise), so rank-0 chains survive pruning most often.
* Committed block state: each position masked with probability 0.75, at
  least min(4, L) masked; unmasked positions hold random token ids.
* Per block state q and position p the generator draws a margin m ~ U(0, m_max)
  and three distinct candidate tokens (t1, t2, t3).  A logit row for that
  position is N(0,1) noise over the vocabulary with t2, t3 raised just above
  the noise maximum (+0.5, +0.25) and t1 set to log(sum of exp of every other
  entry) + m, so that t1's probability is sigmoid(m) before rounding and the
  three largest entries are t1 > t2 > t3 by construction ("lse" mode).
  "raw" mode instead adds m to t1's own noise value (every row is then far
  below any useful threshold); "ties" mode draws every entry from a grid of
  eight bf16-exact values (many exact ties, nothing planted).
* The committed state's confidences/candidates (the previous step's output)
  are planted directly: conf0 = (sigmoid(m), 0.3(1-sigmoid(m)), 0.2(1-sigmoid(m))),
  idx0 = (t1, t2, t3).
* Intended next step of a state: the masked positions whose planted
  probability sigmoid(m) clears tau, else the masked position with the largest
  margin.  With ``gap > 0`` margins within ``gap`` (in logit units) of
  logit(tau) are redrawn and the fallback winner is kept ``gap`` clear of the
  runner-up, so bf16 rounding cannot change the intent.
* Draft tokens: the rank-0 child of a state is its intended next step with
  probability alpha (0.85 at level 1, 0.68 deeper: the paper's measured
  per-level acceptance), otherwise the same with one newly unmasked token
  replaced by t2; rank r >= 1 children replace the first newly unmasked token
  by t_{r+1} (top-3 branching).  ``planted_leaf`` records the deepest node
  reached by following intended rank-0 children.

The paper's benchmarks (GSM8K, MATH, HumanEval, MBPP, IFEval) and model
weights are not available; these seeded inputs stand in for them.
"""

from dataclasses import dataclass, field
import math

import numpy as np
import torch

MASK = -1


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    B: int
    N: int
    L: int
    Hq: int
    Hkv: int
    D: int
    S_prefix: int
    S_suffix: int
    V: int
    logits_dtype: str          # "bf16" or "f32"
    margin_max: float
    parents: tuple = None      # explicit parent array for every sequence
    level_sizes: tuple = None  # 3-ary BFS tree level sizes
    tau: float = 0.9
    k: int = 3
    alpha: tuple = (0.85, 0.68)
    extra: dict = field(default_factory=dict)

    @property
    def S(self):
        return self.S_prefix + self.S_suffix

    @property
    def rows(self):
        return self.B * self.N * self.L

    def with_(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


WORKLOADS = {
    1: Workload(1, "tiny-fp32", B=1, N=4, L=8, Hq=4, Hkv=4, D=64, S_prefix=128, S_suffix=64,
                V=1000, logits_dtype="f32", margin_max=4.0, parents=(-1, 0, 0, 0)),
    2: Workload(2, "8b-siblings", B=1, N=8, L=32, Hq=32, Hkv=32, D=128, S_prefix=512, S_suffix=224,
                V=126464, logits_dtype="bf16", margin_max=3.0, parents=(-1,) * 8),
    3: Workload(3, "8b-tree", B=1, N=32, L=32, Hq=32, Hkv=32, D=128, S_prefix=1024, S_suffix=480,
                V=126464, logits_dtype="bf16", margin_max=3.0, level_sizes=(3, 9, 20)),
    4: Workload(4, "gqa-lookahead", B=1, N=16, L=64, Hq=28, Hkv=4, D=128, S_prefix=1536, S_suffix=512,
                V=152064, logits_dtype="bf16", margin_max=3.0, parents=(-1,) * 16),
    5: Workload(5, "8b-batched", B=16, N=64, L=32, Hq=32, Hkv=32, D=128, S_prefix=3584, S_suffix=512,
                V=126464, logits_dtype="bf16", margin_max=3.0, level_sizes=(3, 9, 27, 25)),
}

RANK_WEIGHT = (0.6, 0.25, 0.15)


def seed_for(cid, salt=0):
    """Default seed of a workload: 1000 + id (plus an optional salt)."""
    return 1000 + int(cid) + 7919 * int(salt)


# --------------------------------------------------------------------------
# trees
# --------------------------------------------------------------------------

def build_tree(level_sizes, rng):
    """3-ary BFS tree: returns (parent [N], rank [N], level [N]) as int arrays."""
    parents, ranks, levels, weights = [], [], [], []
    frontier = [(-1, 1.0)]  # (node id, path weight)
    for lvl, size in enumerate(level_sizes, start=1):
        cands = []
        for node, w in frontier:
            for r in range(3):
                cw = w * RANK_WEIGHT[r] * float(np.exp(0.25 * rng.standard_normal()))
                cands.append((cw, node, r))
        keep_at = sorted(range(len(cands)), key=lambda i: -cands[i][0])[:size]
        keep = sorted(keep_at)  # BFS order: by (parent, rank)
        new_frontier = []
        for i in keep:
            cw, node, r = cands[i]
            nid = len(parents)
            parents.append(node)
            ranks.append(r)
            levels.append(lvl)
            weights.append(cw)
            new_frontier.append((nid, cw))
        frontier = new_frontier
    return (np.array(parents, dtype=np.int32), np.array(ranks, dtype=np.int32),
            np.array(levels, dtype=np.int32))


def tree_structure(wl, rng):
    """Parent/rank/level arrays of shape [B, N] for a workload."""
    B, N = wl.B, wl.N
    parent = np.empty((B, N), dtype=np.int32)
    rank = np.empty((B, N), dtype=np.int32)
    level = np.empty((B, N), dtype=np.int32)
    for b in range(B):
        if wl.level_sizes is not None:
            p, r, lv = build_tree(wl.level_sizes, rng)
            if len(p) != N:
                raise ValueError("level sizes do not add up to N")
        else:
            p = np.array(wl.parents, dtype=np.int32)
            if len(p) != N:
                raise ValueError("explicit parent array does not match N")
            r = np.zeros(N, dtype=np.int32)
            lv = np.zeros(N, dtype=np.int32)
            for n in range(N):
                sib = [c for c in range(n) if p[c] == p[n]]
                r[n] = len(sib)
                lv[n] = 1 if p[n] == -1 else lv[p[n]] + 1
        parent[b], rank[b], level[b] = p, r, lv
    return parent, rank, level


# --------------------------------------------------------------------------
# attention tensors
# --------------------------------------------------------------------------

def attention_inputs(wl, seed, variant="spec", device="cpu"):
    """q, k_cache, v_cache, k_draft, v_draft as bf16 torch tensors on ``device``."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    B, N, L, Hq, Hkv, D, S = wl.B, wl.N, wl.L, wl.Hq, wl.Hkv, wl.D, wl.S
    if variant == "spec":
        sq = sk = sv = 1.0 / math.sqrt(D)
    elif variant == "sharp":
        sq, sk, sv = 3.0, 1.0, 1.0
    else:
        raise ValueError(f"unknown attention variant {variant!r}")

    def draw(shape, std):
        t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        return (t * std).to(torch.bfloat16)

    q = draw((B, N, L, Hq, D), sq)
    k_cache = draw((B, S, Hkv, D), sk)
    v_cache = draw((B, S, Hkv, D), sv)
    k_draft = draw((B, N, L, Hkv, D), sk)
    v_draft = draw((B, N, L, Hkv, D), sv)
    return q, k_cache, v_cache, k_draft, v_draft


# --------------------------------------------------------------------------
# block states, planted candidates and draft tokens
# --------------------------------------------------------------------------

def _logit(x):
    return math.log(x / (1.0 - x))


def _draw_margins(rng, count, margin_max, tau, gap):
    m = rng.uniform(0.0, margin_max, size=count)
    if gap > 0 and 0.0 < tau < 1.0:
        edge = _logit(tau)
        bad = np.abs(m - edge) < gap
        while bad.any():
            m[bad] = rng.uniform(0.0, margin_max, size=int(bad.sum()))
            bad = np.abs(m - edge) < gap
    return m


def _distinct_tokens(rng, V, count):
    out = np.empty((count, 3), dtype=np.int64)
    for i in range(count):
        out[i] = rng.choice(V, size=3, replace=False)
    return out


def _planted_intent(state, margin, top, tau, gap):
    """Intended next state from planted margins; adjusts fallback margins in
    place so the winner stays ``gap`` clear.  Returns (next_state or None,
    newly unmasked positions)."""
    L = len(state)
    masked = [p for p in range(L) if state[p] == MASK]
    if not masked:
        return None, []
    if tau >= 1.0:
        clears = []
    elif tau < 0.0:
        clears = list(masked)
    else:
        edge = _logit(tau)
        clears = [p for p in masked if margin[p] > edge]
    if not clears:
        order = sorted(masked, key=lambda p: -margin[p])
        win = order[0]
        if gap > 0:
            for p in order[1:]:
                if margin[p] > margin[win] - gap:
                    margin[p] = margin[win] - gap
        clears = [win]
    nxt = np.array(state, copy=True)
    for p in clears:
        nxt[p] = top[p, 0]
    return nxt, clears


def decode_inputs(wl, seed, tau=None, gap=0.1, parent=None, rank=None, level=None):
    """Tree, committed state, planted candidates and draft tokens.

    Returns a dict of numpy arrays:
      parent [B,N] int32, rank [B,N], level [B,N],
      committed [B,L] int32, conf0 [B,L,k] float32, idx0 [B,L,k] int32,
      tokens [B,N,L] int32,
      row_margin [B*N*L] float64, row_top [B*N*L,3] int64  (draft rows),
      planted_leaf [B] int64, tau (float).
    """
    tau = wl.tau if tau is None else float(tau)
    rng = np.random.Generator(np.random.PCG64(int(seed)))
    if parent is None:
        parent, rank, level = tree_structure(wl, rng)
    B, N, L, V, k = wl.B, wl.N, wl.L, wl.V, wl.k
    if k != 3:
        raise ValueError("the generator plants exactly three candidates per position")

    committed = rng.integers(0, V, size=(B, L)).astype(np.int32)
    masked = rng.random((B, L)) < 0.75
    need = min(4, L)
    for b in range(B):
        if masked[b].sum() < need:
            extra = rng.choice(np.flatnonzero(~masked[b]), size=need - int(masked[b].sum()), replace=False)
            masked[b, extra] = True
    committed[masked] = MASK

    conf0 = np.zeros((B, L, k), dtype=np.float32)
    idx0 = np.zeros((B, L, k), dtype=np.int32)
    tokens = np.full((B, N, L), MASK, dtype=np.int32)
    row_margin = np.zeros((B, N, L), dtype=np.float64)
    row_top = np.zeros((B, N, L, 3), dtype=np.int64)
    planted_leaf = np.full(B, -1, dtype=np.int64)

    for b in range(B):
        m0 = _draw_margins(rng, L, wl.margin_max, tau, gap)
        t0 = _distinct_tokens(rng, V, L)
        states = {-1: committed[b]}
        margins = {-1: m0}
        tops = {-1: t0}
        intent_ok = {-1: True}
        # children lists in index order
        kids = {q: [c for c in range(N) if parent[b, c] == q] for q in range(-1, N)}
        order = [-1] + list(range(N))
        for q in order:
            if q >= 0:
                margins[q] = _draw_margins(rng, L, wl.margin_max, tau, gap)
                tops[q] = _distinct_tokens(rng, V, L)
            nxt, new_pos = _planted_intent(states[q], margins[q], tops[q], tau, gap)
            for c in kids[q]:
                r = int(rank[b, c])
                lvl = int(level[b, c])
                if nxt is None:
                    states[c] = np.array(states[q], copy=True)
                    intent_ok[c] = False
                    continue
                child = np.array(nxt, copy=True)
                ok = True
                if r == 0:
                    a = wl.alpha[0] if lvl <= 1 else wl.alpha[1]
                    if rng.random() >= a:
                        p = new_pos[int(rng.integers(len(new_pos)))]
                        child[p] = tops[q][p, 1]
                        ok = False
                else:
                    p = new_pos[0]
                    child[p] = tops[q][p, min(r, 2)]
                    ok = False
                states[c] = child
                intent_ok[c] = ok and intent_ok[q]
        for n in range(N):
            tokens[b, n] = states[n]
            row_margin[b, n] = margins[n]
            row_top[b, n] = tops[n]
        sig = 1.0 / (1.0 + np.exp(-m0))
        conf0[b, :, 0] = sig
        conf0[b, :, 1] = 0.3 * (1.0 - sig)
        conf0[b, :, 2] = 0.2 * (1.0 - sig)
        idx0[b] = t0
        # follow intended rank-0 children from the committed state
        cur = -1
        while True:
            nxt_node = -1
            for c in kids[cur]:
                if intent_ok[c] and int(rank[b, c]) == 0:
                    nxt_node = c
                    break
            if nxt_node == -1:
                break
            cur = nxt_node
        planted_leaf[b] = cur

    return {
        "parent": parent.astype(np.int32), "rank": rank, "level": level,
        "committed": committed, "conf0": conf0, "idx0": idx0, "tokens": tokens,
        "row_margin": row_margin.reshape(B * N * L),
        "row_top": row_top.reshape(B * N * L, 3),
        "planted_leaf": planted_leaf, "tau": tau,
    }


# --------------------------------------------------------------------------
# logits
# --------------------------------------------------------------------------

def make_logits(row_margin, row_top, V, dtype, seed, device="cpu", mode="lse", row_chunk=256,
                out=None):
    """Logit rows [R, V] as a torch tensor of ``dtype`` (torch.bfloat16 or
    torch.float32) on ``device``; see the module docstring for the modes."""
    row_margin = np.asarray(row_margin, dtype=np.float64)
    row_top = np.asarray(row_top, dtype=np.int64)
    R = row_margin.shape[0]
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    if out is None:
        out = torch.empty((R, V), dtype=dtype, device=device)
    for r0 in range(0, R, row_chunk):
        r1 = min(R, r0 + row_chunk)
        n = r1 - r0
        if mode == "ties":
            z = torch.randint(0, 8, (n, V), generator=gen, device=device).to(torch.float32) * 0.25
            out[r0:r1] = z.to(dtype)
            continue
        z = torch.randn((n, V), generator=gen, device=device, dtype=torch.float32)
        rows = torch.arange(n, device=device)
        top = torch.as_tensor(row_top[r0:r1], device=device)
        m = torch.as_tensor(row_margin[r0:r1], device=device, dtype=torch.float32)
        if mode == "raw":
            z[rows, top[:, 0]] = z[rows, top[:, 0]] + m
        elif mode == "lse":
            zmax = z.max(dim=1).values
            z[rows, top[:, 2]] = zmax + 0.25
            z[rows, top[:, 1]] = zmax + 0.5
            z[rows, top[:, 0]] = -float("inf")
            others = torch.logsumexp(z.double(), dim=1).to(torch.float32) if V <= 4096 else \
                torch.logsumexp(z, dim=1)
            z[rows, top[:, 0]] = others + m
        else:
            raise ValueError(f"unknown logit mode {mode!r}")
        out[r0:r1] = z.to(dtype)
    return out


def torch_dtype(name):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]
