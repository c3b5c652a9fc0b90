"""Oracle: blockwise trajectory-masked verification attention (fp64, dense mask).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

What is computed (Sec. 3.3, "Blockwise Parallel Verification", attention
masking for trajectory isolation; Sec. 3.2 / Alg. 1 for the draft tree):

* The dual cache (Fast-dLLM, Sec. 1 and App. A) holds S prefix+suffix tokens
  per sequence.  Every draft token attends bidirectionally to all of them.
* Draft block ``i`` attends bidirectionally to all L tokens of its own block.
* The paper's mask isolates a block from every other draft block.  A draft in a
  trajectory tree is a denoising *state* whose earlier steps are its ancestors;
  the verification step therefore also lets block ``i`` see the blocks on its
  own root path (its tree ancestors), never siblings, cousins or descendants.
  With every parent equal to -1 this is exactly the paper's all-isolated mask.
* Only draft tokens are queries: the dual cache keeps prefix/suffix K/V frozen
  within a block and only block-level K/V is recomputed (App. A).
* Softmax scale defaults to 1/sqrt(D) (the paper does not state one).
* Grouped-query attention: query head ``h`` reads K/V head ``h // (Hq // Hkv)``
  (heads of one group are contiguous).
* Inter-block speculation (Sec. 3.4 "Joint tree construction", App. D) verifies
  the trees of two consecutive blocks in one pass and keeps the roots of the two
  blocks visible to each other's drafts.  That visibility is not a parent
  relation, so it comes in as ``peers``: bit j of ``peers[b, n]`` makes every
  token of draft j visible to draft n on top of its root path (one direction;
  symmetric visibility sets both bits).

Layouts (all row-major):
  q        [B, N, L, Hq, D]
  k_cache  [B, S, Hkv, D]       v_cache  [B, S, Hkv, D]
  k_draft  [B, N, L, Hkv, D]    v_draft  [B, N, L, Hkv, D]
  parent   [B, N]  int, -1 = child of the committed state, else parent[n] < n
  out      [B, N, L, Hq, D]  float64
"""

import math

import numpy as np


def _check_parent_row(parent_row):
    n_drafts = len(parent_row)
    for n, p in enumerate(parent_row):
        p = int(p)
        if not (-1 <= p < n):
            raise ValueError(
                f"draft {n} has parent {p}; parents must satisfy -1 <= parent[n] < n "
                f"(topological order) with N={n_drafts}"
            )


def ancestor_sets(parent_row):
    """anc*(i) = {i} together with every node on i's parent chain up to -1.

    ``parent_row`` is the parent array of one sequence (length N).  Returns a
    list of Python sets, one per draft.
    """
    _check_parent_row(parent_row)
    out = []
    for i in range(len(parent_row)):
        chain = {i}
        j = int(parent_row[i])
        while j != -1:
            chain.add(j)
            j = int(parent_row[j])
        out.append(chain)
    return out


def visible_sets(parent_row, peers_row=None):
    """anc*(i) plus the drafts whose bits are set in peers_row[i] (bits >= N ignored)."""
    vis = ancestor_sets(parent_row)
    if peers_row is not None:
        n_drafts = len(parent_row)
        for i in range(n_drafts):
            bits = int(peers_row[i]) & ((1 << 64) - 1)
            vis[i] |= {j for j in range(n_drafts) if (bits >> j) & 1}
    return vis


def trajectory_mask(parent_row, L, S, peers_row=None):
    """Dense boolean visibility mask of shape [N*L, S + N*L].

    Row ``i*L + p`` is query token p of draft i.  Column ``s < S`` is cache
    token s (always visible); column ``S + j*L + p'`` is token p' of draft j,
    visible iff j is in anc*(i) or bit j of peers_row[i] is set.
    """
    vis = visible_sets(parent_row, peers_row)
    n_drafts = len(parent_row)
    mask = np.zeros((n_drafts * L, S + n_drafts * L), dtype=bool)
    mask[:, :S] = True
    for i in range(n_drafts):
        for j in vis[i]:
            mask[i * L:(i + 1) * L, S + j * L:S + (j + 1) * L] = True
    return mask


def verify_attention(q, k_cache, v_cache, k_draft, v_draft, parent, scale=None, peers=None):
    """Trajectory-masked attention for every draft token, fp64.

    Per (sequence b, query head h): build K_all = [cache keys; all draft keys
    flattened], scores = (Q_h K_all^T) * scale, set masked entries to -inf,
    take a row softmax (subtracting the row max) and multiply by V_all.
    """
    q = np.asarray(q, dtype=np.float64)
    k_cache = np.asarray(k_cache, dtype=np.float64)
    v_cache = np.asarray(v_cache, dtype=np.float64)
    k_draft = np.asarray(k_draft, dtype=np.float64)
    v_draft = np.asarray(v_draft, dtype=np.float64)
    parent = np.asarray(parent)

    B, N, L, Hq, D = q.shape
    S = k_cache.shape[1]
    Hkv = k_cache.shape[2]
    if Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    if k_cache.shape != (B, S, Hkv, D) or v_cache.shape != (B, S, Hkv, D):
        raise ValueError("cache shape mismatch")
    if k_draft.shape != (B, N, L, Hkv, D) or v_draft.shape != (B, N, L, Hkv, D):
        raise ValueError("draft K/V shape mismatch")
    if parent.shape != (B, N):
        raise ValueError("parent shape mismatch")
    group = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)

    out = np.zeros((B, N, L, Hq, D), dtype=np.float64)
    for b in range(B):
        mask = trajectory_mask(parent[b], L, S, None if peers is None else peers[b])
        for h in range(Hq):
            g = h // group
            q_h = q[b, :, :, h, :].reshape(N * L, D)
            k_all = np.concatenate([k_cache[b, :, g, :], k_draft[b, :, :, g, :].reshape(N * L, D)])
            v_all = np.concatenate([v_cache[b, :, g, :], v_draft[b, :, :, g, :].reshape(N * L, D)])
            scores = (q_h @ k_all.T) * scale
            scores = np.where(mask, scores, -np.inf)
            scores = scores - scores.max(axis=1, keepdims=True)
            weights = np.exp(scores)
            weights = weights / weights.sum(axis=1, keepdims=True)
            out[b, :, :, h, :] = (weights @ v_all).reshape(N, L, D)
    return out
