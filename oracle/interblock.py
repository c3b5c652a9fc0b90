"""Oracle: inter-block speculation trigger and joint-tree visibility (Sec. 3.4, App. D).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

* Trigger (Sec. 3.4 "Trigger condition"): with c_t and c_{t+1} the top-1 confidences of the
  current block B_t and the next block B_{t+1}, speculation over both blocks starts when
  c_{t+1} > c_t or c_{t+1} > tau.  Reading: a block's top-1 confidence is the largest top-1
  confidence c(x) over its still-masked positions (0 when none is masked: a finished block
  gives no evidence), and the trigger needs a masked position in B_{t+1} (a finished next
  block leaves nothing to speculate on).  The confidences of both blocks come from one
  verification pass whose drafts cover both blocks (2L positions per state).
* Joint verification (Sec. 3.4 "Joint tree construction", App. D): the trees of B_t (drafts
  0 .. n_cur-1) and B_{t+1} (drafts n_cur .. n_cur+n_next-1) are verified in one pass.  Each
  draft of either tree may additionally look at the root draft of the other tree (the
  visibility is mutual between the two trees' roots and everything below them); the other
  tree's non-root drafts stay hidden.  Returned as per-draft peer bit masks for
  the attention oracle's ``peers`` argument.
"""

import numpy as np

MASK = -1


def block_top1_confidence(state, conf):
    """Largest conf[p][0] over the masked positions of a block state (0 when none)."""
    best = 0.0
    for p in range(len(state)):
        if state[p] == MASK and conf[p][0] > best:
            best = float(conf[p][0])
    return best


def interblock_trigger(state, conf, L, tau):
    """state [2L] (B_t then B_{t+1}), conf [2L, k].  Returns (trigger, c_t, c_t1)."""
    c_t = block_top1_confidence(state[:L], conf[:L])
    c_t1 = block_top1_confidence(state[L:2 * L], conf[L:2 * L])
    next_open = any(state[p] == MASK for p in range(L, 2 * L))
    return bool(next_open and (c_t1 > c_t or c_t1 > tau)), c_t, c_t1


def interblock_trigger_batch(state, conf, L, tau):
    res = [interblock_trigger(state[b], conf[b], L, tau) for b in range(len(state))]
    return (np.array([r[0] for r in res]), np.array([r[1] for r in res]), np.array([r[2] for r in res]))


def joint_peers(n_cur, n_next, root_cur, root_next):
    """Peer masks [n_cur + n_next] for a joint tree: every draft of the next block's tree sees
    draft root_cur (the current block's root), every draft of the current block's tree sees
    draft n_cur + root_next (the next block's root)."""
    n = n_cur + n_next
    peers = [0] * n
    for i in range(n_cur):
        peers[i] |= 1 << (n_cur + root_next)
    for i in range(n_cur, n):
        peers[i] |= 1 << root_cur
    return peers
