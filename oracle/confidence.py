"""Oracle: per-position confidence and top-k candidates (fp64).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Sec. 3.2, Eq. 2 defines the token confidence as the largest softmax
probability of a position's logits, c(x) = max softmax(logits(x)); candidate
collection then takes the top-k tokens of each low-confidence position
(Sec. 3.2 "Candidate collection", k about 3).  The softmax is plain (no
temperature, no noise).

For one row of logits l over a vocabulary of V entries:
  m        = max_v l_v
  s        = sum_v exp(l_v - m)
  order    = the k largest entries, larger value first; equal values keep the
             lower vocabulary index first (a stable sort of -l)
  conf[j]  = exp(l_order[j] - m) / s       so conf[0] = c(x)
  idx[j]   = order[j]

The comparison is made on the stored logit values themselves (bf16 or fp32
values are exactly representable in fp64), never on recomputed
probabilities.  Rows must be free of NaN and hold at least one finite value.
"""

import numpy as np


def confidence_topk(logits, k, chunk_rows=256):
    """Return (conf [R,k] float64, idx [R,k] int64) for logits of shape [R,V]."""
    x_all = np.asarray(logits)
    if x_all.ndim != 2:
        raise ValueError("logits must be 2-D [rows, vocab]")
    R, V = x_all.shape
    if not (1 <= k <= V):
        raise ValueError("need 1 <= k <= vocab")
    conf = np.empty((R, k), dtype=np.float64)
    idx = np.empty((R, k), dtype=np.int64)
    for r0 in range(0, R, chunk_rows):
        x = x_all[r0:r0 + chunk_rows].astype(np.float64)
        m = x.max(axis=1, keepdims=True)
        s = np.exp(x - m).sum(axis=1, keepdims=True)
        order = np.argsort(-x, axis=1, kind="stable")[:, :k]
        conf[r0:r0 + chunk_rows] = np.exp(np.take_along_axis(x, order, axis=1) - m) / s
        idx[r0:r0 + chunk_rows] = order
    return conf, idx
