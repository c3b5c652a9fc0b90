"""Reference oracle for the trajectory-verification step (TEST INFRASTRUCTURE ONLY).

This package is a plain, slow, obviously-correct CPU implementation of what the
GPU hot path computes, written from the paper (Trajectory-Level Speculative
Decoding for Diffusion LLMs):

* :mod:`oracle.attention`  -- blockwise trajectory-masked attention with an
  explicit dense mask, fp64 (Sec. 3.3 "Attention masking for trajectory
  isolation"; draft blocks additionally see their tree ancestors).
* :mod:`oracle.confidence` -- per-position confidence c(x) = max softmax and
  top-k candidates, fp64 on the exact stored logit values (Sec. 3.2, Eq. 2).
* :mod:`oracle.accept`     -- threshold decoding with top-1 fallback (Sec. 2.1),
  child consistency, greedy / longest-path traversal (Sec. 3.3 "Verification
  procedure"), the next root's high-confidence set (Alg. 1, phase 1).
* :mod:`oracle.tree`       -- confidence-stratified tree construction (Alg. 1):
  stratification, top-k expansion at the first level, top-1 deeper, pruning
  by path confidence.
* :mod:`oracle.interblock` -- inter-block speculation trigger and the joint
  tree's root-to-root visibility (Sec. 3.4, App. D).
* :mod:`oracle.layer`      -- one verification decoder layer around the attention
  (RMSNorm, projections, rotary positions, SwiGLU MLP) with bf16 storage, and the
  same layer over whole sequences that refreshes the dual cache (App. A).
* :mod:`oracle.brute`      -- scalar-loop re-derivations used only to pin the
  functions above on tiny inputs.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path
(``paper_2608_27514_amd``) never imports it, and this package imports nothing
from the product path: the two share no kernels, helpers, tables or pre/post
processing.  Inputs come from the seeded generators in ``synthetic/``, which
hold none of the method's arithmetic.

Every function here is pinned by ``-m "not gpu"`` tests against closed forms,
invariants, hand-worked fixtures (``tests/golden/``) or brute force.
"""

MASK = -1  # token id used for a still-masked position in block states

from .attention import ancestor_sets, trajectory_mask, verify_attention, visible_sets  # noqa: E402
from .confidence import confidence_topk  # noqa: E402
from .accept import (  # noqa: E402
    threshold_step,
    is_consistent,
    accept_sequence,
    accept_batch,
    fragile_states,
)
from .tree import build_tree, build_tree_batch, gather_state_scores, level_widths  # noqa: E402
from .layer import bf16_round, full_attention, linear, refresh_layer, verify_layer  # noqa: E402
from .interblock import block_top1_confidence, interblock_trigger, interblock_trigger_batch, joint_peers  # noqa: E402

__all__ = [
    "MASK",
    "ancestor_sets",
    "trajectory_mask",
    "verify_attention",
    "confidence_topk",
    "threshold_step",
    "is_consistent",
    "accept_sequence",
    "accept_batch",
    "fragile_states",
    "build_tree",
    "build_tree_batch",
    "gather_state_scores",
    "level_widths",
    "visible_sets",
    "block_top1_confidence",
    "interblock_trigger",
    "interblock_trigger_batch",
    "joint_peers",
    "bf16_round",
    "verify_layer",
]
