"""MI355X (gfx950) trajectory-verification step for trajectory-level speculative
decoding of diffusion language models.

The three calls of one verification step (all HIP kernels in libtrajspec.so):

* :func:`verify_attn`      -- trajectory-masked attention over the dual cache and
  the packed draft blocks (each draft sees the cache, itself and its ancestors).
* :func:`confidence_topk`  -- per-position max-softmax confidence and top-k
  candidates over the vocabulary.
* :func:`accept`           -- threshold-decoding consistency and greedy /
  longest-path acceptance of the draft tree.

and the next step's drafts:

* :func:`build_tree`       -- confidence-stratified draft tree (Alg. 1) from the
  accepted state and the candidates its verification produced.

and inter-block speculation (Sec. 3.4):

* :func:`interblock_trigger` -- whether the next block is confident enough to
  speculate on both blocks; :func:`joint_peers` builds the visibility masks of the
  two blocks' joint trees on the device and :func:`verify_attn` with ``peers``
  verifies them in one pass.

and :func:`verify_layer`, a whole decoder layer of the verification forward pass around the
attention (norms, projections on the library's MFMA GEMM, RoPE, SwiGLU MLP), and
:func:`linear`, that GEMM on its own; :func:`refresh_layer` runs the same layer over whole
sequences at a block boundary and refreshes the dual cache (App. A).
"""

from ._lib import (  # noqa: F401
    DEV_BAD_BLOCK,
    DEV_BAD_ROOT,
    DEV_BAD_LEAF,
    DEV_BAD_PARENT,
    LIB_PATH,
    TrajSpecError,
    accept,
    build_tree,
    built_digest,
    check_build,
    confidence_topk,
    confidence_topk_noalloc,
    confidence_topk_workspace_size,
    device_status,
    interblock_trigger,
    joint_peers,
    layer_workspace_size,
    linear,
    linear_workspace_size,
    refresh_layer,
    refresh_layer_workspace_size,
    verify_layer,
    load,
    tree_max_nodes,
    verify_attn,
    verify_attn_workspace_size,
    version,
)
