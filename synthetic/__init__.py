"""Seeded synthetic inputs shared by the tests, the bench and the oracle checks.

Holds no part of the verification step's arithmetic; see ``workloads``.
"""

from .workloads import (  # noqa: F401
    MASK,
    WORKLOADS,
    Workload,
    attention_inputs,
    build_tree,
    decode_inputs,
    make_logits,
    seed_for,
    torch_dtype,
    tree_structure,
)
