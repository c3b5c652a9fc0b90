"""The allocation-free logit pass (traj_confidence_topk_noalloc, fixed per-device scratch)
against the entry point with a caller workspace, through the C ABI: bit-identical results on
two calls in a row (the second with a smaller input, so the fixed scratch holds the first
call's records when it starts), both split (short-batch) shapes; and the oracle's bar
(indices bit-exact, confidences within 1e-4)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from helpers import CONF_ATOL
from synthetic import WORKLOADS, decode_inputs, make_logits

pytestmark = pytest.mark.gpu


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    wl = WORKLOADS[2].with_(N=2, parents=(-1, -1))
    d = decode_inputs(wl, 11)
    first = make_logits(d["row_margin"][:40], d["row_top"][:40], wl.V, torch.bfloat16, 21, device="cuda")
    second = make_logits(d["row_margin"][:3], d["row_top"][:3], wl.V, torch.bfloat16, 22, device="cuda")
    for lg in (first, second):
        assert tsp.confidence_topk_workspace_size(lg, 3) > 0  # a split plan: the scratch is used
        ref_c, ref_i = tsp.confidence_topk(lg, 3)
        got_c, got_i = tsp.confidence_topk_noalloc(lg, 3)
        torch.cuda.synchronize()
        assert torch.equal(got_i, ref_i)
        assert torch.equal(got_c, ref_c)
        rc, ri = oracle.confidence_topk(lg.float().cpu().numpy(), 3)
        assert np.array_equal(got_i.cpu().numpy(), ri)
        assert np.abs(got_c.cpu().numpy() - rc).max() <= CONF_ATOL


def test_noalloc_unsplit_and_empty_shapes():
    x = torch.randn(600, 5000, device="cuda").to(torch.bfloat16)  # no split: no scratch needed
    ref_c, ref_i = tsp.confidence_topk(x, 4)
    got_c, got_i = tsp.confidence_topk_noalloc(x, 4)
    torch.cuda.synchronize()
    assert torch.equal(got_i, ref_i) and torch.equal(got_c, ref_c)
    e = torch.empty((0, 100), dtype=torch.bfloat16, device="cuda")
    c, i = tsp.confidence_topk_noalloc(e, 3)
    assert c.shape == (0, 3)
