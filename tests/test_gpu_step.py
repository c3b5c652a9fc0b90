"""GPU parity of the whole verification step: attention, then the logit pass,
then acceptance on the GPU's own confidences, against the oracle end to end.

Acceptance decisions taken at a state whose confidences lie within 1e-4 of
tau (or whose fallback winner is within 1e-4 of the runner-up) are excluded
from the bit-exact comparison and counted.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from synthetic import WORKLOADS, attention_inputs, decode_inputs, make_logits, seed_for, torch_dtype
from helpers import attn_close, compare_accept, cuda, np64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cid,gap", [(1, 0.1), (1, 0.0), (2, 0.1), (3, 0.0)])
def test_step_end_to_end(cid, gap):
    wl = WORKLOADS[cid]
    if cid != 1:
        wl = wl.with_(Hq=2, Hkv=2)  # keep the oracle's attention short
    seed = seed_for(cid, 3)
    d = decode_inputs(wl, seed, gap=gap)
    B, N, L, k = wl.B, wl.N, wl.L, wl.k
    q, kc, vc, kd, vd = attention_inputs(wl, seed)
    lg = make_logits(d["row_margin"], d["row_top"], wl.V, torch_dtype(wl.logits_dtype), seed)

    stream = torch.cuda.current_stream()
    out = tsp.verify_attn(q.cuda(), kc.cuda(), vc.cuda(), kd.cuda(), vd.cuda(), cuda(d["parent"], torch.int32))
    conf, idx = tsp.confidence_topk(lg.cuda(), k)
    acc = tsp.accept(conf, idx, cuda(d["tokens"]), cuda(d["parent"]), cuda(d["committed"]), cuda(d["conf0"]),
                     cuda(d["idx0"]), wl.tau)
    stream.synchronize()

    ok, worst, _ = attn_close(out, oracle.verify_attention(*[np64(t) for t in (q, kc, vc, kd, vd)], d["parent"]))
    assert ok, worst
    rc, ri = oracle.confidence_topk(lg.float().numpy(), k)
    assert np.array_equal(idx.cpu().numpy(), ri)
    assert np.abs(conf.cpu().numpy() - rc).max() <= 1e-4
    conf_ref = rc.reshape(B, N, L, k)
    ref = oracle.accept_batch(d["tokens"], d["parent"], d["committed"], d["conf0"].astype(np.float64), d["idx0"],
                              conf_ref, ri.reshape(B, N, L, k), wl.tau)
    msgs, excl_seq, excl_hi = compare_accept(acc, ref, d, conf_ref, wl.tau, B, N, L, k)
    assert not msgs, msgs
    print(f"{wl.name} gap={gap}: excluded sequences {excl_seq}, excluded hi bits {excl_hi}, "
          f"leaf {ref['leaf'].tolist()} n_acc {ref['n_accepted'].tolist()}")
