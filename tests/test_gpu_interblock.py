"""GPU parity for inter-block speculation (Sec. 3.4): attention with per-draft peer
visibility against the attention oracle with the same peers (same tolerance as the plain
attention tests), and the trigger against the trigger oracle (bit-exact: both compare the same
fp32 confidences with the threshold rounded to fp32)."""

import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from helpers import attn_close, cuda, np64
from oracle.interblock import interblock_trigger_batch, joint_peers
from synthetic import Workload, attention_inputs

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "interblock_trigger.json")


def _wl(B, N, L, Hq, Hkv, D, S):
    return Workload(98, "peers", B=B, N=N, L=L, Hq=Hq, Hkv=Hkv, D=D, S_prefix=S, S_suffix=0, V=64,
                    logits_dtype="f32", margin_max=3.0, parents=None, level_sizes=None)


def _peers_tensor(rows):
    arr = np.array([[int(x) & ((1 << 64) - 1) for x in r] for r in rows], dtype=np.uint64)
    return torch.from_numpy(arr.view(np.int64).copy()).cuda()


def _run(wl, parent, peers_rows, variant, seed, seqs=None):
    """GPU output of the sequences `seqs` (default: all) with the oracle's reference for them."""
    inputs = attention_inputs(wl, seed, variant)
    args = [t.cuda() for t in inputs]
    out = tsp.verify_attn(*args, cuda(parent, torch.int32), peers=_peers_tensor(peers_rows))
    torch.cuda.synchronize()
    seqs = list(range(wl.B)) if seqs is None else list(seqs)
    x = [np64(t)[seqs] for t in inputs]
    par = parent[seqs]
    peers = [peers_rows[b] for b in seqs]
    ref = oracle.verify_attention(*x, par, peers=peers)
    aw = None
    if variant == "sharp":
        q, kc, vc, kd, vd = x
        aw = oracle.verify_attention(q, kc, np.abs(vc), kd, np.abs(vd), par, peers=peers)
    return out[seqs], ref, aw


def _batch_for_tiling(N, L, Hq, Hkv, tiling):
    """2 sequences (a one-sequence-sized grid: 16 query rows per wave), or the smallest batch
    whose grid of 16-row workgroups (4 waves x 16 rows) exceeds the CU count, which the library
    runs with 32-row waves."""
    if tiling == "16":
        return 2
    wg16 = -(-((Hq // Hkv) * N * L) // 64)
    return torch.cuda.get_device_properties(0).multi_processor_count // (Hkv * wg16) + 1


@pytest.mark.parametrize("L,N,S,Hq,Hkv,D", [
    (32, 11, 200, 4, 4, 128),   # joint trees 7 + 4 (W3D3 and W1D3)
    (32, 64, 96, 2, 2, 128),    # 64 drafts, random peers
    (40, 6, 70, 4, 2, 64),      # ragged tiles, GQA
    (8, 9, 33, 2, 1, 128),      # several drafts per 32-key tile
])
@pytest.mark.parametrize("variant", ["spec", "sharp"])
@pytest.mark.parametrize("tiling", ["16", "32"])
def test_peers_parity(L, N, S, Hq, Hkv, D, variant, tiling):
    rng = np.random.default_rng(L * 100 + N)
    B = _batch_for_tiling(N, L, Hq, Hkv, tiling)
    wl = _wl(B, N, L, Hq, Hkv, D, S)
    if N == 11:
        parent = np.array([[-1, 0, 0, 0, 1, 2, 4, -1, 7, 8, 9]] * B, dtype=np.int32)
        peers_rows = [joint_peers(7, 4, 0, 0)] * B
    else:
        parent = np.array([[-1] + [int(rng.integers(-1, n)) for n in range(1, N)] for _ in range(B)], dtype=np.int32)
        peers_rows = [[int(rng.integers(0, 1 << 62)) | (int(rng.integers(0, 2)) << 63) for _ in range(N)]
                      for _ in range(B)]
    out, ref, aw = _run(wl, parent, peers_rows, variant, seed=N + L, seqs=sorted({0, B - 1}))
    ok, worst, frac = attn_close(out, ref, aw)
    assert ok, f"{variant}: worst excess {worst:.3g}, {frac:.2%} outside tolerance"


def test_zero_peers_equal_plain_call():
    wl = _wl(2, 8, 32, 4, 4, 128, 300)
    parent = np.array([[-1, 0, 0, 1, 1, 2, 3, -1]] * 2, dtype=np.int32)
    args = [t.cuda() for t in attention_inputs(wl, 5, "sharp")]
    par = cuda(parent, torch.int32)
    a = tsp.verify_attn(*args, par)
    b = tsp.verify_attn(*args, par, peers=torch.zeros((2, 8), dtype=torch.int64, device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_trigger_golden(case):
    g = json.load(open(GOLDEN))
    out = tsp.interblock_trigger(cuda(np.array([case["state"]]), torch.int32),
                                 cuda(np.array([case["conf"]], dtype=np.float32), torch.float32), g["tau"])
    torch.cuda.synchronize()
    assert bool(out["trigger"].item()) == case["trigger"]
    assert out["c_cur"].item() == pytest.approx(case["c_t"]) and out["c_next"].item() == pytest.approx(case["c_t1"])


@pytest.mark.parametrize("L", [1, 13, 32, 64])
def test_trigger_random(L):
    rng = np.random.default_rng(L)
    B, k, tau = 300, 3, 0.9
    state = np.where(rng.random((B, 2 * L)) < rng.random((B, 1)), -1, 7).astype(np.int32)
    conf = rng.random((B, 2 * L, k)).astype(np.float32)
    conf[::7, L:, 0] = conf[::7, :L, 0]  # equal block maxima on some rows
    tau32 = float(np.float32(tau))
    trig, c_t, c_t1 = interblock_trigger_batch(state, conf, L, tau32)
    out = tsp.interblock_trigger(cuda(state, torch.int32), cuda(conf, torch.float32), tau)
    torch.cuda.synchronize()
    assert np.array_equal(out["trigger"].cpu().numpy().astype(bool), trig)
    assert np.array_equal(out["c_cur"].cpu().numpy(), c_t.astype(np.float32))
    assert np.array_equal(out["c_next"].cpu().numpy(), c_t1.astype(np.float32))


@pytest.mark.parametrize("n_cur,n_next", [(3, 2), (7, 4), (60, 4), (1, 63), (32, 32)])
def test_joint_peers_match_oracle(n_cur, n_next):
    """traj_joint_peers against the oracle's joint-packing rule, bit for bit, with per-sequence
    roots (and root 0 when no root arrays are given)."""
    B = 5
    rng = np.random.default_rng(n_cur * 64 + n_next)
    rc = rng.integers(0, n_cur, B).astype(np.int32)
    rn = rng.integers(0, n_next, B).astype(np.int32)
    got = tsp.joint_peers(B, n_cur, n_next, cuda(rc), cuda(rn)).cpu().numpy().view(np.uint64)
    for b in range(B):
        assert [int(x) for x in got[b]] == joint_peers(n_cur, n_next, int(rc[b]), int(rn[b])), b
    got0 = tsp.joint_peers(B, n_cur, n_next, device="cuda").cpu().numpy().view(np.uint64)
    for b in range(B):
        assert [int(x) for x in got0[b]] == joint_peers(n_cur, n_next, 0, 0)


def test_joint_peers_bad_root_is_flagged():
    tsp.device_status(reset=True)
    rc = cuda(np.array([0, 5], dtype=np.int32))   # 5 is outside a 3-draft tree
    rn = cuda(np.array([1, 1], dtype=np.int32))
    got = tsp.joint_peers(2, 3, 2, rc, rn).cpu().numpy().view(np.uint64)
    assert tsp.device_status(reset=True) & tsp.DEV_BAD_ROOT
    assert [int(x) for x in got[1]] == joint_peers(3, 2, 0, 1)
