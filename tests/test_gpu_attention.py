"""GPU parity: traj_verify_attn against the fp64 dense-mask oracle.

Tolerance: |gpu - oracle| <= 2e-3 + 2e-2 |oracle| elementwise (bf16 inputs,
fp32 accumulation, bf16 output).  Besides the spec-distributed inputs
(N(0,1)/sqrt(D), nearly uniform attention) every shape is also run "sharp"
(q ~ 3 N(0,1), k, v ~ N(0,1)), where a wrong mask is far outside tolerance.
With spec inputs at the full cache lengths the weights are nearly uniform over
thousands of keys and a dropped ancestor block stays inside the tolerance, so
the full-size launches are checked on sharp inputs together with wrong-mask
negative controls (test_full_size_sharp_sampled_heads_and_wrong_masks).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from synthetic import WORKLOADS, Workload, attention_inputs, decode_inputs, seed_for
from helpers import attn_close, cuda, np64

pytestmark = pytest.mark.gpu


def _parents(wl, seed):
    return decode_inputs(wl.with_(V=64), seed)["parent"]


def _run(wl, seed, variant="spec", parent=None, scale=0.0, device_gen="cpu"):
    q, kc, vc, kd, vd = attention_inputs(wl, seed, variant, device=device_gen)
    if parent is None:
        parent = _parents(wl, seed)
    args = [t.cuda() for t in (q, kc, vc, kd, vd)]
    out = tsp.verify_attn(*args, cuda(parent, torch.int32), scale=scale)
    torch.cuda.synchronize()
    return (q, kc, vc, kd, vd), parent, out


def _oracle(inputs, parent, scale=None):
    return oracle.verify_attention(*[np64(t) for t in inputs], parent, scale=scale)


def _abs_weighted(inputs, parent, scale=None):
    """sum_i w_i |v_i| per output element (the oracle run with |V|)."""
    q, kc, vc, kd, vd = [np64(t) for t in inputs]
    return oracle.verify_attention(q, kc, np.abs(vc), kd, np.abs(vd), parent, scale=scale)


def _check(out, inputs, parent, variant, scale=None):
    ref = _oracle(inputs, parent, scale)
    aw = _abs_weighted(inputs, parent, scale) if variant == "sharp" else None
    return attn_close(out, ref, aw)


def _cus():
    return torch.cuda.get_device_properties(0).multi_processor_count


def _wg16(wl):
    """Workgroups per (sequence, K/V head) with 16-row waves (4 waves x 16 rows each)."""
    return -(-((wl.Hq // wl.Hkv) * wl.N * wl.L) // 64)


def _tiling_batch(wl, tiling):
    """The batch that makes the library launch the given row tiling: one-sequence-sized grids
    (16-row grid at most one workgroup per CU) run with 16-row waves, larger ones with 32-row
    waves.  '16' keeps wl.B (asserting that it is in that regime); '32' takes the smallest batch
    past the threshold."""
    if tiling == "16":
        assert wl.B * wl.Hkv * _wg16(wl) <= _cus(), "shape is not in the 16-row regime"
        return wl.B
    return _cus() // (wl.Hkv * _wg16(wl)) + 1


def _check_seqs(out, inputs, parent, variant, seqs):
    """Oracle check of the sequences `seqs` only (sequences are independent)."""
    for b in seqs:
        sub = [t[b:b + 1] for t in inputs]
        ok, worst, frac = _check(out[b:b + 1], sub, parent[b:b + 1], variant)
        if not ok:
            return False, worst, frac, b
    return True, 0.0, 0.0, None


SMALL = {
    # name: workload (reduced heads where the full one would be slow for the oracle)
    "tiny": WORKLOADS[1],
    "8b-siblings-4h": WORKLOADS[2].with_(Hq=4, Hkv=4),
    "8b-tree-2h": WORKLOADS[3].with_(Hq=2, Hkv=2),
    "gqa-14q2kv": WORKLOADS[4].with_(Hq=14, Hkv=2),
    "batched-2seq-1h": WORKLOADS[5].with_(B=2, Hq=1, Hkv=1, S_prefix=1000, S_suffix=37),
}


@pytest.mark.parametrize("variant", ["spec", "sharp"])
@pytest.mark.parametrize("name", list(SMALL))
def test_parity_elementwise(name, variant):
    wl = SMALL[name]
    inputs, parent, out = _run(wl, seed_for(wl.cid, 1), variant)
    ok, worst, frac = _check(out, inputs, parent, variant)
    assert ok, f"{name}/{variant}: worst excess {worst:.3g}, {frac:.2%} outside tolerance"


@pytest.mark.parametrize("name", ["8b-tree-2h", "tiny", "gqa-14q2kv"])
def test_wrong_mask_is_detected(name):
    """Discriminating power: the GPU output must NOT match an oracle whose mask
    lets siblings see each other and drops ancestors."""
    wl = SMALL[name]
    inputs, parent, out = _run(wl, seed_for(wl.cid, 2), "sharp")
    wrong_parent = np.where(parent >= 0, -1, parent)  # every draft a root: ancestors dropped
    if (parent >= 0).any():
        ok, _, _ = _check(out, inputs, wrong_parent, "sharp")  # even the widened bound fails
        assert not ok
    # siblings visible: chain every draft to its predecessor
    chain = np.tile(np.arange(-1, wl.N - 1, dtype=np.int32), (wl.B, 1))
    ok, _, _ = _check(out, inputs, chain, "sharp")
    assert not ok


@pytest.mark.parametrize("tiling", ["16", "32"])
@pytest.mark.parametrize("L,N,S,Hq,Hkv,D", [
    (8, 4, 192, 4, 4, 64),      # rows of one wave span 4 drafts
    (40, 5, 70, 2, 1, 128),     # L not a multiple of 32, ragged cache tile
    (1, 7, 3, 3, 1, 64),        # one-token blocks
    (33, 2, 0, 2, 2, 128),      # no cache at all
    (64, 3, 65, 6, 2, 128),     # half-draft row blocks, GQA group 3
    (32, 64, 64, 1, 1, 64),     # 64 drafts (deepest chains)
    (64, 64, 100, 2, 1, 128),   # both maxima: 64 drafts of 64 tokens, a 64-deep chain
    (5, 1, 1, 1, 1, 128),       # single draft, single cache key
])
def test_odd_shapes(L, N, S, Hq, Hkv, D, tiling):
    """Edge shapes under both row tilings of the kernel (16 query rows per wave on one-sequence
    grids, 32 on larger ones: the batch is chosen to fall on either side of the threshold; with
    the larger batch the first and last sequences are checked)."""
    wl = Workload(99, "odd", B=2, N=N, L=L, Hq=Hq, Hkv=Hkv, D=D, S_prefix=S, S_suffix=0, V=64,
                  logits_dtype="f32", margin_max=3.0, parents=None, level_sizes=None)
    B = _tiling_batch(wl, tiling)
    wl = wl.with_(B=B)
    rng = np.random.default_rng(L * 1000 + N)
    parent = np.array([[-1] + [int(rng.integers(-1, n)) for n in range(1, N)] for _ in range(B)],
                      dtype=np.int32)
    if N == 64:
        parent[0] = np.arange(-1, N - 1)
    for variant in ("spec", "sharp"):
        inputs, _, out = _run(wl, 7 + L, variant, parent=parent)
        ok, worst, frac, b = _check_seqs(out, inputs, parent, variant, sorted({0, B - 1}))
        assert ok, f"{variant} B={B} b={b}: worst excess {worst:.3g}, {frac:.2%} bad"


def test_explicit_scale():
    wl = SMALL["tiny"]
    inputs, parent, out = _run(wl, 3, "spec", scale=0.5)
    ok, worst, _ = attn_close(out, _oracle(inputs, parent, scale=0.5))
    assert ok, worst


def test_non_ancestor_perturbation_is_bitwise_invisible():
    wl = SMALL["8b-tree-2h"]
    q, kc, vc, kd, vd = [t.cuda() for t in attention_inputs(wl, 11, "sharp")]
    parent = _parents(wl, 11)
    par = cuda(parent, torch.int32)
    base = tsp.verify_attn(q, kc, vc, kd, vd, par).clone()
    anc = oracle.ancestor_sets(parent[0])
    j = wl.N - 1  # a leaf-level draft; perturb it
    kd2, vd2 = kd.clone(), vd.clone()
    kd2[0, j] = torch.randn_like(kd2[0, j].float()).to(torch.bfloat16)
    vd2[0, j] = torch.randn_like(vd2[0, j].float()).to(torch.bfloat16)
    out = tsp.verify_attn(q, kc, vc, kd2, vd2, par)
    torch.cuda.synchronize()
    for i in range(wl.N):
        same = torch.equal(out[0, i], base[0, i])
        assert same == (j not in anc[i]), i


def test_deterministic_across_runs():
    wl = SMALL["gqa-14q2kv"]
    q, kc, vc, kd, vd = [t.cuda() for t in attention_inputs(wl, 13, "sharp")]
    par = cuda(_parents(wl, 13), torch.int32)
    a = tsp.verify_attn(q, kc, vc, kd, vd, par).clone()
    for _ in range(5):
        b = tsp.verify_attn(q, kc, vc, kd, vd, par)
        assert torch.equal(a, b)


@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_full_size_sampled_heads(cid):
    """Full shapes in the launch configuration the bench times; the oracle
    recomputes a few (sequence, query head) pairs on their own."""
    wl = WORKLOADS[cid]
    q, kc, vc, kd, vd = attention_inputs(wl, seed_for(cid), "spec", device="cuda")
    parent = _parents(wl, seed_for(cid))
    out = tsp.verify_attn(q, kc, vc, kd, vd, cuda(parent, torch.int32))
    torch.cuda.synchronize()
    rng = np.random.default_rng(cid)
    G = wl.Hq // wl.Hkv
    picks = [(0, 0), (wl.B - 1, wl.Hq - 1)] + [(int(rng.integers(wl.B)), int(rng.integers(wl.Hq))) for _ in range(2)]
    for b, h in picks:
        g = h // G
        sub = [q[b:b + 1, :, :, h:h + 1], kc[b:b + 1, :, g:g + 1], vc[b:b + 1, :, g:g + 1],
               kd[b:b + 1, :, :, g:g + 1], vd[b:b + 1, :, :, g:g + 1]]
        ref = _oracle(sub, parent[b:b + 1])
        ok, worst, frac = attn_close(out[b:b + 1, :, :, h:h + 1], ref)
        assert ok, f"{wl.name} b={b} h={h}: worst {worst:.3g} frac {frac:.3%}"


def _wrong_parents(parent, N):
    """Negative controls: every ancestor dropped (when the tree has any), and siblings made
    visible by chaining every draft to its predecessor."""
    out = {"siblings_chained": np.tile(np.arange(-1, N - 1, dtype=np.int32), (parent.shape[0], 1))}
    if (parent >= 0).any():
        out["ancestors_dropped"] = np.full_like(parent, -1)
    return out


@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_full_size_sharp_sampled_heads_and_wrong_masks(cid):
    """The timed launch (full batch, all heads, the workload's parent array) on sharp inputs
    (q ~ 3 N(0,1), k, v ~ N(0,1)): sampled (sequence, query head) slices must match the oracle
    within the sharp-input bound, and the same GPU slices must FAIL that bound against an oracle
    with a wrong mask (ancestors dropped; siblings chained), so a mask error cannot pass here."""
    wl = WORKLOADS[cid]
    q, kc, vc, kd, vd = attention_inputs(wl, seed_for(cid, 3), "sharp", device="cuda")
    parent = _parents(wl, seed_for(cid))
    out = tsp.verify_attn(q, kc, vc, kd, vd, cuda(parent, torch.int32))
    torch.cuda.synchronize()
    rng = np.random.default_rng(100 + cid)
    G = wl.Hq // wl.Hkv
    picks = [(0, 0), (wl.B - 1, wl.Hq - 1)] + [(int(rng.integers(wl.B)), int(rng.integers(wl.Hq))) for _ in range(3)]
    wrong = _wrong_parents(parent, wl.N)
    for b, h in picks:
        g = h // G
        sub = [q[b:b + 1, :, :, h:h + 1], kc[b:b + 1, :, g:g + 1], vc[b:b + 1, :, g:g + 1],
               kd[b:b + 1, :, :, g:g + 1], vd[b:b + 1, :, :, g:g + 1]]
        got = out[b:b + 1, :, :, h:h + 1]
        ok, worst, frac = _check(got, sub, parent[b:b + 1], "sharp")
        assert ok, f"{wl.name} b={b} h={h}: worst excess {worst:.3g}, {frac:.3%} outside"
        for name, wp in wrong.items():
            ok_w, _, frac_w = _check(got, sub, wp[b:b + 1], "sharp")
            assert not ok_w, f"{wl.name} b={b} h={h}: the GPU output also matches a mask with {name}"
            assert frac_w > 0.01, f"{wl.name} b={b} h={h} {name}: only {frac_w:.3%} outside"


def test_invalid_parent_is_flagged_and_bounded():
    wl = SMALL["tiny"]
    tsp.device_status(reset=True)
    bad = np.array([[-1, 3, 0, 9]], dtype=np.int32)  # 3 >= 1 and 9 >= 3: not topological
    inputs, _, out = _run(wl, 5, "sharp", parent=bad)
    assert tsp.device_status(reset=True) & tsp.DEV_BAD_PARENT
    fixed = np.array([[-1, -1, 0, -1]], dtype=np.int32)  # what the kernel falls back to
    ok, worst, _ = _check(out, inputs, fixed, "sharp")
    assert ok, worst


def test_bad_shapes_raise():
    wl = SMALL["tiny"]
    q, kc, vc, kd, vd = [t.cuda() for t in attention_inputs(wl, 1)]
    par = cuda(_parents(wl, 1), torch.int32)
    with pytest.raises(tsp.TrajSpecError):  # head_dim 96 unsupported
        tsp.verify_attn(q[..., :48].contiguous(), kc[..., :48].contiguous(), vc[..., :48].contiguous(),
                        kd[..., :48].contiguous(), vd[..., :48].contiguous(), par)


@pytest.mark.parametrize("tiling", ["16", "32"])
@pytest.mark.parametrize("S", [1, 63, 64, 65, 127, 128, 129, 191, 192, 193, 255, 256, 257, 320, 383, 384, 449])
def test_cache_lengths_cover_every_tail_path(S, tiling):
    """The cache loop runs full tiles in pairs and peels 0-2 full tiles plus a last
    (ragged or full) tile: every cache length class in 64-key tiles must agree, under both row
    tilings."""
    wl = Workload(98, "cache-len", B=1, N=3, L=32, Hq=2, Hkv=1, D=128, S_prefix=S, S_suffix=0, V=64,
                  logits_dtype="f32", margin_max=3.0, parents=(-1, 0, 0), level_sizes=None)
    B = _tiling_batch(wl, tiling)
    wl = wl.with_(B=B)
    parent = np.tile(np.array([[-1, 0, 0]], dtype=np.int32), (B, 1))
    for variant in ("spec", "sharp"):
        inputs, _, out = _run(wl, 1000 + S, variant, parent=parent)
        ok, worst, frac, b = _check_seqs(out, inputs, parent, variant, sorted({0, B - 1}))
        assert ok, f"S={S} {variant} B={B} b={b}: worst excess {worst:.3g}, {frac:.2%} bad"


@pytest.mark.parametrize("tiling", ["16", "32"])
@pytest.mark.parametrize("where", ["block0", "main_loop", "tail_stage", "partial_block", "ancestor_draft", "own_draft"])
def test_reference_moves_late(where, tiling):
    """Keys whose scores jump far above every earlier block (about 25 powers of two on the
    sharp inputs) force the lazy reference to move and O and the running sum to be rescaled at
    that point: in the first block, inside the paired stage loop, in the tail stages, in the
    partial last block, or in the draft phase.  The result must still match the oracle."""
    wl = Workload(97, "jump", B=1, N=4, L=32, Hq=2, Hkv=1, D=128, S_prefix=700, S_suffix=0, V=64,
                  logits_dtype="f32", margin_max=3.0, parents=(-1, 0, 1, 1), level_sizes=None)
    wl = wl.with_(B=_tiling_batch(wl, tiling))
    parent = np.tile(np.array([[-1, 0, 1, 1]], dtype=np.int32), (wl.B, 1))
    q, kc, vc, kd, vd = attention_inputs(wl, 4242, "sharp")
    # 700 keys = 22 blocks of 32: blocks 0-15 run in the paired stage loop, 16-21 in the tail
    # stages, block 21 is partial (keys 672-699)
    sel = {"block0": (kc, slice(0, 32)), "main_loop": (kc, slice(200, 210)), "tail_stage": (kc, slice(580, 600)),
           "partial_block": (kc, slice(680, 690)), "ancestor_draft": (kd, 1), "own_draft": (kd, 3)}[where]
    t, idx = sel
    kc, kd = kc.clone(), kd.clone()
    if t is kc:
        kc[0, idx] = (kc[0, idx].float() * 3.0).to(torch.bfloat16)
    else:
        kd[0, idx] = (kd[0, idx].float() * 3.0).to(torch.bfloat16)
    inputs = (q, kc, vc, kd, vd)
    out = tsp.verify_attn(*[x.cuda() for x in inputs], cuda(parent, torch.int32))
    torch.cuda.synchronize()
    ok, worst, frac, _ = _check_seqs(out, inputs, parent, "sharp", [0])  # the jump is in sequence 0
    assert ok, f"{where}: worst excess {worst:.3g}, {frac:.2%} outside tolerance"
