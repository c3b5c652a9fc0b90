"""GPU parity: traj_verify_layer against the layer oracle (same bf16 rounding points, fp64
arithmetic).  The two differ by fp32 accumulation order in the GEMMs and the attention and by
the bf16 roundings those move across a boundary (2^-8 relative each), compounded through the
layer: elementwise |gpu - ref| <= 0.03 |ref| + 0.03 rms(ref), and the mean error below 2e-3
rms(ref)."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_27514_amd as tsp
from helpers import cuda
from paper_2608_27514_amd import _lib
from oracle.layer import bf16_round

pytestmark = pytest.mark.gpu


def _weights(rng, hidden, Hq, Hkv, D, inter):
    f = lambda *s: bf16_round(rng.standard_normal(s) / math.sqrt(s[0]))  # noqa: E731
    return {"attn_norm": bf16_round(1 + 0.1 * rng.standard_normal(hidden)), "w_qkv": f(hidden, (Hq + 2 * Hkv) * D),
            "w_o": f(Hq * D, hidden), "mlp_norm": bf16_round(1 + 0.1 * rng.standard_normal(hidden)),
            "w_gate_up": f(hidden, 2 * inter), "w_down": f(inter, hidden)}


@pytest.mark.parametrize("B,N,L,Hq,Hkv,D,S,inter,tree", [
    (2, 4, 8, 2, 2, 128, 64, 512, [-1, 0, 0, 1]),
    (1, 7, 32, 4, 2, 64, 100, 384, [-1, 0, 0, 0, 1, 2, 4]),   # W3D3 hybrid tree, GQA, D 64
    (3, 2, 5, 1, 1, 128, 0, 136, [-1, -1]),                   # no cache, ragged sizes
    (1, 3, 8, 8, 4, 128, 40, 3072, [-1, 0, 1]),               # few rows: split-K projections
    (1, 64, 64, 2, 1, 128, 50, 256, [-1] + list(range(63))),  # both maxima: a 64-deep chain of 64-token drafts
])
def test_layer_parity(B, N, L, Hq, Hkv, D, S, inter, tree):
    rng = np.random.default_rng(B * 100 + N)
    hidden = Hq * D
    x = bf16_round(rng.standard_normal((B, N, L, hidden)))
    w = _weights(rng, hidden, Hq, Hkv, D, inter)
    kc = bf16_round(rng.standard_normal((B, S, Hkv, D)))
    vc = bf16_round(rng.standard_normal((B, S, Hkv, D)))
    parent = np.array([tree] * B, dtype=np.int32)
    pos0 = rng.integers(0, 4000, B).astype(np.int32)
    ref = oracle.verify_layer(x, w, kc, vc, parent, Hq, pos0=pos0, rms_eps=1e-5, rope_theta=500000.0)
    bf = lambda a: cuda(np.asarray(a, dtype=np.float32), torch.bfloat16)  # noqa: E731
    xg = bf(x)
    out = tsp.verify_layer(xg, {k: bf(v) for k, v in w.items()}, bf(kc), bf(vc), cuda(parent, torch.int32), Hq,
                           pos0=cuda(pos0, torch.int32), rms_eps=1e-5, rope_theta=500000.0)
    torch.cuda.synchronize()
    g = out.float().cpu().numpy().astype(np.float64)
    err = np.abs(g - ref)
    rms = math.sqrt(float(np.mean(ref * ref)))
    assert (err <= 0.03 * np.abs(ref) + 0.03 * rms).all(), float((err - 0.03 * np.abs(ref) - 0.03 * rms).max())
    assert float(err.mean()) < 2e-3 * rms, float(err.mean()) / rms


def test_layer_is_in_place_and_reports_bad_arguments():
    rng = np.random.default_rng(5)
    B, N, L, Hq, Hkv, D, S, inter = 1, 2, 4, 1, 1, 128, 16, 256
    bf = lambda a: cuda(np.asarray(a, dtype=np.float32), torch.bfloat16)  # noqa: E731
    x = bf(rng.standard_normal((B, N, L, Hq * D)))
    w = {k: bf(v) for k, v in _weights(rng, Hq * D, Hq, Hkv, D, inter).items()}
    kc, vc = bf(rng.standard_normal((B, S, Hkv, D))), bf(rng.standard_normal((B, S, Hkv, D)))
    par = cuda(np.array([[-1, 0]]), torch.int32)
    ptr = x.data_ptr()
    out = tsp.verify_layer(x, w, kc, vc, par, Hq)
    assert out.data_ptr() == ptr
    small = torch.empty(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(tsp.TrajSpecError):
        tsp.verify_layer(x, w, kc, vc, par, Hq, workspace=small)


# ---------------------------------------------------------------- the projection GEMM alone
# The GPU accumulates bf16 products in fp32 (K / 16 dependent MFMA steps) and rounds once to
# bf16; against the exact value: |gpu - ref| <= 2^-8 |ref| + 2^-15 (|x| @ |w| + |y0|).

def _linear_bound(a, w, y0, ref):
    mag = np.abs(a) @ np.abs(w) + (0 if y0 is None else np.abs(y0))
    return 2.0 ** -8 * np.abs(ref) + 2.0 ** -15 * mag


@pytest.mark.parametrize("M,K,N,acc", [
    (1, 8, 8, False), (37, 512, 1000, False), (130, 72, 136, True), (129, 200, 264, True),
    (256, 4096, 256, False), (300, 136, 1032, True), (5, 4104, 8, False), (128, 64, 128, True),
    # grids of >= 256 tiles of 256 x 256 take the large-tile kernel: ragged M, N and K edges
    (4133, 200, 4104, False), (4133, 136, 4104, True), (4096, 8, 4096, False), (4352, 4160, 3848, True),
    # few tiles: K split over workgroups (fp32 partials in the workspace, then one reduction)
    (300, 2048, 264, True), (130, 1088, 136, True), (224, 3080, 520, False),
    # one or two drafts' rows (17 .. 64) and up to 255: ragged rows, columns and k, split and not
    (17, 1000, 264, True), (32, 72, 4104, False), (33, 136, 520, True), (64, 4104, 136, True),
    (50, 8, 8, False), (129, 4096, 1032, True), (255, 520, 8200, False),
])
def test_linear_parity(M, K, N, acc):
    rng = np.random.default_rng(M * 7 + K + N)
    a = bf16_round(rng.standard_normal((M, K)))
    w = bf16_round(rng.standard_normal((K, N)) / math.sqrt(K))
    y0 = bf16_round(rng.standard_normal((M, N))) if acc else None
    ref = oracle.linear(a, w, y0)
    bf = lambda v: cuda(np.asarray(v, dtype=np.float32), torch.bfloat16)  # noqa: E731
    y = bf(y0) if acc else None
    out = tsp.linear(bf(a), bf(w), y=y, accumulate=acc)
    torch.cuda.synchronize()
    g = out.float().cpu().numpy().astype(np.float64)
    assert (np.abs(g - ref) <= _linear_bound(a, w, y0, ref)).all()
    assert np.mean(g == bf16_round(ref)) > 0.95  # mostly the correctly rounded value


@pytest.mark.parametrize("M,K,N,acc", [
    (3584, 4096, 12288, False),   # QKV projection, 16 sequences x W3D3 drafts (7 x 32 tokens)
    (3584, 12288, 4096, True),    # down projection + residual
    (32768, 4096, 12288, False),  # QKV projection, 16 sequences x 64 drafts x 32 tokens
    (224, 4096, 126464, False),   # LM head of one sequence's W3D3 drafts
    (224, 12288, 4096, True),     # one sequence's down projection + residual (split K)
    (224, 4096, 4096, True),      # one sequence's O projection + residual (split K)
    (32, 4096, 12288, False),     # one draft: QKV projection (split K)
    (32, 12288, 4096, True),      # one draft: down projection + residual (split K)
    (64, 4096, 24576, False),     # two drafts: gate / up projection
    (64, 4096, 126464, False),    # two drafts: LM head
])
def test_linear_full_size_sampled_rows(M, K, N, acc):
    """8B-shaped projections in the launch configuration the benchmark times; the oracle checks
    48 sampled rows (first, last, random) in full."""
    g = torch.Generator(device="cuda")
    g.manual_seed(M + N)
    a = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn(K, N, device="cuda", generator=g) / math.sqrt(K)).to(torch.bfloat16)
    y0 = torch.randn(M, N, device="cuda", generator=g).to(torch.bfloat16) if acc else None
    y = y0.clone() if acc else None
    out = tsp.linear(a, w, y=y, accumulate=acc)
    torch.cuda.synchronize()
    rng = np.random.default_rng(M)
    rows = np.unique(np.concatenate([[0, M - 1], rng.integers(0, M, 46)]))
    ridx = torch.as_tensor(rows, device="cuda")
    a_s = a[ridx].double().cpu().numpy()
    w_h = w.double().cpu().numpy()
    y_s = y0[ridx].double().cpu().numpy() if acc else None
    ref = oracle.linear(a_s, w_h, y_s)
    got = out[ridx].double().cpu().numpy()
    assert (np.abs(got - ref) <= _linear_bound(a_s, w_h, y_s, ref)).all()


def test_linear_split_and_unsplit_agree():
    """A shape that splits K runs unsplit without a workspace; both are within the bound of the
    exact product, and the split path is the one taken with a workspace."""
    M, K, N = 224, 12288, 4096
    assert tsp.linear_workspace_size(M, K, N) > 0
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    a = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn(K, N, device="cuda", generator=g) / math.sqrt(K)).to(torch.bfloat16)
    split = tsp.linear(a, w)
    unsplit = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    st = _lib._lib().traj_linear(a.data_ptr(), w.data_ptr(), unsplit.data_ptr(), M, K, N, 0, None, 0,
                                 torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    rows = np.array([0, 17, 111, 223])
    a_s = a[torch.as_tensor(rows, device="cuda")].double().cpu().numpy()
    w_h = w.double().cpu().numpy()
    ref = oracle.linear(a_s, w_h)
    for out in (split, unsplit):
        got = out[torch.as_tensor(rows, device="cuda")].double().cpu().numpy()
        assert (np.abs(got - ref) <= _linear_bound(a_s, w_h, None, ref)).all()


def test_linear_rejects_bad_shapes():
    x = torch.zeros(4, 60, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tsp.TrajSpecError):
        tsp.linear(x, torch.zeros(60, 64, dtype=torch.bfloat16, device="cuda"))
    with pytest.raises(ValueError):
        tsp.linear(x, torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda"))


# ---------------------------------------------------------------- dual-cache refresh (App. A)

@pytest.mark.parametrize("B,S,L,Hq,Hkv,D,inter,starts", [
    (2, 40, 8, 2, 2, 128, 512, [0, 40]),          # block first / last
    (1, 70, 5, 4, 2, 64, 384, [33]),              # GQA, D 64, ragged lengths
    (2, 100, 32, 8, 4, 128, 3072, [64, 0]),       # few rows: split-K projections
])
def test_refresh_layer_parity(B, S, L, Hq, Hkv, D, inter, starts):
    rng = np.random.default_rng(S * 10 + L)
    hidden = Hq * D
    x = bf16_round(rng.standard_normal((B, S + L, hidden)))
    w = _weights(rng, hidden, Hq, Hkv, D, inter)
    ref, ref_k, ref_v = oracle.refresh_layer(x, w, starts, L, Hq, Hkv)
    bf = lambda a: cuda(np.asarray(a, dtype=np.float32), torch.bfloat16)  # noqa: E731
    xg = bf(x)
    out, kc, vc = tsp.refresh_layer(xg, {k: bf(v) for k, v in w.items()}, cuda(np.array(starts), torch.int32),
                                    Hq, Hkv, L)
    torch.cuda.synchronize()
    assert out.data_ptr() == xg.data_ptr()
    for got, want in ((out, ref), (kc, ref_k), (vc, ref_v)):
        g = got.float().cpu().numpy().astype(np.float64)
        err = np.abs(g - want)
        rms = math.sqrt(float(np.mean(want * want)))
        assert (err <= 0.03 * np.abs(want) + 0.03 * rms).all(), float((err - 0.03 * np.abs(want) - 0.03 * rms).max())
        assert float(err.mean()) < 2e-3 * rms


def test_refresh_then_verify_root_state_agrees():
    """Refresh a sequence's cache at a block boundary, then verify the block's current state as
    the only draft against that cache: the verification layer's output equals the refresh
    layer's output for the block rows (same visible keys and positions, different kernels)."""
    rng = np.random.default_rng(77)
    B, S, L, Hq, Hkv, D, inter = 2, 96, 32, 4, 2, 128, 1024
    hidden = Hq * D
    x = bf16_round(rng.standard_normal((B, S + L, hidden)))
    w = {k: cuda(np.asarray(v, dtype=np.float32), torch.bfloat16)
         for k, v in _weights(rng, hidden, Hq, Hkv, D, inter).items()}
    starts = np.array([32, 96], dtype=np.int32)
    xg = cuda(np.asarray(x, dtype=np.float32), torch.bfloat16)
    blocks = torch.stack([xg[b, starts[b]:starts[b] + L] for b in range(B)])[:, None].contiguous()  # [B,1,L,h]
    out, kc, vc = tsp.refresh_layer(xg, w, cuda(starts, torch.int32), Hq, Hkv, L)
    ver = tsp.verify_layer(blocks, w, kc, vc, cuda(np.full((B, 1), -1), torch.int32), Hq,
                           pos0=cuda(starts, torch.int32))
    torch.cuda.synchronize()
    # both sides round every stored activation to bf16 but accumulate in different orders
    # (one pass over all keys against cache-then-block; different GEMM tilings), so they agree
    # to the layer's compounded rounding: the bound of the layer parity test
    for b in range(B):
        a = ver[b, 0].float().cpu().numpy().astype(np.float64)
        r = out[b, starts[b]:starts[b] + L].float().cpu().numpy().astype(np.float64)
        err = np.abs(a - r)
        rms = math.sqrt(float(np.mean(r * r)))
        assert (err <= 0.03 * np.abs(r) + 0.03 * rms).all()
        assert float(err.mean()) < 2e-3 * rms


def test_refresh_reports_a_block_outside_the_sequence():
    rng = np.random.default_rng(5)
    B, S, L, Hq, Hkv, D, inter = 2, 16, 4, 1, 1, 64, 128
    x = cuda(np.asarray(bf16_round(rng.standard_normal((B, S + L, Hq * D))), dtype=np.float32), torch.bfloat16)
    w = {k: cuda(np.asarray(v, dtype=np.float32), torch.bfloat16)
         for k, v in _weights(rng, Hq * D, Hq, Hkv, D, inter).items()}
    tsp.device_status(reset=True)
    _, kc, _ = tsp.refresh_layer(x, w, cuda(np.array([3, 99]), torch.int32), Hq, Hkv, L)
    assert tsp.device_status(reset=True) & tsp.DEV_BAD_BLOCK
    assert torch.isfinite(kc.float()).all()


# ---------------------------------------------------------------- full size, sampled root paths
# The layer at the 8B shape (hidden 4096, 32 heads of 128, MLP 12288) in the two launch
# configurations the benchmark times.  A draft's output rows depend only on the drafts of its
# root path (trajectory mask) and its own rows elsewhere, so the oracle checks a sampled draft
# by running the whole layer on that path alone (re-indexed parents, same cache and positions).

def _root_path(parent_row, n):
    path = [n]
    while parent_row[path[-1]] != -1:
        path.append(int(parent_row[path[-1]]))
    return path[::-1]


@pytest.mark.parametrize("config", ["batched", "one_sequence"])
def test_layer_full_size_sampled_paths(config):
    from synthetic.workloads import build_tree
    Hq = Hkv = 32
    D, L, hidden, inter = 128, 32, 4096, 12288
    rng = np.random.default_rng(606)
    if config == "batched":  # 16 sequences x 64 drafts (3/9/27/25 per level), cache 3584 + 512
        B, N, S, S_prefix = 16, 64, 4096, 3584
        parent = np.stack([build_tree((3, 9, 27, 25), rng)[0] for _ in range(B)]).astype(np.int32)
        samples = [(0, N - 1), (B - 1, int(rng.integers(0, N))), (int(rng.integers(1, B - 1)), 0)]
    else:  # one sequence, W3D3 hybrid tree, cache 512 + 224
        B, N, S, S_prefix = 1, 7, 736, 512
        parent = np.array([[-1, 0, 0, 0, 1, 2, 4]], dtype=np.int32)
        samples = [(0, 6), (0, 3)]
    g = torch.Generator(device="cuda")
    g.manual_seed(607)

    def r(*shape, scale=1.0):
        return (torch.randn(*shape, device="cuda", generator=g) * scale).to(torch.bfloat16)

    w = {"attn_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16), "w_qkv": r(hidden, 3 * hidden,
                                                                                   scale=hidden ** -0.5),
         "w_o": r(hidden, hidden, scale=hidden ** -0.5), "mlp_norm": (1 + 0.1 * r(hidden).float()).to(torch.bfloat16),
         "w_gate_up": r(hidden, 2 * inter, scale=hidden ** -0.5), "w_down": r(inter, hidden, scale=inter ** -0.5)}
    x0 = r(B, N, L, hidden)
    kc, vc = r(B, S, Hkv, D), r(B, S, Hkv, D)
    pos0 = torch.full((B,), S_prefix, dtype=torch.int32, device="cuda")
    ws = torch.empty(tsp.layer_workspace_size(B, N, L, Hq, Hkv, D, S, hidden, inter), dtype=torch.uint8,
                     device="cuda")
    x = x0.clone()
    tsp.verify_layer(x, w, kc, vc, cuda(parent, torch.int32), Hq, pos0=pos0, workspace=ws)
    torch.cuda.synchronize()
    f64 = lambda t: t.float().cpu().numpy().astype(np.float64)  # noqa: E731
    wn = {k: f64(v) for k, v in w.items()}
    for b, n in samples:
        path = _root_path(parent[b], n)
        sub_parent = np.array([[-1] + list(range(len(path) - 1))], dtype=np.int32)
        idx = torch.tensor(path, device="cuda")
        ref = oracle.verify_layer(f64(x0[b, idx])[None], wn, f64(kc[b])[None], f64(vc[b])[None], sub_parent, Hq,
                                  pos0=np.array([S_prefix]), rms_eps=1e-5, rope_theta=500000.0)[0]
        got = f64(x[b, idx])
        err = np.abs(got - ref)
        rms = math.sqrt(float(np.mean(ref * ref)))
        assert (err <= 0.03 * np.abs(ref) + 0.03 * rms).all(), (b, n, float((err - 0.03 * np.abs(ref)).max()))
        assert float(err.mean()) < 2e-3 * rms, (b, n, float(err.mean()) / rms)
