"""The C-ABI library loads, exports every declared symbol, and rejects invalid
arguments before touching the device (CPU only: no compute calls)."""

import ctypes
import os
import re

import pytest

from paper_2608_27514_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "traj_spec.h")

needs_lib = pytest.mark.skipif(not os.path.exists(_lib.LIB_PATH), reason="libtrajspec.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(traj_[a-z_]+)\s*\(", text)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for fn in ("traj_verify_attn", "traj_confidence_topk", "traj_accept"):
        assert fn in names


@needs_lib
def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(_lib.EXPORTS)


@needs_lib
def test_status_strings_and_version():
    lib = _lib.load()
    assert lib.traj_version().decode().startswith("libtrajspec")
    # the binary carries the digest of the sources it was built from: it must be these
    from paper_2608_27514_amd.build import source_digest
    assert _lib.built_digest() == source_digest()
    assert _lib.check_build() == source_digest()
    for st in range(8):
        assert lib.traj_status_string(st)
    assert lib.traj_status_string(1234) == b"unknown status"


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


@needs_lib
def test_attention_argument_errors():
    lib = _lib.load()
    good = _lib.AttnShape(1, 4, 8, 4, 4, 64, 192, 0.0)

    def call(shape, ptrs=None):
        p = ptrs or [FAKE] * 7
        return lib.traj_verify_attn(*p, ctypes.byref(shape), None, 0, None)

    assert call(good, [None] + [FAKE] * 6) == 1
    assert call(good, [FAKE] * 6 + [None]) == 1
    assert call(_lib.AttnShape(1, 4, 8, 4, 3, 64, 192, 0.0)) == 2    # Hq % Hkv
    assert call(_lib.AttnShape(1, 65, 8, 4, 4, 64, 192, 0.0)) == 2   # N > 64
    assert call(_lib.AttnShape(1, 4, 0, 4, 4, 64, 192, 0.0)) == 2    # L = 0
    assert call(_lib.AttnShape(1, 4, 8, 4, 4, 96, 192, 0.0)) == 4    # head dim
    # one sequence's cache slice (S * Hkv * D * 2 bytes) is addressed with 32-bit offsets
    assert call(_lib.AttnShape(1, 4, 8, 8, 8, 128, 1 << 20, 0.0)) == 4
    assert call(_lib.AttnShape(1, 4, 8, 4, 4, 64, 192, float("nan"))) == 7
    mis = [ctypes.c_void_p(0x1002)] + [FAKE] * 6
    assert call(good, mis) == 2                                       # misaligned q
    assert lib.traj_verify_attn(*([FAKE] * 7), None, None, 0, None) == 1
    assert lib.traj_verify_attn_workspace_size(ctypes.byref(good)) == 0


@needs_lib
def test_logits_argument_errors():
    lib = _lib.load()

    def call(shape, k, logits=FAKE, ws=None, ws_bytes=0):
        return lib.traj_confidence_topk(logits, k, FAKE, FAKE, ctypes.byref(shape), ws, ws_bytes, None)

    good = _lib.LogitsShape(256, 126464, 126464, 0)
    assert call(_lib.LogitsShape(4, 100, 100, 9), 3) == 3            # dtype
    assert call(_lib.LogitsShape(4, 100, 99, 0), 3) == 2             # stride < vocab
    assert call(good, 0) == 7 and call(good, 9) == 7                  # k range
    assert call(_lib.LogitsShape(4, 2, 2, 1), 3) == 7                 # k > vocab
    assert call(good, 3, logits=None) == 1
    few = _lib.LogitsShape(40, 126464, 126464, 0)                    # a short batch: rows are split
    need = lib.traj_confidence_topk_workspace_size(ctypes.byref(few), 3)
    assert need > 0
    assert call(few, 3, ws=FAKE, ws_bytes=need - 1) == 5              # too small
    assert call(few, 3, ws=ctypes.c_void_p(0x1004), ws_bytes=need) == 5  # misaligned
    for rows in (256, 1024, 32768):                                   # enough rows: never split
        big = _lib.LogitsShape(rows, 126464, 126464, 0)
        assert lib.traj_confidence_topk_workspace_size(ctypes.byref(big), 3) == 0


@needs_lib
def test_noalloc_logit_pass_arguments_and_scratch_bound():
    lib = _lib.load()

    def call(shape, k, logits=FAKE):
        return lib.traj_confidence_topk_noalloc(logits, k, FAKE, FAKE, ctypes.byref(shape), None)

    assert call(_lib.LogitsShape(4, 100, 100, 9), 3) == 3
    assert call(_lib.LogitsShape(4, 100, 99, 0), 3) == 2
    assert call(_lib.LogitsShape(4, 100, 100, 0), 9) == 7
    assert call(_lib.LogitsShape(4, 100, 100, 0), 3, logits=None) == 1
    assert call(_lib.LogitsShape(0, 100, 100, 0), 3, logits=None) == 0  # no rows: nothing to do
    assert lib.traj_confidence_topk_noalloc(FAKE, 3, FAKE, FAKE, None, None) == 1
    # every shape the plan splits fits the fixed scratch (so the entry point never refuses one)
    limit = int(re.search(r"#define TRAJ_TOPK_SCRATCH_BYTES (\d+)", open(HEADER).read()).group(1))
    worst = 0
    for dtype in (0, 1):
        for rows in range(1, 600):
            for vocab in (1000, 32000, 126464, 152064, 262144, (1 << 31) - 1):
                sh = _lib.LogitsShape(rows, vocab, vocab, dtype)
                worst = max(worst, lib.traj_confidence_topk_workspace_size(ctypes.byref(sh), 8))
    assert 0 < worst <= limit, worst


@needs_lib
def test_accept_argument_errors():
    lib = _lib.load()
    f = 0x1000
    acc = _lib.Accepted(f, f, f, f, f)

    def call(dr, conf=FAKE, tau=0.9, ac=acc):
        return lib.traj_accept(conf, FAKE, ctypes.byref(dr), tau, ctypes.byref(ac), None)

    good = dict(B=1, N=4, L=8, k=3, tokens=f, parent=f, committed=f, conf0=f, idx0=f, mode=0, traversal=0)
    assert call(_lib.Drafts(**good), conf=None) == 1
    assert call(_lib.Drafts(**{**good, "tokens": None})) == 1
    assert call(_lib.Drafts(**good), ac=_lib.Accepted(f, f, f, f, 0)) == 1
    assert call(_lib.Drafts(**{**good, "N": 65})) == 2
    assert call(_lib.Drafts(**{**good, "L": 65})) == 2
    assert call(_lib.Drafts(**{**good, "k": 9})) == 7
    assert call(_lib.Drafts(**{**good, "mode": 3})) == 7
    assert call(_lib.Drafts(**{**good, "traversal": 2})) == 7
    assert call(_lib.Drafts(**good), tau=float("nan")) == 7


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2608_27514_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "oracle/" not in text, fn


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "nope.so"))
    monkeypatch.setattr(_lib, "_LIB", None)
    with pytest.raises(RuntimeError, match="not built"):
        _lib.load()


@needs_lib
def test_tree_argument_errors_and_max_nodes():
    from oracle.tree import level_widths

    lib = _lib.load()

    def shape(**kw):
        d = dict(B=2, L=8, k=3, n_prev=0, width=3, depth=3, branch=3, full=0, n_max=7, branch_deep=1)
        d.update(kw)
        return _lib.TreeShape(**d)

    def call(sh, tau=0.9, state=FAKE, conf0=FAKE, leaf=None, conf=None, idx=None, nxt=(None, None)):
        return lib.traj_build_tree(state, leaf, conf, idx, conf0, FAKE, ctypes.byref(sh), tau, FAKE, FAKE, FAKE,
                                   None, nxt[0], nxt[1], None)

    assert call(shape(), state=None) == 1
    assert call(shape(), conf0=None) == 1
    assert call(shape(n_prev=4), leaf=FAKE) == 1                 # leaf given, conf/idx missing
    assert call(shape(), nxt=(FAKE, None)) == 1                  # conf_next without idx_next
    assert call(shape(k=9)) == 7 and call(shape(branch=4)) == 7 and call(shape(full=2)) == 7
    assert call(shape(branch_deep=0)) == 7 and call(shape(branch_deep=4)) == 7
    assert call(shape(), tau=float("nan")) == 7
    assert call(shape(L=65)) == 2 and call(shape(n_max=6)) == 2 and call(shape(n_max=65)) == 2
    assert call(shape(width=0)) == 2 and call(shape(depth=-1)) == 2
    for W, D, br, full, L, bd in [(3, 3, 3, 0, 8, 1), (3, 3, 3, 1, 8, 1), (2, 5, 3, 0, 8, 1), (4, 2, 2, 0, 8, 1),
                                  (1, 1, 1, 0, 8, 1), (3, 0, 3, 0, 8, 1), (3, 6, 2, 1, 4, 1), (8, 8, 8, 1, 64, 1),
                                  (2, 2, 2, 1, 8, 2), (4, 3, 2, 1, 8, 2), (6, 4, 1, 0, 16, 3)]:
        cnt, total = 0, 1
        for level, w in enumerate(level_widths(W, min(D, L), bool(full)), start=1):
            cnt = min(br, w) if level == 1 else min(w, cnt * bd)
            total += cnt
        sh = shape(width=W, depth=D, branch=br, full=full, L=L, k=8, branch_deep=bd)
        assert lib.traj_tree_max_nodes(ctypes.byref(sh)) == total


@needs_lib
def test_interblock_argument_errors():
    lib = _lib.load()
    sh = _lib.AttnShape(1, 4, 8, 4, 4, 64, 192, 0.0)
    p7 = [FAKE] * 6
    assert lib.traj_verify_attn_peers(*p7, None, None, ctypes.byref(sh), None, 0, None) == 1   # out NULL
    assert lib.traj_verify_attn_peers(None, *([FAKE] * 5), None, FAKE, ctypes.byref(sh), None, 0, None) == 1
    bad = _lib.AttnShape(1, 65, 8, 4, 4, 64, 192, 0.0)
    assert lib.traj_verify_attn_peers(*p7, FAKE, FAKE, ctypes.byref(bad), None, 0, None) == 2

    def trig(state=FAKE, conf=FAKE, B=2, L=8, k=3, tau=0.9, out=FAKE):
        return lib.traj_interblock_trigger(state, conf, B, L, k, tau, out, None, None, None)

    assert trig(state=None) == 1 and trig(conf=None) == 1 and trig(out=None) == 1
    assert trig(B=0) == 2 and trig(L=0) == 2 and trig(L=65) == 2
    assert trig(k=0) == 7 and trig(k=9) == 7 and trig(tau=float("nan")) == 7


@needs_lib
def test_joint_peers_argument_errors():
    lib = _lib.load()
    assert lib.traj_joint_peers(2, 3, 2, None, None, None, None) == 1      # peers NULL
    assert lib.traj_joint_peers(0, 3, 2, None, None, FAKE, None) == 2
    assert lib.traj_joint_peers(2, 0, 2, None, None, FAKE, None) == 2
    assert lib.traj_joint_peers(2, 3, 0, None, None, FAKE, None) == 2
    assert lib.traj_joint_peers(2, 60, 5, None, None, FAKE, None) == 2     # more than 64 drafts


@needs_lib
def test_layer_and_linear_argument_errors():
    lib = _lib.load()
    odd = ctypes.c_void_p(0x1008)  # 8-byte aligned only
    def lin(M, K, N, acc=0, x=FAKE, y=FAKE, ws=None, ws_bytes=0):
        return lib.traj_linear(x, FAKE, y, M, K, N, acc, ws, ws_bytes, None)

    assert lin(0, 64, 64) == 0                      # M == 0: nothing to do
    assert lin(4, 60, 64) == 2                      # K % 8
    assert lin(4, 64, 4) == 2                       # N < 8
    assert lin(-1, 64, 64) == 2
    assert lin(4, 64, 1 << 31) == 4                 # N past 32-bit offsets
    assert lin(4, (1 << 22) + 8, 64) == 4
    assert lin(4, 64, 64, x=None) == 1
    assert lin(4, 64, 64, acc=1, y=odd) == 2        # alignment
    need = lib.traj_linear_workspace_size(224, 12288, 4096)  # one sequence's down projection: split
    assert need >= 224 * 4096 * 4 * 2 and need % (224 * 4096 * 4) == 0
    assert lib.traj_linear_workspace_size(32768, 4096, 12288) == 0   # fills the chip unsplit
    assert lib.traj_linear_workspace_size(37, 512, 1000) == 0        # too little K to split
    assert lin(224, 12288, 4096, ws=FAKE, ws_bytes=need - 16) == 5
    assert lin(224, 12288, 4096, ws=odd, ws_bytes=need) == 5
    sh = _lib.AttnShape(1, 2, 4, 2, 2, 64, 16, 0.0)
    assert lib.traj_verify_layer_workspace_size(ctypes.byref(sh), ctypes.byref(_lib.LayerDims(128, 256, 1e-5, 5e5))) > 0
    for dims in (_lib.LayerDims(96, 256, 1e-5, 5e5), _lib.LayerDims(128, 12, 1e-5, 5e5),
                 _lib.LayerDims(128, 256, -1.0, 5e5), _lib.LayerDims(128, 256, 1e-5, 0.0)):
        assert lib.traj_verify_layer_workspace_size(ctypes.byref(sh), ctypes.byref(dims)) == 0
    w = _lib.LayerWeights(*[0x1000] * 6)
    dims = _lib.LayerDims(128, 256, 1e-5, 5e5)

    def call(shape=sh, dm=dims, weights=w, ws_bytes=1 << 30, x=FAKE):
        return lib.traj_verify_layer(x, ctypes.byref(weights), ctypes.byref(dm), FAKE, FAKE, FAKE, None,
                                     ctypes.byref(shape), FAKE, ws_bytes, None)

    assert call(dm=_lib.LayerDims(96, 256, 1e-5, 5e5)) == 2
    assert call(x=None) == 1
    assert call(weights=_lib.LayerWeights(*([0x1000] * 5 + [0]))) == 1
    assert call(weights=_lib.LayerWeights(*([0x1000] * 5 + [0x1008]))) == 2
    assert call(ws_bytes=16) == 5


FLOOR_LIB = os.path.join(ROOT, "paper_2608_27514_amd", "libtrajfloor.so")


@pytest.mark.skipif(not os.path.exists(FLOOR_LIB), reason="libtrajfloor.so not built")
def test_floor_library_rejects_shapes_off_the_vector_path():
    """The logit pass's read-only floor (a measurement aid) refuses what the pass's vector path
    would not take, before any launch."""
    lib = ctypes.CDLL(FLOOR_LIB)
    fn = lib.traj_floor_logit_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p]
    sink = FAKE
    assert fn(None, 4, 1024, 1024, 2, sink, None, None) == -1            # no data
    assert fn(FAKE, 4, 1024, 1024, 2, None, None, None) == -1            # no sink
    assert fn(FAKE, 4, 1001, 1001, 2, sink, None, None) == -1            # rows not whole 16-byte vectors
    assert fn(ctypes.c_void_p(0x1002), 4, 1024, 1024, 2, sink, None, None) == -1  # misaligned
    assert fn(FAKE, 4, 1024, 1000, 2, sink, None, None) == -1            # stride < vocab
    assert fn(FAKE, 4, 1024, 1024, 3, sink, None, None) == -1            # element size
