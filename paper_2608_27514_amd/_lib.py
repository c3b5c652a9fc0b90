"""ctypes binding of libtrajspec (include/traj_spec.h).

Argument marshalling only: every step of the verification path runs in the HIP
kernels of the library.  PyTorch supplies device memory and the current stream.
If the library is not built the calls raise -- there is no fallback.
"""

import ctypes
import os

import torch

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "libtrajspec.so")

TRAJ_OK = 0
STATUS_NAMES = {0: "TRAJ_OK", 1: "TRAJ_E_NULL", 2: "TRAJ_E_SHAPE", 3: "TRAJ_E_DTYPE",
                4: "TRAJ_E_UNSUPPORTED", 5: "TRAJ_E_WORKSPACE", 6: "TRAJ_E_HIP", 7: "TRAJ_E_ARG"}
TRAJ_BF16, TRAJ_F32 = 0, 1
MODES = {"exact": 0, "top1": 1, "topk": 2}
TRAVERSALS = {"greedy": 0, "longest": 1}
DEV_BAD_PARENT = 0x1
DEV_BAD_LEAF = 0x2
DEV_BAD_BLOCK = 0x4
DEV_BAD_ROOT = 0x8


class TrajSpecError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = _lib().traj_status_string(status).decode()
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({msg})")


class AttnShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("L", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32), ("S", ctypes.c_int32), ("scale", ctypes.c_float)]


class LogitsShape(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("vocab", ctypes.c_int64), ("row_stride", ctypes.c_int64),
                ("dtype", ctypes.c_int32)]


class Drafts(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("L", ctypes.c_int32), ("k", ctypes.c_int32),
                ("tokens", ctypes.c_void_p), ("parent", ctypes.c_void_p), ("committed", ctypes.c_void_p),
                ("conf0", ctypes.c_void_p), ("idx0", ctypes.c_void_p), ("mode", ctypes.c_int32),
                ("traversal", ctypes.c_int32)]


class Accepted(ctypes.Structure):
    _fields_ = [("leaf", ctypes.c_void_p), ("on_path", ctypes.c_void_p), ("n_accepted", ctypes.c_void_p),
                ("out_tokens", ctypes.c_void_p), ("hi", ctypes.c_void_p)]


class TreeShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("L", ctypes.c_int32), ("k", ctypes.c_int32), ("n_prev", ctypes.c_int32),
                ("width", ctypes.c_int32), ("depth", ctypes.c_int32), ("branch", ctypes.c_int32),
                ("full", ctypes.c_int32), ("n_max", ctypes.c_int32), ("branch_deep", ctypes.c_int32)]


class LayerDims(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float)]


class RefreshShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("S", ctypes.c_int32), ("L", ctypes.c_int32), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32), ("scale", ctypes.c_float)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")]


_LIB = None

EXPORTS = {
    "traj_verify_attn_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(AttnShape)]),
    "traj_verify_attn": (ctypes.c_int32, [ctypes.c_void_p] * 7 + [ctypes.POINTER(AttnShape), ctypes.c_void_p,
                                                                   ctypes.c_size_t, ctypes.c_void_p]),
    "traj_confidence_topk_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(LogitsShape), ctypes.c_int32]),
    "traj_confidence_topk": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.POINTER(LogitsShape), ctypes.c_void_p, ctypes.c_size_t,
                                              ctypes.c_void_p]),
    "traj_confidence_topk_noalloc": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                                      ctypes.c_void_p, ctypes.POINTER(LogitsShape), ctypes.c_void_p]),
    "traj_accept": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Drafts), ctypes.c_float,
                                     ctypes.POINTER(Accepted), ctypes.c_void_p]),
    "traj_verify_attn_peers": (ctypes.c_int32, [ctypes.c_void_p] * 8 + [ctypes.POINTER(AttnShape), ctypes.c_void_p,
                                                                         ctypes.c_size_t, ctypes.c_void_p]),
    "traj_joint_peers": (ctypes.c_int32, [ctypes.c_int32] * 3 + [ctypes.c_void_p] * 4),
    "traj_interblock_trigger": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                                 ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                                 ctypes.c_void_p, ctypes.c_void_p]),
    "traj_tree_max_nodes": (ctypes.c_int32, [ctypes.POINTER(TreeShape)]),
    "traj_verify_layer_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(AttnShape), ctypes.POINTER(LayerDims)]),
    "traj_refresh_layer_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(RefreshShape), ctypes.POINTER(LayerDims)]),
    "traj_refresh_layer": (ctypes.c_int32, [ctypes.c_void_p, ctypes.POINTER(LayerWeights), ctypes.POINTER(LayerDims),
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.POINTER(RefreshShape), ctypes.c_void_p, ctypes.c_size_t,
                                            ctypes.c_void_p]),
    "traj_verify_layer": (ctypes.c_int32, [ctypes.c_void_p, ctypes.POINTER(LayerWeights), ctypes.POINTER(LayerDims),
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.POINTER(AttnShape), ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_void_p]),
    "traj_linear_workspace_size": (ctypes.c_size_t, [ctypes.c_int64] * 3),
    "traj_linear": (ctypes.c_int32, [ctypes.c_void_p] * 3 + [ctypes.c_int64] * 3 +
                    [ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "traj_build_tree": (ctypes.c_int32, [ctypes.c_void_p] * 6 + [ctypes.POINTER(TreeShape), ctypes.c_float]
                        + [ctypes.c_void_p] * 7),
    "traj_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "traj_version": (ctypes.c_char_p, []),
    "traj_get_device_status": (ctypes.c_int32, [ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_void_p]),
}


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_27514_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def load():
    """Load the library (raises if it is missing) and return its ctypes handle."""
    return _lib()


def version():
    return _lib().traj_version().decode()


def built_digest():
    """Source digest the loaded library was built from (stamped into traj_version())."""
    return version().rsplit(" ", 1)[-1]


def check_build():
    """Raise unless the loaded library was built from the sources checked out next to it."""
    from .build import source_digest
    want = source_digest()
    got = built_digest()
    if got != want:
        raise RuntimeError(f"{LIB_PATH} was built from other sources (digest {got[:16]}, sources {want[:16]}); "
                           "rebuild with `python -m paper_2608_27514_amd.build`")
    return got


def _check(status, where):
    if status != TRAJ_OK:
        raise TrajSpecError(status, where)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, name, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr() if t is not None and t.numel() > 0 else 0)


# ---------------------------------------------------------------- attention

def attn_shape(q, k_cache, scale=0.0):
    B, N, L, Hq, D = q.shape
    S, Hkv = k_cache.shape[1], k_cache.shape[2]
    return AttnShape(B, N, L, Hq, Hkv, D, S, float(scale))


def verify_attn_workspace_size(shape):
    return int(_lib().traj_verify_attn_workspace_size(ctypes.byref(shape)))


def verify_attn(q, k_cache, v_cache, k_draft, v_draft, draft_parent, out=None, scale=0.0, workspace=None,
                stream=None, peers=None):
    """Trajectory-masked attention; returns ``out`` [B,N,L,Hq,D] bf16.  ``peers`` ([B,N]
    int64 holding uint64 bit masks) adds visible drafts per draft (traj_verify_attn_peers)."""
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("k_draft", k_draft),
                    ("v_draft", v_draft)):
        _dev(t, name, torch.bfloat16)
    _dev(draft_parent, "draft_parent", torch.int32)
    if peers is not None:
        _dev(peers, "peers", torch.int64)
        if tuple(peers.shape) != tuple(draft_parent.shape):
            raise ValueError("peers must be [B,N] like draft_parent")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", torch.bfloat16)
    shape = attn_shape(q, k_cache, scale)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if peers is None:
        st = _lib().traj_verify_attn(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_draft), _ptr(v_draft),
                                     _ptr(draft_parent), _ptr(out), ctypes.byref(shape), _ptr(workspace),
                                     ws_bytes, _stream(stream))
        _check(st, "traj_verify_attn")
    else:
        st = _lib().traj_verify_attn_peers(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_draft), _ptr(v_draft),
                                           _ptr(draft_parent), _ptr(peers), _ptr(out), ctypes.byref(shape),
                                           _ptr(workspace), ws_bytes, _stream(stream))
        _check(st, "traj_verify_attn_peers")
    return out


def joint_peers(B, n_cur, n_next, root_cur=None, root_next=None, out=None, device=None, stream=None):
    """Peer masks of a joint packing (traj_joint_peers): drafts [0, n_cur) hold block t's
    tree, [n_cur, n_cur + n_next) block t+1's; root_cur / root_next are [B] int32 device
    tensors (None = root 0).  Returns a [B, n_cur + n_next] int64 device tensor holding the
    uint64 bit masks traj_verify_attn_peers takes."""
    for name, t in (("root_cur", root_cur), ("root_next", root_next)):
        if t is not None:
            _dev(t, name, torch.int32)
            if t.numel() != B:
                raise ValueError(f"{name} must hold B entries")
    if out is None:
        dev = device or (root_cur.device if root_cur is not None else
                         root_next.device if root_next is not None else torch.device("cuda"))
        out = torch.empty((B, n_cur + n_next), dtype=torch.int64, device=dev)
    _dev(out, "out", torch.int64)
    _check(_lib().traj_joint_peers(B, n_cur, n_next, _ptr(root_cur), _ptr(root_next), _ptr(out), _stream(stream)),
           "traj_joint_peers")
    return out


def interblock_trigger(state, conf, threshold, out=None, stream=None):
    """Inter-block trigger per sequence from state [B,2L] int32 and conf [B,2L,k] (or
    [B*2L,k]) float32; returns dict trigger [B] uint8, c_cur [B], c_next [B] float32."""
    B, L2 = state.shape
    if L2 % 2:
        raise ValueError("state must hold two blocks (2L positions) per sequence")
    k = conf.numel() // (B * L2)
    if conf.numel() != B * L2 * k:
        raise ValueError("conf must hold B*2L*k entries")
    _dev(state, "state", torch.int32)
    _dev(conf, "conf", torch.float32)
    dev = state.device
    if out is None:
        out = {"trigger": torch.empty(B, dtype=torch.uint8, device=dev),
               "c_cur": torch.empty(B, dtype=torch.float32, device=dev),
               "c_next": torch.empty(B, dtype=torch.float32, device=dev)}
    st = _lib().traj_interblock_trigger(_ptr(state), _ptr(conf), B, L2 // 2, k, float(threshold),
                                        _ptr(out["trigger"]), _ptr(out.get("c_cur")), _ptr(out.get("c_next")),
                                        _stream(stream))
    _check(st, "traj_interblock_trigger")
    return out


# ---------------------------------------------------------------- confidence / top-k

def logits_shape(logits):
    rows, vocab = logits.shape
    dt = {torch.bfloat16: TRAJ_BF16, torch.float32: TRAJ_F32}.get(logits.dtype)
    if dt is None:
        raise TypeError("logits must be bfloat16 or float32")
    return LogitsShape(rows, vocab, logits.stride(0), dt)


def confidence_topk_workspace_size(logits, k):
    return int(_lib().traj_confidence_topk_workspace_size(ctypes.byref(logits_shape(logits)), int(k)))


def confidence_topk(logits, k, conf=None, idx=None, workspace=None, stream=None):
    """Returns (conf [R,k] float32, idx [R,k] int32).  ``logits`` [R,V] may have a row
    stride larger than V (its last dimension must be contiguous)."""
    if not isinstance(logits, torch.Tensor) or not logits.is_cuda:
        raise TypeError("logits must be a CUDA (HIP) tensor")
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be 2-D with a contiguous last dimension")
    shape = logits_shape(logits)
    R = logits.shape[0]
    if conf is None:
        conf = torch.empty((R, k), dtype=torch.float32, device=logits.device)
    if idx is None:
        idx = torch.empty((R, k), dtype=torch.int32, device=logits.device)
    _dev(conf, "conf", torch.float32)
    _dev(idx, "idx", torch.int32)
    if workspace is None:
        need = int(_lib().traj_confidence_topk_workspace_size(ctypes.byref(shape), int(k)))
        if need > 0:
            workspace = torch.empty(need, dtype=torch.uint8, device=logits.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib().traj_confidence_topk(ctypes.c_void_p(logits.data_ptr()), int(k), _ptr(conf), _ptr(idx),
                                     ctypes.byref(shape), _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "traj_confidence_topk")
    return conf, idx


def confidence_topk_noalloc(logits, k, conf=None, idx=None, stream=None):
    """traj_confidence_topk_noalloc: the same results as :func:`confidence_topk` without a
    workspace (the library's fixed per-device scratch holds the split records)."""
    if not isinstance(logits, torch.Tensor) or not logits.is_cuda:
        raise TypeError("logits must be a CUDA (HIP) tensor")
    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be 2-D with a contiguous last dimension")
    shape = logits_shape(logits)
    R = logits.shape[0]
    if conf is None:
        conf = torch.empty((R, k), dtype=torch.float32, device=logits.device)
    if idx is None:
        idx = torch.empty((R, k), dtype=torch.int32, device=logits.device)
    _dev(conf, "conf", torch.float32)
    _dev(idx, "idx", torch.int32)
    st = _lib().traj_confidence_topk_noalloc(ctypes.c_void_p(logits.data_ptr()), int(k), _ptr(conf), _ptr(idx),
                                             ctypes.byref(shape), _stream(stream))
    _check(st, "traj_confidence_topk_noalloc")
    return conf, idx


# ---------------------------------------------------------------- acceptance

def accept(conf, idx, tokens, parent, committed, conf0, idx0, threshold, mode="exact", traversal="greedy",
           out=None, stream=None):
    """Acceptance; returns a dict of device tensors (leaf, on_path, n_accepted,
    out_tokens, hi).  conf/idx may be [B*N*L, k] or [B,N,L,k]."""
    B, N, L = tokens.shape
    k = conf0.shape[-1]
    if conf.numel() != B * N * L * k or idx.numel() != B * N * L * k:
        raise ValueError("conf/idx must hold B*N*L*k entries")
    for name, t, dt in (("conf", conf, torch.float32), ("idx", idx, torch.int32), ("tokens", tokens, torch.int32),
                        ("parent", parent, torch.int32), ("committed", committed, torch.int32),
                        ("conf0", conf0, torch.float32), ("idx0", idx0, torch.int32)):
        _dev(t, name, dt)
    dev = tokens.device
    if out is None:
        out = {
            "leaf": torch.empty(B, dtype=torch.int32, device=dev),
            "on_path": torch.empty((B, N), dtype=torch.uint8, device=dev),
            "n_accepted": torch.empty(B, dtype=torch.int32, device=dev),
            "out_tokens": torch.empty((B, L), dtype=torch.int32, device=dev),
            "hi": torch.empty((B, N, L), dtype=torch.uint8, device=dev),
        }
    dr = Drafts(B, N, L, k, tokens.data_ptr(), parent.data_ptr(), committed.data_ptr(), conf0.data_ptr(),
                idx0.data_ptr(), MODES[mode], TRAVERSALS[traversal])
    ac = Accepted(out["leaf"].data_ptr(), out["on_path"].data_ptr(), out["n_accepted"].data_ptr(),
                  out["out_tokens"].data_ptr(), out["hi"].data_ptr())
    st = _lib().traj_accept(_ptr(conf), _ptr(idx), ctypes.byref(dr), float(threshold), ctypes.byref(ac),
                            _stream(stream))
    _check(st, "traj_accept")
    return out


# ---------------------------------------------------------------- tree construction
def tree_shape(B, L, k, width, depth, branch, full=False, n_prev=0, n_max=None, branch_deep=1):
    sh = TreeShape(B, L, k, n_prev, width, depth, branch, 1 if full else 0, 0, branch_deep)
    if n_max is None:
        n_max = int(_lib().traj_tree_max_nodes(ctypes.byref(sh)))
        if n_max < 0:
            raise ValueError("invalid tree shape")
    sh.n_max = n_max
    return sh


def tree_max_nodes(B, L, k, width, depth, branch, full=False, branch_deep=1):
    return int(_lib().traj_tree_max_nodes(ctypes.byref(tree_shape(B, L, k, width, depth, branch, full, n_max=0,
                                                                  branch_deep=branch_deep))))


def build_tree(state, conf0, idx0, threshold, width, depth, branch, full=False, leaf=None, conf=None, idx=None,
               n_max=None, out=None, stream=None, branch_deep=1):
    """Next step's draft tree (Alg. 1) from the accepted state; returns a dict of device
    tensors tokens [B,n_max,L], parent [B,n_max], n_nodes [B], score [B,n_max],
    conf_next / idx_next [B,L,k].  With ``leaf`` (traj_accept's leaf) the candidates come
    from conf/idx [B,N,L,k] (or [B*N*L,k]) of the verified tree, else from conf0/idx0."""
    B, L = state.shape
    k = conf0.shape[-1]
    for name, t, dt in (("state", state, torch.int32), ("conf0", conf0, torch.float32), ("idx0", idx0, torch.int32)):
        _dev(t, name, dt)
    n_prev = 0
    if leaf is not None:
        _dev(leaf, "leaf", torch.int32)
        _dev(conf, "conf", torch.float32)
        _dev(idx, "idx", torch.int32)
        n_prev = conf.numel() // (B * L * k)
        if conf.numel() != B * n_prev * L * k or idx.numel() != conf.numel():
            raise ValueError("conf/idx must hold B*N*L*k entries")
    sh = tree_shape(B, L, k, width, depth, branch, full, n_prev, n_max, branch_deep)
    dev = state.device
    if out is None:
        out = {
            "tokens": torch.empty((B, sh.n_max, L), dtype=torch.int32, device=dev),
            "parent": torch.empty((B, sh.n_max), dtype=torch.int32, device=dev),
            "n_nodes": torch.empty(B, dtype=torch.int32, device=dev),
            "score": torch.empty((B, sh.n_max), dtype=torch.float32, device=dev),
            "conf_next": torch.empty((B, L, k), dtype=torch.float32, device=dev),
            "idx_next": torch.empty((B, L, k), dtype=torch.int32, device=dev),
        }
    st = _lib().traj_build_tree(_ptr(state), _ptr(leaf), _ptr(conf), _ptr(idx), _ptr(conf0), _ptr(idx0),
                                ctypes.byref(sh), float(threshold), _ptr(out["tokens"]), _ptr(out["parent"]),
                                _ptr(out["n_nodes"]), _ptr(out.get("score")), _ptr(out.get("conf_next")),
                                _ptr(out.get("idx_next")), _stream(stream))
    _check(st, "traj_build_tree")
    return out


# ---------------------------------------------------------------- verification layer
LAYER_WEIGHTS = ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")


def layer_workspace_size(B, N, L, Hq, Hkv, D, S, hidden, inter, rms_eps=1e-5, rope_theta=500000.0):
    sh = AttnShape(B, N, L, Hq, Hkv, D, S, 0.0)
    return int(_lib().traj_verify_layer_workspace_size(ctypes.byref(sh),
                                                       ctypes.byref(LayerDims(hidden, inter, rms_eps, rope_theta))))


def _expect_shape(t, name, shape):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def verify_layer(x, weights, k_cache, v_cache, draft_parent, Hq, pos0=None, inter=None, rms_eps=1e-5,
                 rope_theta=500000.0, scale=0.0, workspace=None, stream=None):
    """One verification decoder layer over the packed draft tokens; updates x [B,N,L,hidden]
    (bf16) in place and returns it.  ``weights`` maps LAYER_WEIGHTS names to bf16 tensors."""
    B, N, L, hidden = x.shape
    D = hidden // Hq
    S, Hkv = k_cache.shape[1], k_cache.shape[2]
    if inter is None:
        inter = weights["w_down"].shape[0]
    _dev(x, "x", torch.bfloat16)
    for n in LAYER_WEIGHTS:
        _dev(weights[n], n, torch.bfloat16)
    for n, shape in (("attn_norm", (hidden,)), ("w_qkv", (hidden, (Hq + 2 * Hkv) * D)), ("w_o", (Hq * D, hidden)),
                     ("mlp_norm", (hidden,)), ("w_gate_up", (hidden, 2 * inter)), ("w_down", (inter, hidden))):
        _expect_shape(weights[n], n, shape)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, n, torch.bfloat16)
        _expect_shape(t, n, (B, S, Hkv, D))
    _dev(draft_parent, "draft_parent", torch.int32)
    _expect_shape(draft_parent, "draft_parent", (B, N))
    if pos0 is not None:
        _dev(pos0, "pos0", torch.int32)
        _expect_shape(pos0, "pos0", (B,))
    sh = AttnShape(B, N, L, Hq, Hkv, D, S, float(scale))
    dims = LayerDims(hidden, inter, rms_eps, rope_theta)
    need = int(_lib().traj_verify_layer_workspace_size(ctypes.byref(sh), ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    lw = LayerWeights(*[weights[n].data_ptr() for n in LAYER_WEIGHTS])
    st = _lib().traj_verify_layer(_ptr(x), ctypes.byref(lw), ctypes.byref(dims), _ptr(k_cache), _ptr(v_cache),
                                  _ptr(draft_parent), _ptr(pos0), ctypes.byref(sh), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "traj_verify_layer")
    return x


def refresh_layer_workspace_size(B, S, L, Hq, Hkv, D, hidden, inter, rms_eps=1e-5, rope_theta=500000.0):
    sh = RefreshShape(B, S, L, Hq, Hkv, D, 0.0)
    return int(_lib().traj_refresh_layer_workspace_size(ctypes.byref(sh),
                                                        ctypes.byref(LayerDims(hidden, inter, rms_eps, rope_theta))))


def refresh_layer(x, weights, block_start, Hq, Hkv, L, k_cache=None, v_cache=None, inter=None, rms_eps=1e-5,
                  rope_theta=500000.0, scale=0.0, workspace=None, stream=None):
    """Dual-cache refresh: one decoder layer over whole sequences x [B, S + L, hidden] (bf16,
    updated in place) with bidirectional attention; the rotated K and the V of every position
    outside each sequence's block [block_start[b], block_start[b] + L) go to k_cache / v_cache
    [B, S, Hkv, D] (allocated when None).  Returns (x, k_cache, v_cache)."""
    B, T, hidden = x.shape
    S = T - L
    D = hidden // Hq
    if inter is None:
        inter = weights["w_down"].shape[0]
    _dev(x, "x", torch.bfloat16)
    for n in LAYER_WEIGHTS:
        _dev(weights[n], n, torch.bfloat16)
    for n, shape in (("attn_norm", (hidden,)), ("w_qkv", (hidden, (Hq + 2 * Hkv) * D)), ("w_o", (Hq * D, hidden)),
                     ("mlp_norm", (hidden,)), ("w_gate_up", (hidden, 2 * inter)), ("w_down", (inter, hidden))):
        _expect_shape(weights[n], n, shape)
    _dev(block_start, "block_start", torch.int32)
    _expect_shape(block_start, "block_start", (B,))
    if k_cache is None:
        k_cache = torch.empty(B, S, Hkv, D, dtype=torch.bfloat16, device=x.device)
    if v_cache is None:
        v_cache = torch.empty(B, S, Hkv, D, dtype=torch.bfloat16, device=x.device)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _dev(t, n, torch.bfloat16)
        _expect_shape(t, n, (B, S, Hkv, D))
    sh = RefreshShape(B, S, L, Hq, Hkv, D, float(scale))
    dims = LayerDims(hidden, inter, rms_eps, rope_theta)
    need = int(_lib().traj_refresh_layer_workspace_size(ctypes.byref(sh), ctypes.byref(dims)))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=x.device)
    lw = LayerWeights(*[weights[n].data_ptr() for n in LAYER_WEIGHTS])
    st = _lib().traj_refresh_layer(_ptr(x), ctypes.byref(lw), ctypes.byref(dims), _ptr(block_start), _ptr(k_cache),
                                   _ptr(v_cache), ctypes.byref(sh), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "traj_refresh_layer")
    return x, k_cache, v_cache


def linear_workspace_size(M, K, N):
    return int(_lib().traj_linear_workspace_size(M, K, N))


def linear(x, w, y=None, accumulate=False, workspace=None, stream=None):
    """y = x @ w (+ y when accumulate) for bf16 x [..., K] and w [K, N]; returns y [..., N].
    Few-row shapes split K when given a workspace (allocated here when None)."""
    _dev(x, "x", torch.bfloat16)
    _dev(w, "w", torch.bfloat16)
    K, N = w.shape
    if x.shape[-1] != K:
        raise ValueError(f"x has {x.shape[-1]} columns, w has {K} rows")
    M = x.numel() // K
    if y is None:
        if accumulate:
            raise ValueError("accumulate needs y")
        y = torch.empty(x.shape[:-1] + (N,), dtype=torch.bfloat16, device=x.device)
    _dev(y, "y", torch.bfloat16)
    _expect_shape(y, "y", x.shape[:-1] + (N,))
    if workspace is None:
        need = linear_workspace_size(M, K, N)
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device) if need > 0 else None
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib().traj_linear(_ptr(x), _ptr(w), _ptr(y), M, K, N, 1 if accumulate else 0, _ptr(workspace), ws_bytes,
                              _stream(stream)), "traj_linear")
    return y


def device_status(reset=True, stream=None):
    """Synchronises the stream and returns the device status bits (TRAJ_DEV_*)."""
    flags = ctypes.c_int32(0)
    _check(_lib().traj_get_device_status(ctypes.byref(flags), 1 if reset else 0, _stream(stream)),
           "traj_get_device_status")
    return flags.value
