"""Measurement aids of libtrajfloor.  The read-only floor of the logit pass reads each logit row's
bytes exactly once with the pass's launch plan: the XOR of the per-wave words it writes equals the
XOR of every 32-bit word of the rows' first `vocab` elements (a word read twice or skipped breaks
the equality).  Shapes cover every launch plan, rows that are a single partial sweep, ragged last
sweeps, row slices and a row stride larger than the vocabulary.  The sustained-MFMA-rate kernel
executes the products the benchmark counts (all-ones operands make every lane's result exact)
and rejects arguments it cannot use."""
import ctypes
import os

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FLOOR_LIB = os.path.join(ROOT, "paper_2608_27514_amd", "libtrajfloor.so")

pytestmark = pytest.mark.gpu


def _floor_lib():
    if not os.path.exists(FLOOR_LIB):
        raise RuntimeError("libtrajfloor.so is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(FLOOR_LIB)
    fn = lib.traj_floor_logit_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p]
    return fn


# rows, vocab, row stride, element bytes; every case keeps rows x slices x waves <= 4096 so that
# each wave owns one sink word
CASES = [
    (1, 126464, 126464, 2),     # one row: eight row slices of eight waves
    (37, 1000, 1000, 2),        # few rows, each a single partial sweep
    (37, 1000, 1024, 2),        # the same with a padded row stride
    (200, 126488, 126488, 2),   # 128..511 rows: eight waves per row, ragged last sweep
    (1000, 4104, 4104, 2),      # 512..4095 rows: four waves per row, one full and one partial sweep
    (64, 2052, 2052, 4),        # fp32 rows
    (4096, 264, 272, 2),        # one wave per row, a single partial sweep, padded stride
]


@pytest.mark.parametrize("rows,vocab,stride,eb", CASES)
def test_floor_reads_every_word_once(rows, vocab, stride, eb):
    fn = _floor_lib()
    dev = torch.device("cuda")
    g = torch.Generator(device="cpu").manual_seed(rows * 7919 + vocab)
    words_per_row = stride * eb // 4
    host = torch.randint(-(2 ** 31), 2 ** 31 - 1, (rows, words_per_row), generator=g, dtype=torch.int64)
    host = host.to(torch.int32)
    data = host.to(dev)
    sink = torch.zeros(4096, dtype=torch.int32, device=dev)
    shape = (ctypes.c_int32 * 4)()
    stream = torch.cuda.current_stream()
    rc = fn(ctypes.c_void_p(data.data_ptr()), rows, vocab, stride, eb, ctypes.c_void_p(sink.data_ptr()), shape,
            ctypes.c_void_p(stream.cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    threads, _, _, splits = list(shape)
    assert rows * splits * (threads // 64) <= 4096
    want = np.bitwise_xor.reduce(host[:, : vocab * eb // 4].numpy().astype(np.uint32).ravel())
    got = np.bitwise_xor.reduce(sink.cpu().numpy().astype(np.uint32))
    assert int(got) == int(want)


def _rate_fn():
    if not os.path.exists(FLOOR_LIB):
        raise RuntimeError("libtrajfloor.so is not built (run __graft_entry__.build())")
    fn = ctypes.CDLL(FLOOR_LIB).traj_floor_mfma_rate
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    return fn


@pytest.mark.parametrize("grid,iters", [(1, 1), (8, 3), (512, 5)])
def test_mfma_rate_kernel_executes_the_counted_products(grid, iters):
    """The sustained-MFMA-rate kernel performs the work the benchmark divides by: with every operand
    1.0, each of a wave's 4 accumulators gains 16 per element per MFMA and takes 4 MFMAs per round,
    so lane 0 of every wave reports 4 x 16 x (4 x 16 x iters) (exact in fp32 at these sizes), and
    the clock words are written."""
    fn = _rate_fn()
    dev = torch.device("cuda")
    ones = torch.ones(4096, dtype=torch.bfloat16, device=dev)
    sink = torch.full((4096,), -1.0, dtype=torch.float32, device=dev)
    clock = torch.zeros(2, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    rc = fn(ctypes.c_void_p(ones.data_ptr()), ones.numel() * 2, ctypes.c_void_p(ones.data_ptr()), ones.numel() * 2,
            grid, iters, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(clock.data_ptr()),
            ctypes.c_void_p(stream.cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    waves = grid * 4
    got = sink.cpu().numpy()
    assert np.all(got[:waves] == 4 * 16 * (4 * 16 * iters))
    assert np.all(got[waves:] == -1.0)
    cyc, ticks = clock.cpu().tolist()
    assert cyc > 0 and ticks > 0


def test_mfma_rate_kernel_rejects_bad_arguments():
    fn = _rate_fn()
    dev = torch.device("cuda")
    x = torch.ones(64, dtype=torch.bfloat16, device=dev)
    sink = torch.zeros(4096, dtype=torch.float32, device=dev)
    clock = torch.zeros(2, dtype=torch.int64, device=dev)
    p = lambda t, off=0: ctypes.c_void_p(t.data_ptr() + off)  # noqa: E731
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert fn(p(x), 128, p(x), 128, 0, 1, p(sink), p(clock), s) == -1      # empty grid
    assert fn(p(x), 128, p(x), 128, 1, 0, p(sink), p(clock), s) == -1      # no rounds
    assert fn(p(x), 8, p(x), 128, 1, 1, p(sink), p(clock), s) == -1        # fewer than 16 operand bytes
    assert fn(p(x, 2), 64, p(x), 128, 1, 1, p(sink), p(clock), s) == -1    # misaligned operands
    assert fn(None, 128, p(x), 128, 1, 1, p(sink), p(clock), s) == -1
