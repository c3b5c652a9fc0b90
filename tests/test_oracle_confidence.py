"""Pins for the confidence / top-k oracle (CPU only)."""

import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from synthetic import WORKLOADS, decode_inputs, make_logits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_rows():
    with open(os.path.join(GOLDEN, "confidence_rows.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        conf, idx = oracle.confidence_topk(np.array([case["logits"]]), case["k"])
        if "conf" in case:
            expect = case["conf"]
        else:
            expect = [eval(e, {"exp": math.exp}) for e in case["conf_expr"]]  # noqa: S307 (fixture)
        np.testing.assert_allclose(conf[0], expect, rtol=1e-14, atol=1e-15, err_msg=case["name"])
        assert idx[0].tolist() == case["idx"], case["name"]


def _topk_by_scan(row, k):
    """Brute force: repeatedly take the largest remaining value, the lowest
    index among equals, with a plain Python scan."""
    taken = []
    for _ in range(k):
        best = None
        for v in range(len(row)):
            if v in taken:
                continue
            if best is None or row[v] > row[best]:
                best = v
        taken.append(best)
    return taken


def test_indices_match_scan_on_rows_with_many_ties():
    rng = np.random.default_rng(7)
    rows = rng.integers(0, 6, size=(64, 40)).astype(np.float64) * 0.5
    for k in (1, 3, 8):
        _, idx = oracle.confidence_topk(rows, k)
        for r in range(rows.shape[0]):
            assert idx[r].tolist() == _topk_by_scan(rows[r].tolist(), k)


def test_confidence_equals_library_softmax():
    rng = np.random.default_rng(8)
    rows = rng.standard_normal((16, 300)) * 3
    conf, idx = oracle.confidence_topk(rows, 5)
    sm = scipy.special.softmax(rows, axis=1)
    np.testing.assert_allclose(conf, np.take_along_axis(sm, idx, axis=1), rtol=1e-12)
    np.testing.assert_allclose(conf[:, 0], sm.max(axis=1), rtol=1e-12)


def test_full_k_probabilities_sum_to_one():
    rng = np.random.default_rng(9)
    rows = rng.standard_normal((8, 12))
    conf, idx = oracle.confidence_topk(rows, 12)
    np.testing.assert_allclose(conf.sum(axis=1), 1.0, rtol=1e-14)
    for r in range(8):
        assert sorted(idx[r].tolist()) == list(range(12))
    assert np.all(np.diff(conf, axis=1) <= 0)


def test_uniform_row():
    conf, idx = oracle.confidence_topk(np.zeros((3, 1000)), 3)
    np.testing.assert_allclose(conf, 1e-3, rtol=1e-13)
    assert idx.tolist() == [[0, 1, 2]] * 3


def test_lse_construction_gives_sigmoid_of_margin():
    """The generator's 'lse' rows put probability sigmoid(m) on the planted
    token before rounding; bf16 rounding of a logit near 12 moves it by at most
    1/32, so the confidence stays within ~1e-2 of sigmoid(m)."""
    wl = WORKLOADS[2].with_(B=1, N=2, V=8192, parents=(-1, -1))
    d = decode_inputs(wl, 123)
    lg = make_logits(d["row_margin"], d["row_top"], wl.V, torch.bfloat16, 5)
    conf, idx = oracle.confidence_topk(lg.float().numpy(), 3)
    sig = 1.0 / (1.0 + np.exp(-d["row_margin"]))
    assert np.max(np.abs(conf[:, 0] - sig)) < 1e-2
    assert np.array_equal(idx, d["row_top"])
    # the same rows in fp32 are within fp32 rounding of sigmoid(m)
    lg32 = make_logits(d["row_margin"], d["row_top"], wl.V, torch.float32, 5)
    conf32, idx32 = oracle.confidence_topk(lg32.numpy(), 3)
    assert np.max(np.abs(conf32[:, 0] - sig)) < 1e-5
    assert np.array_equal(idx32, d["row_top"])


def test_signed_zero_is_a_tie():
    conf, idx = oracle.confidence_topk(np.array([[-0.0, 0.0, -0.0]]), 3)
    assert idx[0].tolist() == [0, 1, 2]
    np.testing.assert_allclose(conf[0], 1 / 3)


def test_bad_arguments():
    with pytest.raises(ValueError):
        oracle.confidence_topk(np.zeros((2, 3)), 4)
    with pytest.raises(ValueError):
        oracle.confidence_topk(np.zeros((2, 3)), 0)
    with pytest.raises(ValueError):
        oracle.confidence_topk(np.zeros(3), 1)
