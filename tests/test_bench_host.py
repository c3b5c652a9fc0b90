"""Host side of the benchmark (CPU only): the algorithmic work it divides by, checked against
the oracle's dense trajectory mask, and the one-GPU contract of its command line."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle.attention import trajectory_mask
from synthetic import WORKLOADS, decode_inputs, seed_for

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_attention_flops_count_the_visible_pairs_of_the_mask(cid):
    """4 D flops (QK and PV, a multiply-add each) per visible (query token, key) pair per query
    head: the pairs counted on the oracle's dense mask of the workload's own tree."""
    wl = WORKLOADS[cid]
    parent = decode_inputs(wl, seed_for(cid))["parent"]
    pairs = sum(int(trajectory_mask(parent[b], wl.L, wl.S).sum()) for b in range(wl.B))
    assert bench.attn_flops(wl, parent) == 4 * wl.D * wl.Hq * pairs


def test_attention_flops_of_the_batched_tree_match_the_stated_figure():
    """16 sequences of the 3+9+27+25 tree (sum of draft depths 202 per sequence), 32 heads of
    128, L 32, cache 4096: 2.253 TFLOP per launch."""
    wl = WORKLOADS[5]
    parent = decode_inputs(wl, seed_for(5))["parent"]
    assert all(sum(bench.depths(parent[b])) == 202 for b in range(wl.B))
    assert abs(bench.attn_flops(wl, parent) / 1e12 - 2.253) < 5e-4


def test_bytes_per_launch():
    wl = WORKLOADS[5]
    # K and V cache once, q and out, draft K and V, all bf16
    expect = 2 * (2 * wl.B * wl.S * wl.Hkv * wl.D + 2 * wl.B * wl.N * wl.L * wl.Hq * wl.D
                  + 2 * wl.B * wl.N * wl.L * wl.Hkv * wl.D)
    assert bench.attn_bytes(wl) == expect
    assert bench.logit_bytes(wl) == wl.B * wl.N * wl.L * (wl.V * 2 + wl.k * 8)


def test_depths_follow_the_parent_chain():
    assert bench.depths(np.array([-1, 0, 1, 0, -1, 4])) == [1, 2, 3, 2, 1, 2]


def test_more_than_one_gpu_is_refused_with_a_message():
    env = dict(os.environ, WORLD_SIZE="1")
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, cwd=ROOT, env=env, timeout=300)
    assert res.returncode == 2
    line = [ln for ln in res.stdout.splitlines() if ln.startswith("{")][-1]
    assert "one GPU" in json.loads(line)["error"]
