"""CPU checks of bench.py's contract: one GPU only, the workload table at the
configurations' sizes (blocks and attention FLOP per call), and the replay
that counts a fused update's block loads and stores."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stderr


@pytest.mark.parametrize("name,blk,flop", [("tiny-fp32", 32768, 1.887e7), ("wan1.3b-1layer", 4792320, 1.0765e12),
                                           ("wan14b-1layer", 36864000, 1.9110e13)])
def test_workloads_at_the_configured_sizes(name, blk, flop):
    w = bench.WORKLOADS[name]
    elt = 2 if w["dtype"] == "bf16" else 4
    assert w["tokens_per_block"] * w["heads"] * w["head_dim"] * elt == blk
    lq = w["frames"] * w["tokens_per_block"]
    lk = (w["budget"] + w["frames"]) * w["tokens_per_block"]
    assert abs(4.0 * lq * lk * w["head_dim"] * w["heads"] / flop - 1.0) < 1e-3


@pytest.mark.parametrize("js,count0,F,M,anchor,op,expect", [
    ([], 2, 1, 5, True, "sqrt_span", (1, 1)),               # no merge: the frame is copied in
    ([1], 2, 1, 2, True, "sqrt_span", (2, 1)),              # frame merged into the newest old entry
    ([1, 1], 2, 2, 2, True, "sqrt_span", (3, 1)),           # chained: the second merge reuses the result
    ([0], 2, 1, 2, True, "sqrt_span", (1, 1)),              # anchor pair: no bytes, the frame is copied
    ([0], 2, 1, 2, False, "select_nearest", (1, 1)),        # the newer old entry kept: the frame is copied
    ([1, 0], 2, 2, 2, False, "sqrt_span", (4, 2)),          # merge, then its result merged with an old entry; frame 1 kept
])
def test_fused_update_block_count(js, count0, F, M, anchor, op, expect):
    assert bench.fused_block_ios(js, count0, F, M, anchor, op) == expect


def test_measured_traffic_is_tied_to_its_workload():
    assert bench.attn_traffic("wan14b-1layer") is None
    assert bench.measured_traffic(bench.SPEC_TRAFFIC, "spectral.hip", "wan1.3b-1layer") is None
    assert bench.measured_traffic(bench.ATTN_TRAFFIC, "no_such_file.hip", "wan1.3b-1layer") is None


@pytest.mark.parametrize("budget", ["0", "1"])
def test_budget_override_rejects_a_memory_without_an_eligible_pair(budget):
    """`--budget` replaces the workload's M; the library needs M >= 2 (one
    pair besides the newest entry), and bench.py refuses less before any GPU work."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--budget", budget], capture_output=True,
                       text=True, timeout=300, cwd=root)
    assert r.returncode != 0
    assert "--budget must be at least 2" in r.stderr


@pytest.mark.parametrize("js,count0,F,M,anchor,op,expect", [
    ([], 2, 1, 5, True, "sqrt_span", (0, 0)),               # no merge: the staged frame stays in its slot
    ([1], 2, 1, 2, True, "sqrt_span", (2, 1)),              # frame merged: loaded from its staging slot
    ([0], 2, 1, 2, True, "sqrt_span", (0, 0)),              # anchor pair: no bytes, the frame stays
    ([18, 17, 18], 21, 3, 21, True, "sqrt_span", (5, 2)),   # steady state: three merges (one chained), two results kept
])
def test_staged_update_block_count(js, count0, F, M, anchor, op, expect):
    assert bench.fused_block_ios(js, count0, F, M, anchor, op, staged=True) == expect
