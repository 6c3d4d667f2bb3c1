"""CPU tests of the benchmark's host-side arithmetic: the algorithmic byte counts the roofline
divides by, the K/V tokens a step reads (for sizing the input rotation), the sum over
decoding rounds of the per-round trace, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2510_09883_amd import configs  # noqa: E402


def test_full_layer_bytes_by_hand():
    w = configs.get(3)
    lens = [32768] * 16
    kv = 16 * 32768 * 4 * 8 * 128          # K and V, bf16, 8 KV heads, d = 128
    qo = 4 * 32 * 128 * 16                 # q in, o out, bf16
    pt = 16 * 4 * 2048                     # one int32 page-table entry per page
    assert bench.full_layer_bytes(w, lens) == kv + qo + pt == 2147483648 + 262144 + 131072


def test_sparse_layer_bytes_counts_partial_units():
    w = configs.get(1)                      # 2 KV heads, d = 64, budget 8 pages
    w.batch = 2
    lens = [100, 1024]
    # sequence 0: units 0..6 (6 full pages + 4 tokens of page 6); sequence 1: 8 full pages
    idx = np.array([[0, 1, 2, 3, 4, 5, 6, -1], [0, 3, 9, 20, 40, 61, 62, 63]])
    cnt = np.array([7, 8])
    toks = 100 + 8 * 16
    want = 4 * 2 * 64 * toks + 4 * 8 * 64 * 2 + 4 * 8 * 2
    assert bench.sparse_layer_bytes(w, lens, idx, cnt) == want


def test_step_tokens():
    w = configs.get(2)                      # F F D S*13 D S*15, budget 2048 tokens
    # before the context exceeds the budget every layer reads everything
    assert bench.step_tokens(w, w.roles, 1000) == 32 * 1000
    # after: 4 dense layers read s, 28 sparse layers read the budget
    assert bench.step_tokens(w, w.roles, 8192) == 4 * 8192 + 28 * 2048
    # sparse layers before the first Delta layer run full
    roles = [configs.ROLE_SPARSE, configs.ROLE_DELTA, configs.ROLE_SPARSE]
    assert bench.step_tokens(w, roles, 8192) == 2 * 8192 + 2048


def test_trapezoid_rounds():
    # constant per-round time: S rounds of t us
    assert bench.trapezoid_rounds([(1, 5.0), (101, 5.0)]) == pytest.approx(101 * 5e-6)
    # linear growth t(c) = c us sampled at its ends: sum over c = 1..S of c is S(S+1)/2
    S = 1000
    got = bench.trapezoid_rounds([(1, 1.0), (S, float(S))])
    assert got == pytest.approx(S * (S + 1) / 2 * 1e-6, rel=1e-3)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_cpu_baseline_reports_cores_and_per_role_times():
    from paper_2510_09883_amd import synth
    w = configs.get(1)
    inp = synth.make_inputs(w, "cpu", poison_tail=False)
    r = bench.cpu_baseline(w, inp, w.roles, 0.5)
    assert r["kind"] == "oracle" and r["unit"] == "us/step" and r["value"] > 0
    assert r["cores"] >= 1 and r["host_cpus"] >= 1
    assert set(r["seconds_per_sequence_layer"]) == {"full", "delta", "sparse"}
