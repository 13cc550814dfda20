"""Host-side parts of bench.py: the CPU oracle leg on reduced inputs of each
workload kind (reduce, quantize + reduce, split-phase share, top-k, bucketed
top-k, DSAR node step), and the refusal of more than one GPU."""
import os
import subprocess
import sys
import types

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1802_08021_amd import inputs  # noqa: E402


def workload(cfg, scale_log2, share=False, bucketed=None):
    c = inputs.config(cfg, scale_log2=scale_log2)
    d = inputs.generate(c, 0, workers=1)
    w = types.SimpleNamespace(c=c, d_host=d, seed=0, rng={}, bucketed=bucketed)
    if c.kind == "topk":
        w.nnz = c.P * c.k
        return w
    if share:
        lo, hi = 0, c.N // c.P
        keep = [a < hi for a in d["idx"]]
        w.d_host = {"idx": [a[m] for a, m in zip(d["idx"], keep)], "val": [v[m] for v, m in zip(d["val"], keep)]}
        w.rng = {"lo": lo, "hi": hi}
    w.nnz = sum(a.size for a in w.d_host["idx"])
    return w


@pytest.mark.parametrize("cfg,scale_log2,kw", [
    (1, 0, {}), (2, 4, {}), (3, 8, {}), (3, 8, {"bucketed": (512, 4)}), (4, 8, {}), (5, 9, {}),
    (5, 9, {"share": True})])
def test_oracle_leg_runs(cfg, scale_log2, kw):
    leg = bench.oracle_leg(workload(cfg, scale_log2, **kw), 3)
    assert leg["threads"] == 3 and leg["kind"] == "oracle"
    for key in ("ms_per_step", "single_thread_ms_per_step", "input_nnz_per_s"):
        assert np.isfinite(leg[key]) and leg[key] > 0, key
    assert leg["sample"]


def test_oracle_leg_dsar():
    c = inputs.config(5, scale_log2=10)
    w = bench.DsarWorkload.__new__(bench.DsarWorkload)
    w.c, w.d_host, w.seed, w.bits, w.bucket = c, inputs.generate(c, 0, workers=1), 0, 4, 64
    w.bounds = [s * (c.N // c.P) for s in range(c.P)] + [c.N]
    w.nnz = 1
    leg = bench.oracle_leg(w, 2)
    assert leg["ms_per_step"] > 0 and "stand-ins" in leg["sample"]


def test_oracle_threads_respects_omp(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "1")
    assert bench.oracle_threads() == 1
    monkeypatch.setenv("OMP_NUM_THREADS", "")
    assert bench.oracle_threads() >= 1


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
