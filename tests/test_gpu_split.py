"""Parity of the split-phase share (sparse reduce over an index range,
§5.3.2) through the C ABI with the CPU oracle, at the bar of the full
reduce: representation, nnz, indices, node decisions and union sizes
bit-exact; values within 1e-6 rel / 1e-7 abs and bitwise.  Ranges start at
unaligned offsets (tiles begin at lo), end in a ragged tail, reach the top of
the 32-bit index space, and cover the slow path, QSGD inputs and P = 1."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, assert_values, gpu_reduce, say, to_dev, torch_dev

pytestmark = pytest.mark.gpu


def check_range(idx, val, N, lo, hi, delta, label):
    say(f"[split] {label}: P={len(idx)} N={N} [{lo}, {hi}) delta={delta} "
        f"nnz={sum(a.size for a in idx)}")
    o = oracle.sparse_reduce_range(idx, val, N, lo, hi, delta)
    g = gpu_reduce(idx, val, N, delta, rng=(lo, hi))
    assert_reduce_equal(g, o, label)
    return g, o


def sub_streams(rng, P, lo, hi, kmax):
    idx, val = [], []
    for _ in range(P):
        k = int(rng.integers(0, min(hi - lo, kmax) + 1))
        idx.append((inputs.uniform_subset(rng, hi - lo, k).astype(np.uint64) + lo).astype(np.uint32))
        val.append(inputs.normal(rng, k))
    return idx, val


def restrict(idx, val, lo, hi):
    out_i, out_v = [], []
    for a, v in zip(idx, val):
        m = (a >= lo) & (a < hi)
        out_i.append(a[m].copy())
        out_v.append(v[m].copy())
    return out_i, out_v


def test_random_ranges():
    rng = np.random.default_rng(300)
    for case in range(50):
        P = int(rng.choice([2, 4, 8, 16, 32, 64, 128, 256]))
        N = int(rng.choice([50, 9000, 70001, 1000003]))
        lo = int(rng.integers(0, N))
        hi = int(min(N, lo + rng.choice([1, 33, 4097, 30011, 300007])))
        kmax = int(rng.choice([1, 16, 300, 4000]))
        delta = float(rng.choice([1e-9, 0.01, 0.1, 0.5, 4.0]))
        idx, val = sub_streams(rng, P, lo, hi, kmax)
        check_range(idx, val, N, lo, hi, delta, f"random#{case}")


@pytest.mark.parametrize("cfg,scale", [(2, 0), (4, 4), (5, 5)])
def test_equal_split_shares(cfg, scale):
    """The first, a middle and the last share of an equal P-way split of a
    workload's index space (the last one ragged)."""
    c = inputs.config(cfg, scale_log2=scale)
    d = inputs.generate(c, seed=2)
    P, N = c.P, c.N
    bounds = [N * s // P for s in range(P + 1)]
    for s in sorted({0, P // 2, P - 1}):
        lo, hi = bounds[s], bounds[s + 1]
        idx, val = restrict(d["idx"], d["val"], lo, hi)
        check_range(idx, val, N, lo, hi, c.delta, f"{c.name}/2^{scale} share {s}")


def test_gathered_shares_equal_full_reduce():
    """Property at any size: the shares of an equal split, gathered, give the
    full reduce (values compared with +0.0 == -0.0)."""
    rng = np.random.default_rng(301)
    P, N = 32, 600007
    idx = [inputs.uniform_subset(rng, N, int(rng.integers(1000, 20000))) for _ in range(P)]
    val = [inputs.normal(rng, a.size) for a in idx]
    for delta in (0.02, 0.5):
        full = gpu_reduce(idx, val, N, delta)
        ref = full["val"] if full["dense"] else oracle.densify(full["idx"], full["val"], N)
        got = np.zeros(N, np.float32)
        bounds = [N * s // P for s in range(P + 1)]
        say(f"[split] gathered P={P} N={N} delta={delta}")
        for s in range(P):
            lo, hi = bounds[s], bounds[s + 1]
            si, sv = restrict(idx, val, lo, hi)
            g = gpu_reduce(si, sv, N, delta, rng=(lo, hi))
            if g["dense"]:
                got[lo:hi] = g["val"]
            else:
                assert np.all((g["idx"] >= lo) & (g["idx"] < hi))
                got[g["idx"].astype(np.int64)] = g["val"]
        assert_values(got + np.float32(0), ref + np.float32(0), f"gathered delta={delta}")


def test_range_at_top_of_index_space():
    rng = np.random.default_rng(302)
    N = 2**32 - 1
    for lo, hi, delta in ((N - 200000, N, 0.05), (N - 200000, N, 1.0), (N - 5, N, 0.5),
                          (2**31 - 7000, 2**31 + 9000, 0.2)):
        idx, val = sub_streams(rng, 16, lo, hi, 30000)
        check_range(idx, val, N, lo, hi, delta, f"top [{lo}, {hi})")


def test_range_slow_path_and_full_tiles():
    rng = np.random.default_rng(303)
    P, N = 128, 10**7
    lo, hi = 3333333, 3333333 + 50000
    # every rank clustered in the first 3000 indices of the range
    idx = [(np.sort(rng.choice(3000, 60, replace=False)) + lo).astype(np.uint32) for _ in range(P)]
    val = [inputs.normal(rng, 60) for _ in range(P)]
    check_range(idx, val, N, lo, hi, 0.5, "clustered, sparse")
    check_range(idx, val, N, lo, hi, 1e-6, "clustered, dense")
    # every index of the range in every rank
    idx = [np.arange(lo, lo + 5000, dtype=np.uint32)] * 4
    val = [inputs.normal(rng, 5000) for _ in range(4)]
    check_range(idx, val, N, lo, lo + 5000, 0.5, "k = range, dense")
    check_range(idx, val, N, lo, lo + 5000, 4.0, "k = range, sparse")


def test_range_quantized_inputs():
    rng = np.random.default_rng(304)
    N, lo, hi, P = 400000, 123457, 223457, 32
    torch, dev = torch_dev()
    for bits in (2, 4, 8):
        idx, val = sub_streams(rng, P, lo, hi, 4000)
        q, scale, deq = oracle.quantize(val, bits, seed=40 + bits)
        codes = [to_dev(a if a.size else np.zeros(1, np.uint8)) for a in q]
        scales = to_dev(scale)
        for delta in (0.05, 5.0):
            say(f"[split] quantized bits={bits} delta={delta}")
            o = oracle.sparse_reduce_range(idx, deq, N, lo, hi, delta)
            g = gpu_reduce(idx, None, N, delta, qbits=bits, codes=codes, scales=scales, rng=(lo, hi))
            assert_reduce_equal(g, o, f"range q{bits}")


def test_range_single_rank_and_empty():
    rng = np.random.default_rng(305)
    N, lo, hi = 100000, 4321, 14321
    idx, val = sub_streams(rng, 1, lo, hi, 3000)
    idx[0], val[0] = idx[0][:3000], val[0][:3000]
    check_range(idx, val, N, lo, hi, 0.5, "P=1 sparse")
    check_range(idx, val, N, lo, hi, 1e-4, "P=1 dense")
    e, ev = np.zeros(0, np.uint32), np.zeros(0, np.float32)
    check_range([e] * 8, [ev] * 8, N, lo, hi, 0.5, "all empty")
    check_range([e] * 8, [ev] * 8, N, lo, hi, 1e-9, "all empty thr 0")
