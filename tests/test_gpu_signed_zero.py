"""Signed zeros through the C ABI, compared with the oracle bitwise.

A stream value may be -0.0.  The oracle's sparse sums keep the sign of zero
as fp32 addition gives it (-0 + -0 = -0, -0 + +0 = +0, a lone -0 stays
-0), and its dense nodes start from +0.0, so a dense value is never -0.0.
These cases put -0.0 (and +0.0) at indices held by one, two, three and
more ranks, into sparse roots, dense roots, a range, tiles that take the
slow pass, the concatenation (sparse and dense results) and top-k rows
whose zeros of both signs tie for the last selected places."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, assert_values, gpu_reduce, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu

NZ = np.float32(-0.0)


def zero_streams(rng, P, N, k, frac_neg_zero=0.5, frac_pos_zero=0.1, hot=()):
    """Uniform streams whose values are -0.0 (frac_neg_zero), +0.0
    (frac_pos_zero) or N(0,1); every rank also holds the indices in ``hot``
    (shared by all ranks) with -0.0 values."""
    idx, val = [], []
    for _ in range(P):
        a = inputs.uniform_subset(rng, N, k)
        a = np.union1d(a, np.asarray(hot, dtype=np.uint32)).astype(np.uint32)
        v = inputs.normal(rng, a.size)
        u = rng.random(a.size)
        v[u < frac_neg_zero] = NZ
        v[(u >= frac_neg_zero) & (u < frac_neg_zero + frac_pos_zero)] = np.float32(0.0)
        v[np.isin(a, np.asarray(hot, dtype=np.uint32))] = NZ
        idx.append(a)
        val.append(v)
    return idx, val


def check(idx, val, N, delta, label, rng_=None):
    say(f"[-0] {label}: P={len(idx)} N={N} delta={delta} nnz={sum(a.size for a in idx)}")
    if rng_ is None:
        o = oracle.sparse_reduce(idx, val, N, delta)
    else:
        o = oracle.sparse_reduce_range(idx, val, N, rng_[0], rng_[1], delta)
    g = gpu_reduce(idx, val, N, delta, rng=rng_)
    assert_reduce_equal(g, o, label)
    return g, o


@pytest.mark.parametrize("P", [2, 3, 4, 8, 16, 64, 128])
def test_reduce_sparse_and_dense_roots(P):
    rng = np.random.default_rng(900 + P)
    N = 50021
    hot = [0, 7, 4095, 4096, 12345, N - 1]  # held by every rank
    idx, val = zero_streams(rng, P, N, max(8, 6000 // P), hot=hot)
    g, o = check(idx, val, N, 50.0, f"P={P} sparse root")
    assert not g["dense"]
    assert np.signbit(o["val"]).any()  # the case does exercise -0.0 in the output
    g, o = check(idx, val, N, 1e-7, f"P={P} dense root")
    assert g["dense"]
    # a dense level over sparse ones
    check(idx, val, N, 0.25 * sum(a.size for a in idx) / N, f"P={P} mixed levels")


def test_reduce_counts_of_ranks_per_index():
    """-0.0 at indices held by exactly 1, 2, 3, 4, 5, 6 and 9 ranks of 16
    (the paths for two, three or four, five and more ranks)."""
    P, N = 16, 12000  # indices up to 279 * 37
    sets = [set() for _ in range(P)]
    vals = [dict() for _ in range(P)]
    j = 0
    for m in (1, 2, 3, 4, 5, 6, 9):
        for rep in range(40):
            ranks = np.random.default_rng(j).choice(P, size=m, replace=False)
            for t, r in enumerate(ranks):
                sets[r].add(j)
                # all -0, or one +0 among -0 (the sum is then +0)
                vals[r][j] = np.float32(0.0) if (rep % 3 == 1 and t == 0) else NZ
            j += 37
    idx = [np.array(sorted(s), np.uint32) for s in sets]
    val = [np.array([vals[r][i] for i in idx[r]], np.float32) for r in range(P)]
    g, o = check(idx, val, N, 100.0, "ranks per index, sparse")
    assert not g["dense"]
    check(idx, val, N, 1e-9, "ranks per index, dense")


def test_reduce_range_and_slow_tiles():
    rng = np.random.default_rng(910)
    N = 200003
    lo, hi = 70001, 170003
    P = 256
    # dense per-rank streams in a narrow window overflow the fast pass
    idx, val = [], []
    for r in range(P):
        a = np.arange(lo + 100, lo + 100 + 3000, dtype=np.uint32)
        v = inputs.normal(rng, a.size)
        v[rng.random(a.size) < 0.6] = NZ
        idx.append(a)
        val.append(v)
    check(idx, val, N, 50.0, "overfull tiles, sparse root", rng_=(lo, hi))
    check(idx, val, N, 1e-6, "overfull tiles, dense root", rng_=(lo, hi))
    idx, val = zero_streams(rng, 32, hi - lo, 3000)
    idx = [(a.astype(np.uint64) + lo).astype(np.uint32) for a in idx]
    check(idx, val, N, 0.5, "range, sparse root", rng_=(lo, hi))
    check(idx, val, N, 1e-5, "range, dense root", rng_=(lo, hi))


def test_concat_keeps_negative_zero():
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(920)
    N, P = 100003, 6
    b = S.split_bounds(P, N)
    hp, dp = [], []
    for s in range(P):
        lo, hi = b[s], b[s + 1]
        if s == 2:  # a dense part with -0.0 values
            v = inputs.normal(rng, hi - lo)
            v[::3] = NZ
            hp.append({"idx": None, "val": v})
            dp.append({"idx": None, "val": to_dev(v)})
            continue
        a = (inputs.uniform_subset(rng, hi - lo, 2000).astype(np.uint64) + lo).astype(np.uint32)
        v = inputs.normal(rng, a.size)
        v[::2] = NZ
        hp.append({"idx": a, "val": v})
        dp.append({"idx": to_dev(a), "val": to_dev(v)})
    say("[-0] concat, dense result")
    o = oracle.concat(hp, b, N, 0.5)
    g = S.concat(dp, b, N, 0.5)
    torch.cuda.synchronize()
    assert g["dense"] and o["dense"]
    assert_values(to_np(g["val"]), o["val"], "dense concat")
    assert np.signbit(o["val"]).any()
    # all sparse: the parts' entries in order, -0.0 kept
    hs = [h for s, h in enumerate(hp) if s != 2]
    ds = [d for s, d in enumerate(dp) if s != 2]
    b2 = b[:2] + b[3:]  # part 1's range also covers part 2's
    for thr_delta, want_dense in ((0.5, False), (1e-6, True)):
        say(f"[-0] concat, sparse parts, delta={thr_delta}")
        o = oracle.concat(hs, b2, N, thr_delta)
        g = S.concat(ds, b2, N, thr_delta)
        torch.cuda.synchronize()
        assert g["dense"] == o["dense"] == want_dense
        assert g["nnz"] == o["nnz"]
        if not want_dense:
            np.testing.assert_array_equal(to_np(g["idx"], np.uint32), o["idx"])
        assert_values(to_np(g["val"]), o["val"], f"sparse parts, delta={thr_delta}")


@pytest.mark.parametrize("residual", [None, "copy", "inplace"])
def test_topk_signed_zero_ties(residual):
    """Rows with few nonzeros and many zeros of both signs, k above the
    nonzero count: the zeros tie (the key ignores the sign) and are taken
    lowest index first, with their signs; the residual gets +0.0 at every
    selected position."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(930)
    for P, N, nz, k in ((3, 5000, 40, 300), (2, 70001, 1000, 9000), (4, 4096, 0, 17)):
        x = np.zeros((P, N), np.float32)
        x[:, rng.random((P, N))[0] < 0.5] = NZ
        for r in range(P):
            pos = rng.choice(N, size=nz, replace=False)
            x[r, pos] = inputs.normal(rng, nz)
        say(f"[-0] topk P={P} N={N} nonzeros={nz} k={k} residual={residual}")
        oi, ov, orr = oracle.topk(x, k, residual=residual is not None)
        tx = to_dev(x)
        res = torch.empty_like(tx) if residual == "copy" else ("inplace" if residual == "inplace" else None)
        gi, gv = S.topk_sparsify(tx, k, residual=res)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_np(gi, np.uint32), oi)
        np.testing.assert_array_equal(to_np(gv).view(np.uint32), ov.view(np.uint32))
        assert np.signbit(ov).any()
        if residual is not None:
            gr = to_np(res) if residual == "copy" else to_np(tx)
            np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32))
