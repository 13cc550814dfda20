"""The segmented merge path (every tree node sparse, 9..64 tree slots or more
entries than the one-workgroup path takes, at most 2^21 entries: the range
cut into segments of about 2048 expected entries, one workgroup each, output
offsets by look-back) against the oracle, bitwise: roots, per-node union
sizes and decisions.  Cases: c3's shape (32 ranks, 2^24 indices, 0.1%
density: 263 segments), the entry limit (1024 segments) and one past it (the tile
path), segments with no entry, a segment holding far more entries
than a workgroup's LDS (merged piece by piece), heavy overlap, rank counts
that are not powers of two, 64 ranks, QSGD codes, the range and the
asynchronous entry points."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, gpu_reduce, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def uniform_streams(rng, P, N, k, dist="normal"):
    idx, val = [], []
    for _ in range(P):
        a = inputs.uniform_subset(rng, N, k)
        idx.append(a)
        val.append(inputs.normal(rng, a.size) if dist == "normal" else inputs.laplace(rng, 1e-3, a.size))
    return idx, val


def check(idx, val, N, delta, label, rng_=None):
    say(f"[seg] {label}: P={len(idx)} N={N} delta={delta} nnz={sum(a.size for a in idx)}")
    if rng_ is None:
        o = oracle.sparse_reduce(idx, val, N, delta)
    else:
        o = oracle.sparse_reduce_range(idx, val, N, rng_[0], rng_[1], delta)
    g = gpu_reduce(idx, val, N, delta, rng=rng_)
    assert_reduce_equal(g, o, label)
    return g


def test_c3_shape():
    rng = np.random.default_rng(2000)
    N, P = 1 << 24, 32
    idx, val = uniform_streams(rng, P, N, N // 1000, dist="laplace")
    g = check(idx, val, N, 0.25, "c3 shape")
    assert not g["dense"]


@pytest.mark.parametrize("P", [9, 16, 33, 48, 64])
def test_rank_counts(P):
    rng = np.random.default_rng(2100 + P)
    N = 1 << 22
    idx, val = uniform_streams(rng, P, N, 3000)
    idx[3] = np.zeros(0, np.uint32)
    val[3] = np.zeros(0, np.float32)
    check(idx, val, N, 0.5, f"P={P}")


def test_entry_limit_and_many_segments():
    """2^21 entries (1024 segments, the most the path takes) and one more
    (the tile path)."""
    rng = np.random.default_rng(2200)
    N, P = 1 << 26, 32
    idx, val = uniform_streams(rng, P, N, (1 << 21) // P)
    assert sum(a.size for a in idx) == 1 << 21
    check(idx, val, N, 0.5, "2^21 entries")
    extra = np.setdiff1d(np.array([7, 8, 9], np.uint32), idx[0])[:1]
    idx[0] = np.union1d(idx[0], extra).astype(np.uint32)
    val[0] = inputs.normal(rng, idx[0].size)
    check(idx, val, N, 0.5, "2^21 + 1 entries")


def test_overfull_segment_and_empty_segments():
    """All ranks crowd one narrow window (a segment far beyond a workgroup's
    LDS, merged in pieces), a few entries elsewhere, most segments empty."""
    rng = np.random.default_rng(2300)
    N, P = 1 << 24, 32
    idx, val = [], []
    for r in range(P):
        a = np.union1d(np.arange(5000, 5000 + 3000, dtype=np.uint32)[rng.random(3000) < 0.8],
                       inputs.uniform_subset(rng, N, 40)).astype(np.uint32)
        idx.append(a)
        val.append(inputs.normal(rng, a.size))
    g = check(idx, val, N, 0.5, "one overfull segment")
    assert not g["dense"]
    # every rank the same indices, crowded: the pieces sum the heaviest overlap
    a = np.arange(100, 100 + 6000, dtype=np.uint32)
    check([a.copy() for _ in range(P)], [inputs.normal(rng, a.size) for _ in range(P)], N, 0.5,
          "identical crowded streams")


def test_quantized_codes_and_range():
    rng = np.random.default_rng(2400)
    N, P = 1 << 22, 24
    idx, _ = uniform_streams(rng, P, N, 4000)
    val = [inputs.laplace(rng, 1e-3, a.size) for a in idx]
    for bits in (2, 4, 8):
        q, scale, deq = oracle.quantize(val, bits, seed=77 + bits)
        say(f"[seg] QSGD {bits}-bit")
        o = oracle.sparse_reduce(idx, deq, N, 0.5)
        codes = [to_dev(c if c.size else np.zeros(1, np.uint8)) for c in q]
        g = gpu_reduce(idx, None, N, 0.5, qbits=bits, codes=codes, scales=to_dev(scale))
        assert_reduce_equal(g, o, f"q{bits}")
    lo, hi = 1000003, 3000017
    ridx = [a[(a >= lo) & (a < hi)] for a in idx]
    rval = [inputs.normal(rng, a.size) for a in ridx]
    check(ridx, rval, N, 0.5, "range", rng_=(lo, hi))


def test_async_entry_point_repeated():
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(2500)
    N, P = 1 << 24, 32
    idx, val = uniform_streams(rng, P, N, N // 1000)
    o = oracle.sparse_reduce(idx, val, N, 0.25)
    call = S.ReduceCall([to_dev(a) for a in idx], N, 0.25, vals=[to_dev(v) for v in val], node_info=True)
    for rep in range(3):
        say(f"[seg] async, call {rep}")
        call.run_async()
        nnz, dense = call.result_header()
        assert (nnz, dense) == (o["nnz"], False)
        assert int(call.result.cpu()[1]) >> 32 == 0  # no look-back gave up
        np.testing.assert_array_equal(to_np(call.out_idx, np.uint32)[:nnz], o["idx"])
        np.testing.assert_array_equal(to_np(call.out_val)[:nnz].view(np.uint32), o["val"].view(np.uint32))
        np.testing.assert_array_equal(to_np(call.node_nnz).astype(np.uint64), o["node_nnz"])
        assert not to_np(call.node_dense).any()


@pytest.mark.parametrize("P", [16, 37, 64])
def test_one_pass_heavy_overlap(P):
    """Segments of at most two entries a thread take the one-pass order:
    every index held by a random half of the ranks (long runs of slots with
    gaps, the summation stack up to the tree's depth), then by every rank,
    then QSGD codes."""
    rng = np.random.default_rng(2600 + P)
    N = 1 << 16
    cand = inputs.uniform_subset(rng, N, 1000)
    idx = [cand[rng.random(cand.size) < 0.5] for _ in range(P)]
    val = [inputs.normal(rng, a.size) for a in idx]
    g = check(idx, val, N, 1.0, f"random halves, P={P}")
    assert not g["dense"]
    few = cand[::5]
    check([few.copy() for _ in range(P)], [inputs.normal(rng, few.size) for _ in range(P)], N, 1.0,
          f"every rank every index, P={P}")
    q, scale, deq = oracle.quantize([inputs.laplace(rng, 1e-3, a.size) for a in idx], 4, seed=99 + P)
    say(f"[seg] one pass, QSGD 4-bit, P={P}")
    o = oracle.sparse_reduce(idx, deq, N, 1.0)
    codes = [to_dev(c if c.size else np.zeros(1, np.uint8)) for c in q]
    g = gpu_reduce(idx, None, N, 1.0, qbits=4, codes=codes, scales=to_dev(scale))
    assert_reduce_equal(g, o, f"one pass q4 P={P}")
