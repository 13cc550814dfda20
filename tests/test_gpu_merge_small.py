"""The small-data path (the whole recursive-doubling merge tree in one
workgroup, taken for at most 8 tree slots whose entries, at most thr
together, number at most 16384 / 8192 / 1024 for 2 / 4 / 8 slots) against
the oracle, bitwise: roots, per-node union sizes and decisions.  Cases at
its boundaries (the largest totals it takes and one more entry, which goes
to the tile path), thr = the entry count and one less, 2..8 ranks including
3, 5, 6, 7 (App. A's step in front), empty ranks and an empty input, full
overlap (every rank the same indices), the top of the index space, QSGD
codes of 2/4/8 bits, the range entry point and the asynchronous entry
point."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, gpu_reduce, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def streams_with_total(rng, P, N, total, empty=()):
    """P sorted uniform streams whose sizes sum to ``total``."""
    live = [r for r in range(P) if r not in empty]
    cuts = np.sort(rng.integers(0, total + 1, size=len(live) - 1)) if live else []
    sizes = np.diff(np.concatenate([[0], cuts, [total]])).astype(int) if live else []
    idx = [np.zeros(0, np.uint32) for _ in range(P)]
    val = [np.zeros(0, np.float32) for _ in range(P)]
    for r, k in zip(live, sizes):
        idx[r] = inputs.uniform_subset(rng, N, int(min(k, N)))
        val[r] = inputs.normal(rng, idx[r].size)
    return idx, val


def check(idx, val, N, delta, label, rng_=None):
    say(f"[merge] {label}: P={len(idx)} N={N} delta={delta} nnz={sum(a.size for a in idx)}")
    if rng_ is None:
        o = oracle.sparse_reduce(idx, val, N, delta)
    else:
        o = oracle.sparse_reduce_range(idx, val, N, rng_[0], rng_[1], delta)
    g = gpu_reduce(idx, val, N, delta, rng=rng_)
    assert_reduce_equal(g, o, label)
    return g


LIMIT = {2: 16384, 3: 8192, 4: 8192, 5: 1024, 6: 1024, 7: 1024, 8: 1024}  # per rank count


@pytest.mark.parametrize("P", [2, 3, 4, 5, 6, 7, 8])
def test_rank_counts(P):
    rng = np.random.default_rng(1100 + P)
    N = 1 << 20
    for total in (1, 100, LIMIT[P] // 2 + 7):
        idx, val = streams_with_total(rng, P, N, total, empty=(1,) if P > 3 else ())
        g = check(idx, val, N, 0.5, f"P={P} total={total}")
        assert not g["dense"]


@pytest.mark.parametrize("P", [2, 4, 8])
def test_capacity_boundary(P):
    rng = np.random.default_rng(1200 + P)
    N = 1 << 18
    for total in (LIMIT[P] - 1, LIMIT[P], LIMIT[P] + 1):
        idx, val = streams_with_total(rng, P, N, total)
        check(idx, val, N, 1.0, f"P={P} total={total}")


def test_threshold_boundary():
    """thr equal to the entry count (all sparse, merge path) and one below
    it (the tile path, whose decisions may switch a node to dense)."""
    rng = np.random.default_rng(1300)
    N = 100000
    idx, val = streams_with_total(rng, 4, N, 5000)
    tot = sum(a.size for a in idx)
    assert oracle.threshold(N, (tot + 0.5) / N) == tot and oracle.threshold(N, (tot - 0.5) / N) == tot - 1
    check(idx, val, N, (tot + 0.5) / N, "thr = entries")
    check(idx, val, N, (tot - 0.5) / N, "thr = entries - 1")


def test_empty_and_overlap_and_top_index():
    rng = np.random.default_rng(1400)
    N = 5000
    check([np.zeros(0, np.uint32)] * 4, [np.zeros(0, np.float32)] * 4, N, 0.5, "all empty")
    a = inputs.uniform_subset(rng, N, 900)
    idx = [a.copy() for _ in range(4)]
    val = [inputs.normal(rng, a.size) for _ in range(4)]
    check(idx, val, N, 16.0, "every rank the same indices")
    b = a[:120]
    check([b.copy() for _ in range(8)], [inputs.normal(rng, b.size) for _ in range(8)], N, 16.0,
          "eight ranks, the same indices")
    N = 2**32 - 1  # indices up to 2^32 - 2, in the range [N - 5000, N)
    top = [np.array([N - 5000, N - 4000, N - 2, N - 1], np.uint32), np.array([N - 4000, N - 1], np.uint32),
           np.array([N - 3], np.uint32)]
    check(top, [inputs.normal(rng, t.size) for t in top], N, 0.5, "top of the index space",
          rng_=(N - 5000, N))


def test_range_entry_point():
    rng = np.random.default_rng(1500)
    N, lo, hi = 1 << 22, 1000003, 2000003
    idx, val = streams_with_total(rng, 4, hi - lo, 8000)
    idx = [(a.astype(np.uint64) + lo).astype(np.uint32) for a in idx]
    check(idx, val, N, 0.5, "range", rng_=(lo, hi))


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantized_codes(bits):
    rng = np.random.default_rng(1600 + bits)
    P, N = 4, 300000
    idx, val = streams_with_total(rng, P, N, 8000, empty=(2,))
    val = [inputs.laplace(rng, 1e-3, a.size) for a in idx]
    q, scale, deq = oracle.quantize(val, bits, seed=321 + bits)
    say(f"[merge] QSGD {bits}-bit")
    o = oracle.sparse_reduce(idx, deq, N, 0.5)
    codes = [to_dev(c if c.size else np.zeros(1, np.uint8)) for c in q]
    g = gpu_reduce(idx, None, N, 0.5, qbits=bits, codes=codes, scales=to_dev(scale))
    assert_reduce_equal(g, o, f"q{bits}")


def test_async_entry_point_and_repeat():
    """The asynchronous entry point (header on the device), run twice on
    the same buffers: the same bits both times."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(1700)
    N = 1 << 20
    idx, val = streams_with_total(rng, 4, N, 8192)
    o = oracle.sparse_reduce(idx, val, N, 0.25)
    call = S.ReduceCall([to_dev(a) for a in idx], N, 0.25, vals=[to_dev(v) for v in val], node_info=True)
    for rep in range(2):
        say(f"[merge] async, call {rep}")
        call.run_async()
        nnz, dense = call.result_header()
        assert (nnz, dense) == (o["nnz"], False)
        np.testing.assert_array_equal(to_np(call.out_idx, np.uint32)[:nnz], o["idx"])
        np.testing.assert_array_equal(to_np(call.out_val)[:nnz].view(np.uint32), o["val"].view(np.uint32))
        np.testing.assert_array_equal(to_np(call.node_nnz).astype(np.uint64), o["node_nnz"])
        assert not to_np(call.node_dense).any()
