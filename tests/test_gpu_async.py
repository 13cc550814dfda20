"""The asynchronous reduce (sparcml_sparse_reduce_async) through the C ABI:
the same outputs as the synchronous call and the oracle, with the root
header written on the device, for dense and sparse roots, a dense guess
ending in a sparse root, ranges, P = 1 and non-power-of-two P; and the call
captured in a HIP graph, replayed several times with eager work and
synchronizations between replays, every replay checked."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, assert_values, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def async_reduce(idx, val, N, delta, rng=None):
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    ti = [to_dev(a) for a in idx]
    tv = [to_dev(v) for v in val]
    kw = {} if rng is None else {"lo": rng[0], "hi": rng[1]}
    c = S.ReduceCall(ti, N, delta, vals=tv, node_info=True, **kw)
    c.run_async()
    torch.cuda.synchronize()
    nnz, dense = c.result_header()
    P = len(idx)
    return c, {
        "dense": dense, "nnz": nnz,
        "idx": None if dense else to_np(c.out_idx[:nnz], np.uint32).copy(),
        "val": to_np(c.out_val if dense else c.out_val[:nnz]).copy(),
        "node_nnz": to_np(c.node_nnz).astype(np.uint64) if P > 1 else np.zeros(0, np.uint64),
        "node_dense": to_np(c.node_dense) if P > 1 else np.zeros(0, np.uint8),
    }


def check(idx, val, N, delta, label, rng=None):
    say(f"[async] {label}: P={len(idx)} N={N} delta={delta} range={rng}")
    o = oracle.sparse_reduce(idx, val, N, delta) if rng is None else \
        oracle.sparse_reduce_range(idx, val, N, rng[0], rng[1], delta)
    c, g = async_reduce(idx, val, N, delta, rng)
    assert_reduce_equal(g, o, label)
    return c, g, o


def streams(rng, P, N, k, lo=0):
    idx = [(inputs.uniform_subset(rng, N - lo, k).astype(np.uint64) + lo).astype(np.uint32) for _ in range(P)]
    return idx, [inputs.normal(rng, a.size) for a in idx]


def test_async_matches_oracle():
    rng = np.random.default_rng(800)
    idx, val = streams(rng, 32, 300007, 4000)
    check(idx, val, 300007, 0.05, "dense root")
    check(idx, val, 300007, 2.0, "sparse root")
    base = inputs.uniform_subset(rng, 100000, 1000)
    check([base] * 16, [inputs.normal(rng, 1000) for _ in range(16)], 100000, 0.03, "dense guess, sparse root")
    idx, val = streams(rng, 24, 400000, 3000, lo=100000)
    check(idx, val, 400000, 0.05, "range, P = 24", rng=(100000, 400000))
    idx, val = streams(rng, 1, 50000, 3000)
    check(idx, val, 50000, 0.5, "P = 1 sparse")
    check(idx, val, 50000, 0.01, "P = 1 dense")


def test_async_in_a_graph_replayed():
    """Captured once, replayed four times on changing inputs with eager work
    and synchronizations between replays; every replay against the
    oracle."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(801)
    P, N, k = 16, 200003, 3000
    idx, _ = streams(rng, P, N, k)
    ti = [to_dev(a) for a in idx]
    tv = [torch.zeros(a.size, dtype=torch.float32, device=dev) for a in idx]
    for delta in (0.05, 3.0):  # dense root, sparse root
        c = S.ReduceCall(ti, N, delta, vals=tv, node_info=True)
        for t, v in zip(tv, [inputs.normal(rng, a.size) for a in idx]):
            t.copy_(torch.from_numpy(v))
        c.run_async()  # eager warm-up
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                c.run_async()
        torch.cuda.synchronize()
        for rep in range(4):
            vals = [inputs.normal(rng, a.size) for a in idx]
            for t, v in zip(tv, vals):
                t.copy_(torch.from_numpy(v))
            _ = torch.ones(1000, device=dev).sum().item()  # eager work between replays
            say(f"[async] graph delta={delta} replay {rep}")
            g.replay()
            torch.cuda.synchronize()
            o = oracle.sparse_reduce(idx, vals, N, delta)
            nnz, dense = c.result_header()
            assert dense == o["dense"] and nnz == o["nnz"], (rep, nnz, o["nnz"])
            if dense:
                assert_values(to_np(c.out_val), o["val"], f"replay {rep}")
            else:
                np.testing.assert_array_equal(to_np(c.out_idx[:nnz], np.uint32), o["idx"])
                assert_values(to_np(c.out_val[:nnz]), o["val"], f"replay {rep}")
            np.testing.assert_array_equal(to_np(c.node_nnz).astype(np.uint64), o["node_nnz"].astype(np.uint64))
        del g
