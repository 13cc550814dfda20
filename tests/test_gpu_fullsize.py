"""Parity at the full workload sizes, in the launch configuration the
benchmark times: bench.Workload builds the same arena-resident inputs and
prepared calls, one step runs the whole path, and its outputs are compared
with the oracle on the same seeded inputs.

  c3  P=32, N=2^24 dense rows: top-k (k = N/1000) of every rank, then the
      sparse reduce of the selected streams;
  c4  P=64, N=2^26, Zipf-overlapping supports: reduce to a dense root;
  c5  P=128, N=2^27: 4-bit QSGD of every rank (codes and scales), then the
      reduce of the dequantized streams to a dense root.

Bar: indices, nnz, per-node union sizes and switch decisions, codes and
scales bit-exact; values within 1e-6 rel / 1e-7 abs and bitwise."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, assert_values, say, to_np, torch_dev

pytestmark = pytest.mark.gpu


def _workload(cfg, seed=0):
    import bench
    torch, dev = torch_dev()
    c = inputs.config(cfg)
    say(f"[full] {c.name}: P={c.P} N={c.N} generating inputs and device buffers")
    return c, bench.Workload(c.name, c, seed, torch, dev, keep_host=cfg == 5), torch


def _gpu_result(call, torch):
    """The reduce outputs of one timed step -- the call the benchmark times,
    sparcml_sparse_reduce_async, with its device result header -- plus
    per-node union sizes and decisions from the synchronous entry point on
    the same prepared inputs (whose root must agree)."""
    from paper_1802_08021_amd import sparcml as S
    call.run_async()
    nnz, dense = call.result_header()
    torch.cuda.synchronize()
    out_idx = None if dense else to_np(call.out_idx, np.uint32)[:nnz].copy()
    out_val = to_np(call.out_val).copy() if dense else to_np(call.out_val)[:nnz].copy()
    idx, vals, codes, scales = call._keep
    node = S.ReduceCall(idx, call.N, call.delta, vals=vals, codes=codes, scales=scales,
                        qbits=0 if codes is None else call.arr[0].qbits, node_info=True)
    n2, d2 = node.run()
    torch.cuda.synchronize()
    assert (n2, d2) == (nnz, dense)
    out = {
        "dense": dense,
        "nnz": nnz,
        "idx": out_idx,
        "val": out_val,
        "node_nnz": to_np(node.node_nnz).astype(np.uint64),
        "node_dense": to_np(node.node_dense),
    }
    del node
    return out


@pytest.mark.timeout(900)
def test_c5_full_quantize_and_reduce():
    c, w, torch = _workload(5)
    w.quant.run()
    torch.cuda.synchronize()
    g = _gpu_result(w.reduce, torch)
    say(f"[full] c5: GPU root nnz={g['nnz']} dense={g['dense']}")
    d = w.d_host
    say("[full] c5: oracle quantize")
    q, scale, deq = oracle.quantize(d["val"], c.qbits, inputs.quant_seed(0, c.cfg))
    codes, gscale = w.quant._keep[1], to_np(w.quant.scale)
    np.testing.assert_array_equal(gscale.view(np.uint32), scale.view(np.uint32), err_msg="scales")
    for r in range(c.P):
        np.testing.assert_array_equal(to_np(codes[r]), q[r], err_msg=f"codes of rank {r}")
    say("[full] c5: codes and scales equal; oracle reduce")
    o = oracle.sparse_reduce(d["idx"], deq, c.N, c.delta)
    assert_reduce_equal(g, o, "c5 full")
    assert g["dense"]


@pytest.mark.timeout(600)
def test_c4_full_reduce():
    c, w, torch = _workload(4)
    g = _gpu_result(w.reduce, torch)
    say(f"[full] c4: GPU root nnz={g['nnz']} dense={g['dense']}; regenerating host inputs")
    d = inputs.generate(c, 0)
    o = oracle.sparse_reduce(d["idx"], d["val"], c.N, c.delta)
    assert_reduce_equal(g, o, "c4 full")
    assert g["dense"]
    assert (~g["node_dense"].astype(bool)).any()  # the lower levels stayed sparse


@pytest.mark.timeout(600)
def test_c3_full_topk_and_reduce():
    c, w, torch = _workload(3)
    w.topk.run()
    torch.cuda.synchronize()
    gi = to_np(w.topk.idx, np.uint32)
    gv = to_np(w.topk.val)
    g = _gpu_result(w.reduce, torch)
    say(f"[full] c3: GPU root nnz={g['nnz']} dense={g['dense']}; oracle top-k")
    x = inputs.generate(c, 0)["x"]
    oi, ov = oracle.topk_by_threshold(x, c.k)
    np.testing.assert_array_equal(gi, oi, err_msg="top-k indices")
    assert_values(gv.ravel(), ov.ravel(), "top-k values")
    say("[full] c3: top-k equal; oracle reduce")
    o = oracle.sparse_reduce([oi[r] for r in range(c.P)], [ov[r] for r in range(c.P)], c.N, c.delta)
    assert_reduce_equal(g, o, "c3 full")
    assert not g["dense"]


@pytest.mark.timeout(900)
def test_c3_bucketed_full_step():
    """c3's rows as gradients with Alg. 1's error feedback and 4 of every 512
    coordinates selected (the c3/bucketed benchmark step): selections, values
    and the updated error of every row, then the reduce, against the oracle."""
    import bench
    torch, dev = torch_dev()
    c = inputs.config(3)
    say(f"[full] c3/bucketed: P={c.P} N={c.N}")
    w = bench.Workload("c3/bucketed", c, 0, torch, dev, bucketed=(512, 4))
    w.topk.run()
    torch.cuda.synchronize()
    gi = to_np(w.topk.idx, np.uint32)[:, : w.topk.K]
    gv = to_np(w.topk.val)[:, : w.topk.K]
    ge = to_np(w.topk.eps)
    g = _gpu_result(w.reduce, torch)
    say("[full] c3/bucketed: oracle (zero error, alpha 0.1)")
    x = inputs.generate(c, 0)["x"]
    oi, ov, oe = oracle.topk_bucketed(np.zeros_like(x), x, 0.1, 512, 4)
    np.testing.assert_array_equal(gi, oi, err_msg="selected indices")
    assert_values(gv.ravel(), ov.ravel(), "selected values")
    assert_values(ge.ravel(), oe.ravel(), "updated error")
    del x, oe, ge
    o = oracle.sparse_reduce([oi[r] for r in range(c.P)], [ov[r] for r in range(c.P)], c.N, c.delta)
    assert_reduce_equal(g, o, "c3/bucketed full")


@pytest.mark.timeout(900)
def test_c4_with_48_ranks_full_reduce():
    """c4 with a rank count that is not a power of two (App. A's step in
    front), at full size."""
    import dataclasses
    import bench
    torch, dev = torch_dev()
    c = dataclasses.replace(inputs.config(4), P=48)
    say(f"[full] c4/p48: P={c.P} N={c.N}")
    w = bench.Workload("c4/p48", c, 0, torch, dev)
    g = _gpu_result(w.reduce, torch)
    d = inputs.generate(c, 0)
    o = oracle.sparse_reduce(d["idx"], d["val"], c.N, c.delta)
    assert_reduce_equal(g, o, "c4/p48 full")


@pytest.mark.timeout(1200)
def test_c5_dsar_full_step_all_shares():
    """One DSAR node step at c5's size (the c5/dsar benchmark step): the
    gathered, decoded vector of 2^27 coordinates compared, share by share,
    with the oracle's pipeline (range reduce of the share, bucketed QSGD,
    decode) for all 128 shares of App. A's partition; the node's own share
    (0) is computed by the timed step itself."""
    import bench
    torch, dev = torch_dev()
    c = inputs.config(5)
    say(f"[full] c5/dsar: P={c.P} N={c.N} preparing the other nodes' shares")
    w = bench.DsarWorkload("c5/dsar", c, 0, torch, dev)
    w.step()
    torch.cuda.synchronize()
    got = to_np(w.concat.out_val)
    d = inputs.generate(c, 0)
    b = w.bounds
    assert b[1] - b[0] == c.N // c.P and b[-1] == c.N
    for sh in range(c.P):
        lo, hi = b[sh], b[sh + 1]
        if sh % 16 == 0:
            say(f"[full] c5/dsar: oracle shares {sh}..{min(sh + 15, c.P - 1)}")
        cut = [np.searchsorted(a, (lo, hi)) for a in d["idx"]]
        o = oracle.sparse_reduce_range([a[x:y] for a, (x, y) in zip(d["idx"], cut)],
                                       [v[x:y] for v, (x, y) in zip(d["val"], cut)], c.N, lo, hi, c.delta)
        assert o["dense"]
        q, sc, deq = oracle.quantize([o["val"]], w.bits, inputs.quant_seed(0, c.cfg) + sh, bucket=w.bucket)
        assert_values(got[lo:hi], deq[0], f"share {sh}")
