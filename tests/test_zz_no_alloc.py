"""The allocation-free reduce entry point (sparcml_sparse_reduce_async_noalloc)
against sparcml_sparse_reduce_async, through the C ABI, on the same prepared
inputs: root header, per-node union sizes and decisions, indices exactly,
values within 1e-6 rel / 1e-7 abs and bitwise.  Two calls in a row share the
library's one scratch array; the second has a smaller input (fewer ranks,
fewer indices, a sparse root after a dense one), so stale contents of the
first would show.  A reduce larger than the array is refused on the host."""
import ctypes

import numpy as np
import pytest

from paper_1802_08021_amd import inputs
from gpu_util import assert_values, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def _prepared(P, N, k, delta, seed, qbits=0):
    from paper_1802_08021_amd import sparcml as S
    rng = np.random.default_rng(seed)
    idx = [to_dev(inputs.uniform_subset(rng, N, k)) for _ in range(P)]
    vals = [to_dev(inputs.laplace(rng, 1e-3, k)) for _ in range(P)]
    if qbits:
        codes, scales, _ = S.quantize(vals, qbits, seed)
        mk = lambda: S.ReduceCall(idx, N, delta, codes=codes, scales=scales, qbits=qbits, node_info=True)
    else:
        mk = lambda: S.ReduceCall(idx, N, delta, vals=vals, node_info=True)
    return mk(), mk()


def _outputs(call):
    nnz, dense = call.result_header()
    return {
        "nnz": nnz, "dense": dense,
        "idx": None if dense else to_np(call.out_idx, np.uint32)[:nnz].copy(),
        "val": to_np(call.out_val).copy() if dense else to_np(call.out_val)[:nnz].copy(),
        "node_nnz": to_np(call.node_nnz).copy(), "node_dense": to_np(call.node_dense).copy(),
    }


def _compare(a, b, label):
    assert (a["nnz"], a["dense"]) == (b["nnz"], b["dense"]), label
    np.testing.assert_array_equal(a["node_nnz"], b["node_nnz"], err_msg=f"{label} node nnz")
    np.testing.assert_array_equal(a["node_dense"], b["node_dense"], err_msg=f"{label} node decisions")
    if not a["dense"]:
        np.testing.assert_array_equal(a["idx"], b["idx"], err_msg=f"{label} indices")
    assert_values(a["val"], b["val"], f"{label} values")


def test_noalloc_matches_workspace_entry_point_twice():
    torch, dev = torch_dev()
    cases = [  # second call smaller: fewer ranks and indices, sparse root
        ("dense root, 64 ranks, 4-bit", dict(P=64, N=1 << 22, k=(1 << 22) // 100, delta=0.1, seed=71, qbits=4)),
        ("sparse root, 16 ranks", dict(P=16, N=1 << 18, k=700, delta=0.25, seed=72)),
    ]
    for label, kw in cases:
        say(f"[noalloc] {label}: {kw}")
        ref, new = _prepared(**kw)
        ref.run_async()
        torch.cuda.synchronize()
        a = _outputs(ref)
        new.run_async_noalloc()
        torch.cuda.synchronize()
        b = _outputs(new)
        _compare(b, a, label)
        if label.startswith("dense"):
            assert b["dense"]
        else:
            assert not b["dense"]


def test_noalloc_rejects_sizes_beyond_its_scratch():
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    limit = 16 << 20
    # what the header promises fits
    for P, N in ((256, 2**32 - 1), (33, 2**32 - 1), (2, 2**31), (32, 2**31), (256, 2**31)):
        assert S.workspace_size(S.OP_REDUCE, P, N, 1, 0.1) <= limit, (P, N)
    # 32 ranks over the whole 32-bit index space need more
    assert S.workspace_size(S.OP_REDUCE, 32, 2**32 - 1, 1, 0.1) > limit
    P, N = 32, 2**32 - 1
    arr = (S.Stream * P)()
    one = to_dev(np.array([5], np.uint32))
    v = to_dev(np.array([1.0], np.float32))
    for r in range(P):
        arr[r] = S.Stream(S._ptr(one), S._ptr(v), None, None, 1, 0, 0)
    out_val = torch.empty(16, dtype=torch.float32, device=dev)
    out = S.Stream(S._ptr(one), S._ptr(out_val), None, None, 1 << 20, 0, 0)
    res = torch.zeros(2, dtype=torch.int64, device=dev)
    rc = S.lib().sparcml_sparse_reduce_async_noalloc(P, arr, N, 0, N, 0.1, ctypes.byref(out), None, None,
                                                     S._ptr(res), S._stream_ptr(dev))
    assert rc == S.EWORKSPACE
    assert "allocation-free" in S.last_error()
