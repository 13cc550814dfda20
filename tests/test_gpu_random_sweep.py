"""Seeded random sweeps against the oracle.  The sparse reduce: across the
paths the library picks by size (one-workgroup merge tree, segmented merge
tree, tile pipeline with a sparse or a dense root, deferred tiles) and
across what the other tests fix one at a time: rank counts that are not
powers of two, QSGD codes of every width, the range entry point, and index
sets that are uniform, clustered (heavy overlap between ranks) or runs of
consecutive indices; bar as for every reduce parity test -- root
representation, nnz, indices, node decisions and sizes bit-exact, values
bitwise (assert_reduce_equal).  Top-k: row lengths around the kernels'
block sizes, k from 0 to N, rows of ties across signs and of signed zeros,
every residual mode; indices, values and residuals bitwise.  QSGD: up to
139 streams of mixed lengths, every width, with and without dequantized
copies; codes, scales and dequantized values bitwise."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_reduce_equal, gpu_reduce, say, to_dev

pytestmark = pytest.mark.gpu


def _indices(rng, N, k, kind, centers):
    """k distinct ascending indices below N (fewer if N is small)."""
    k = min(k, N)
    if k == 0:
        return np.zeros(0, np.uint32)
    if kind == "uniform":
        return inputs.uniform_subset(rng, N, k)
    if kind == "runs":  # a few runs of consecutive indices
        out = set()
        while len(out) < k:
            s = int(rng.integers(0, N))
            out.update(range(s, min(N, s + int(rng.integers(1, 200)))))
        a = np.array(sorted(out), dtype=np.int64)[:k]
        return np.sort(a).astype(np.uint32)
    # clustered: draws around shared centers, so many ranks hit the same indices
    w = max(1, N // 50)
    c = centers[rng.integers(0, len(centers), size=4 * k)]
    a = np.unique(np.clip(c + rng.integers(-w, w + 1, size=4 * k), 0, N - 1))
    if a.size > k:
        a = np.sort(rng.choice(a, size=k, replace=False))
    return a.astype(np.uint32)


def _case(rng, case):
    P = int(rng.choice([1, 2, 3, 5, 8, 13, 16, 31, 33, 48, 64, 65, 100, 128, 129, 200, 256]))
    N = int(rng.choice([1, 63, 4096, 4097, 50000, 300001]))
    kind = str(rng.choice(["uniform", "clustered", "runs"]))
    kmax = int(rng.choice([1, 16, 300, 3000, 20000]))
    qbits = int(rng.choice([0, 0, 2, 4, 8]))
    delta = float(10.0 ** rng.uniform(-6, 1))
    ranged = N > 64 and rng.random() < 0.3
    centers = rng.integers(0, N, size=int(rng.integers(1, 6)))
    idx = [_indices(rng, N, int(rng.integers(0, kmax + 1)), kind, centers) for _ in range(P)]
    lo, hi = 0, N
    if ranged:
        lo = int(rng.integers(0, N // 2))
        hi = int(rng.integers(lo + 1, N + 1))
        idx = [a[(a >= lo) & (a < hi)] for a in idx]
    val = [inputs.laplace(rng, 1.0, a.size) for a in idx]
    label = (f"sweep#{case}: P={P} N={N} {kind} kmax={kmax} q={qbits} delta={delta:.3g}"
             + (f" range=[{lo},{hi})" if ranged else ""))
    return P, N, idx, val, qbits, delta, (lo, hi) if ranged else None, label


def test_random_sweep():
    rng = np.random.default_rng(20261202)
    for case in range(300):
        P, N, idx, val, qbits, delta, rg, label = _case(rng, case)
        say(f"[sweep] {label} nnz={sum(a.size for a in idx)}")
        if qbits:
            q, scale, deq = oracle.quantize(val, qbits, seed=1000 + case)
            codes = [to_dev(a if a.size else np.zeros(1, np.uint8)) for a in q]
            scales = to_dev(scale)
            vals_o = deq
        else:
            codes = scales = None
            vals_o = val
        if rg is None:
            o = oracle.sparse_reduce(idx, vals_o, N, delta)
        else:
            o = oracle.sparse_reduce_range(idx, vals_o, N, rg[0], rg[1], delta)
        g = gpu_reduce(idx, None if qbits else val, N, delta, qbits=qbits, codes=codes, scales=scales, rng=rg)
        assert_reduce_equal(g, o, label)


def _row_values(rng, N, kind):
    """fp32 values of one row: smooth, heavy-tailed, few distinct magnitudes
    (ties across signs), or mostly zeros (signed)."""
    if kind == "laplace":
        return inputs.laplace(rng, 1e-3, N)
    if kind == "normal":
        return inputs.normal(rng, N)
    if kind == "ties":
        return (rng.choice([-2.0, -0.5, 0.5, 2.0, 0.0, -0.0], size=N)).astype(np.float32)
    x = np.zeros(N, np.float32)
    x[rng.random(N) < 0.5] = np.float32(-0.0)
    m = rng.random(N) < 0.01
    x[m] = inputs.laplace(rng, 1.0, int(m.sum()))
    return x


def test_random_sweep_topk():
    import torch
    from gpu_util import to_np
    from paper_1802_08021_amd import sparcml as S
    rng = np.random.default_rng(7042)
    for case in range(60):
        P = int(rng.integers(1, 6))
        N = int(rng.choice([1, 2, 255, 256, 257, 4095, 65536, 65537, 300001]))
        k = int(min(N, rng.choice([0, 1, 2, 17, N // 100 + 1, N // 7 + 1, N - 1, N])))
        kinds = [str(rng.choice(["laplace", "normal", "ties", "zeros"])) for _ in range(P)]
        x = np.stack([_row_values(rng, N, kd) for kd in kinds])
        residual = str(rng.choice(["none", "copy", "inplace"]))
        say(f"[sweep topk] #{case}: P={P} N={N} k={k} rows={kinds} residual={residual}")
        oi, ov, orr = oracle.topk(x, k, residual=residual != "none")
        tx = to_dev(x)
        res = None if residual == "none" else ("inplace" if residual == "inplace" else torch.empty_like(tx))
        gi, gv = S.topk_sparsify(tx, k, residual=res)
        torch.cuda.synchronize()
        gi, gv = to_np(gi, np.uint32), to_np(gv)
        np.testing.assert_array_equal(gi, oi, err_msg=f"#{case} indices")
        np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32), err_msg=f"#{case} values")
        if residual != "none":
            gr = to_np(tx if residual == "inplace" else res)
            np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32), err_msg=f"#{case} residual")


def test_random_sweep_quantize():
    import torch
    from gpu_util import to_np
    from paper_1802_08021_amd import sparcml as S
    rng = np.random.default_rng(9113)
    for case in range(40):
        P = int(rng.integers(1, 140))
        bits = int(rng.choice([2, 4, 8]))
        lens = [int(rng.choice([0, 1, 3, 4, 5, 8191, 8192, 8193, 20000])) for _ in range(P)]
        vals = [_row_values(rng, n, str(rng.choice(["laplace", "normal", "ties", "zeros"]))) for n in lens]
        want_deq = bool(rng.random() < 0.5)
        seed = int(rng.integers(0, 2**63))
        say(f"[sweep quant] #{case}: P={P} bits={bits} deq={want_deq}")
        oq, os_, od = oracle.quantize(vals, bits, seed)
        tv = [to_dev(v if v.size else np.zeros(0, np.float32)) for v in vals]
        codes, scale, deq = S.quantize(tv, bits, seed, want_deq=want_deq)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_np(scale).view(np.uint32), os_.view(np.uint32), err_msg=f"#{case} scales")
        for r in range(P):
            np.testing.assert_array_equal(to_np(codes[r])[: oq[r].size], oq[r], err_msg=f"#{case} codes {r}")
            if want_deq:
                np.testing.assert_array_equal(to_np(deq[r])[: od[r].size].view(np.uint32), od[r].view(np.uint32),
                                              err_msg=f"#{case} dequantized {r}")


def test_random_sweep_async_reduce():
    """The entry point the benchmark times (the asynchronous reduce, root
    header on the device), on the reduce sweep's first cases, each run
    twice on the same buffers."""
    import torch
    from gpu_util import to_np
    from paper_1802_08021_amd import sparcml as S
    rng = np.random.default_rng(20261202)
    for case in range(100):
        P, N, idx, val, qbits, delta, rg, label = _case(rng, case)
        say(f"[sweep async] {label}")
        ti = [to_dev(a) for a in idx]
        kw = {} if rg is None else {"lo": rg[0], "hi": rg[1]}
        if qbits:
            q, scale, deq = oracle.quantize(val, qbits, seed=1000 + case)
            codes = [to_dev(a if a.size else np.zeros(1, np.uint8)) for a in q]
            c = S.ReduceCall(ti, N, delta, codes=codes, scales=to_dev(scale), qbits=qbits, node_info=True, **kw)
            vals_o = deq
        else:
            c = S.ReduceCall(ti, N, delta, vals=[to_dev(v) for v in val], node_info=True, **kw)
            vals_o = val
        o = oracle.sparse_reduce(idx, vals_o, N, delta) if rg is None else \
            oracle.sparse_reduce_range(idx, vals_o, N, rg[0], rg[1], delta)
        for rep in range(2):
            c.run_async()
            torch.cuda.synchronize()
            nnz, dense = c.result_header()
            g = {
                "dense": dense, "nnz": nnz,
                "idx": None if dense else to_np(c.out_idx[:nnz], np.uint32).copy(),
                "val": to_np(c.out_val if dense else c.out_val[:nnz]).copy(),
                "node_nnz": to_np(c.node_nnz).astype(np.uint64) if P > 1 else np.zeros(0, np.uint64),
                "node_dense": to_np(c.node_dense) if P > 1 else np.zeros(0, np.uint8),
            }
            assert_reduce_equal(g, o, f"{label} (async, run {rep})")
