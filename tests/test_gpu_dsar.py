"""Parity of the dense-stage pieces of the split-allgather allreduce through
the C ABI with the CPU oracle: bucketed QSGD (§6) -- codes and scales
bit-exact, dequantized values bitwise -- and the concatenation of gathered
shares (§5.1 case (2), §5.3.2) -- representation, nnz and indices exact,
values bitwise.  Also the whole DSAR node pipeline (share reduce, bucketed
QSGD of the dense share, decoding of all gathered shares) against the
oracle's pipeline on the same seeded inputs."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_values, gpu_reduce, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def gpu_quantize_bucketed(vals, bits, bucket, seed, offset=0):
    """``offset`` > 0 places every stream that many floats past an aligned
    start (unaligned loads)."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    tv = []
    for v in vals:
        buf = to_dev(np.concatenate([np.zeros(offset, np.float32), v]))
        tv.append(buf[offset:])
    q, sc, dq = S.quantize_bucketed(tv, bits, bucket, seed, want_deq=True)
    torch.cuda.synchronize()
    return [to_np(c) for c in q], to_np(sc), [to_np(d) for d in dq]


def check_quant(vals, bits, bucket, seed, label, offset=0):
    say(f"[dsar] quantize {label}: bits={bits} B={bucket} sizes={[v.size for v in vals][:6]}")
    q, sc, dq = gpu_quantize_bucketed(vals, bits, bucket, seed, offset)
    oq, osc, odq = oracle.quantize(vals, bits, seed, bucket=bucket)
    np.testing.assert_array_equal(sc.view(np.uint32), osc.view(np.uint32), err_msg=f"{label} scales")
    for r, v in enumerate(vals):
        np.testing.assert_array_equal(q[r], oq[r], err_msg=f"{label} codes of stream {r}")
        assert_values(dq[r], odq[r], f"{label} dequantized stream {r}")


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("bucket", [4, 64, 512, 1024, 2048, 8192])
def test_quantize_bucketed_lengths(bits, bucket):
    rng = np.random.default_rng(400 + bits * 13 + bucket)
    sizes = [0, 1, 3, bucket - 1, bucket, bucket + 1, 5 * bucket + 3, 70001]
    vals = [inputs.laplace(rng, 1e-3, n) for n in sizes]
    vals[4][:] = 0.0  # an all-zero bucket
    check_quant(vals, bits, bucket, seed=0x5EED + bits, label="lengths")


def test_quantize_bucketed_unaligned_and_many_streams():
    rng = np.random.default_rng(401)
    vals = [inputs.normal(rng, int(n)) for n in rng.integers(0, 9000, size=40)]
    check_quant(vals, 4, 1024, seed=11, label="unaligned", offset=1)
    check_quant(vals, 2, 256, seed=12, label="unaligned", offset=3)


def test_quantize_bucketed_share_size():
    """A c5 split-phase share: 2^20 dense values, 4-bit, B = 1024."""
    rng = np.random.default_rng(402)
    v = inputs.laplace(rng, 1e-3, 1 << 20)
    check_quant([v], 4, 1024, seed=13, label="share")


def make_parts(rng, bounds, kinds, qbits=0, bucket=0, seed=0):
    """Host parts for the oracle and device parts for the binding.  kinds[s]
    in {"sparse", "dense", "empty"}; values are Laplace(0, 1)."""
    hp, dp = [], []
    for s, kind in enumerate(kinds):
        lo, hi = bounds[s], bounds[s + 1]
        if kind == "dense":
            idx = None
            v = inputs.laplace(rng, 1.0, hi - lo)
        else:
            k = 0 if kind == "empty" else int(rng.integers(0, hi - lo + 1))
            idx = (inputs.uniform_subset(rng, hi - lo, k).astype(np.uint64) + lo).astype(np.uint32)
            v = inputs.laplace(rng, 1.0, k)
        h = {"idx": idx, "val": v}
        d = {"idx": None if idx is None else to_dev(idx if idx.size else np.zeros(1, np.uint32))[: idx.size]}
        if qbits:
            q, sc, _ = oracle.quantize([v], qbits, seed=seed + s, bucket=bucket)
            h = {"idx": idx, "codes": q[0], "scales": sc if sc.size else np.zeros(1, np.float32),
                 "qbits": qbits, "bucket": bucket, "n": v.size}
            d["codes"] = to_dev(q[0] if q[0].size else np.zeros(1, np.uint8))
            d["scales"] = to_dev(sc if sc.size else np.zeros(1, np.float32))
        else:
            d["val"] = to_dev(v if v.size else np.zeros(1, np.float32))
        hp.append(h)
        dp.append(d)
    return hp, dp


def check_concat(hp, dp, bounds, N, delta, label, qbits=0, bucket=0):
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    say(f"[dsar] concat {label}: P={len(hp)} N={N} delta={delta} qbits={qbits} B={bucket}")
    o = oracle.concat(hp, bounds, N, delta)
    g = S.concat(dp, bounds, N, delta, qbits=qbits, bucket=bucket)
    torch.cuda.synchronize()
    assert g["dense"] == o["dense"], label
    assert g["nnz"] == o["nnz"], label
    if g["dense"]:
        assert_values(to_np(g["val"]), o["val"], f"{label} dense")
    else:
        np.testing.assert_array_equal(to_np(g["idx"], np.uint32), o["idx"], err_msg=f"{label} indices")
        assert_values(to_np(g["val"]), o["val"], f"{label} values")
    return g, o


def test_concat_sparse_and_threshold():
    rng = np.random.default_rng(410)
    N, P = 300007, 16
    b = [N * s // P for s in range(P + 1)]
    hp, dp = make_parts(rng, b, ["sparse"] * P)
    total = sum(h["idx"].size for h in hp)
    g, _ = check_concat(hp, dp, b, N, total / N + 1e-9, "all sparse, thr = total")
    assert not g["dense"]
    g, _ = check_concat(hp, dp, b, N, (total - 1) / N, "all sparse, thr = total - 1")
    assert g["dense"]


def test_concat_mixed_ragged_and_empty_ranges():
    rng = np.random.default_rng(411)
    N = 1000003
    b = [0, 0, 5, 4096, 4097, 300001, 300001, 777777, N]  # empty and 1-wide ranges
    kinds = ["empty", "dense", "sparse", "dense", "sparse", "empty", "dense", "sparse"]
    hp, dp = make_parts(rng, b, kinds)
    check_concat(hp, dp, b, N, 0.5, "mixed")
    kinds = ["empty", "sparse", "sparse", "sparse", "sparse", "empty", "sparse", "sparse"]
    hp, dp = make_parts(rng, b, kinds)
    check_concat(hp, dp, b, N, 0.5, "mixed sparse")
    check_concat(hp, dp, b, N, 1e-6, "mixed sparse -> dense")


@pytest.mark.parametrize("qbits,bucket", [(2, 0), (4, 1024), (8, 64), (4, 4)])
def test_concat_quantized_parts(qbits, bucket):
    rng = np.random.default_rng(412 + qbits + bucket)
    N, P = 500009, 8
    b = [N * s // P for s in range(P + 1)]
    hp, dp = make_parts(rng, b, ["dense"] * P, qbits, bucket, seed=7)
    check_concat(hp, dp, b, N, 0.1, "dense quantized", qbits, bucket)
    hp, dp = make_parts(rng, b, ["sparse", "dense"] * (P // 2), qbits, bucket, seed=8)
    check_concat(hp, dp, b, N, 0.1, "mixed quantized", qbits, bucket)
    hp, dp = make_parts(rng, b, ["sparse"] * P, qbits, bucket, seed=9)
    check_concat(hp, dp, b, N, 5.0, "sparse quantized", qbits, bucket)


def test_concat_unaligned_code_arrays():
    """Dense QSGD parts whose code arrays start at odd byte addresses (the
    per-element decode path) next to aligned ones."""
    torch, dev = torch_dev()
    rng = np.random.default_rng(414)
    N, P, B = 100003, 4, 64
    b = [N * s // P for s in range(P + 1)]
    for bits in (2, 4, 8):
        hp, dp = make_parts(rng, b, ["dense"] * P, bits, B, seed=11)
        for s_, d in enumerate(dp):
            if s_ % 2:
                buf = torch.zeros(d["codes"].numel() + 1, dtype=torch.uint8, device=dev)
                buf[1:] = d["codes"]
                d["codes"] = buf[1:]  # one byte past an aligned start
        check_concat(hp, dp, b, N, 0.1, "unaligned codes", bits, B)


def test_concat_many_parts_and_single_part():
    rng = np.random.default_rng(413)
    N, P = 2000000, 1000
    b = [N * s // P for s in range(P + 1)]
    hp, dp = make_parts(rng, b, ["sparse"] * P)
    check_concat(hp, dp, b, N, 0.6, "1000 parts")
    hp, dp = make_parts(rng, [0, N], ["dense"])
    check_concat(hp, dp, [0, N], N, 0.5, "one dense part")


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_dsar_node_pipeline(bits):
    """One node's DSAR work for every node of a P-way split: the share of
    each range reduced (dense), quantized in buckets of 1024, and all shares
    decoded into the full vector -- against the oracle's pipeline."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(420 + bits)
    P, N, delta, B = 16, 1 << 20, 0.05, 1024
    idx = [inputs.uniform_subset(rng, N, 6000) for _ in range(P)]
    val = [inputs.laplace(rng, 1e-3, 6000) for _ in range(P)]
    b = [N * s // P for s in range(P + 1)]
    hp, dp = [], []
    for s in range(P):
        lo, hi = b[s], b[s + 1]
        m = [(a >= lo) & (a < hi) for a in idx]
        si = [a[k] for a, k in zip(idx, m)]
        sv = [v[k] for v, k in zip(val, m)]
        say(f"[dsar] pipeline bits={bits} share {s}")
        o = oracle.sparse_reduce_range(si, sv, N, lo, hi, delta)
        g = gpu_reduce(si, sv, N, delta, rng=(lo, hi))
        assert o["dense"] and g["dense"]
        assert_values(g["val"], o["val"], f"share {s}")
        oq, osc, _ = oracle.quantize([o["val"]], bits, seed=1000 + s, bucket=B)
        gq, gsc, _ = S.quantize_bucketed([to_dev(g["val"])], bits, B, 1000 + s)
        np.testing.assert_array_equal(to_np(gq[0]), oq[0], err_msg=f"share {s} codes")
        np.testing.assert_array_equal(to_np(gsc).view(np.uint32), osc.view(np.uint32))
        hp.append({"idx": None, "codes": oq[0], "scales": osc, "qbits": bits, "bucket": B, "n": hi - lo})
        dp.append({"idx": None, "codes": gq[0], "scales": gsc})
    o = oracle.concat(hp, b, N, delta)
    g = S.concat(dp, b, N, delta, qbits=bits, bucket=B)
    torch.cuda.synchronize()
    assert g["dense"] and o["dense"]
    assert_values(to_np(g["val"]), o["val"], "gathered DSAR result")


@pytest.mark.parametrize("bits", [4])
def test_dsar_pipeline_appendix_a_partition(bits):
    """The DSAR node pipeline over App. A's partition with N not divisible
    by P (N = 2^20 + 12345, P = 48: 47 ranges of floor(N/P) indices, the
    last one 45 longer), and with every rank's share taken from the full
    streams: share reduce, bucketed QSGD, decode of all shares."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(440)
    P, N, delta, B = 48, (1 << 20) + 12345, 0.05, 1024
    b = S.split_bounds(P, N)
    assert b[1] == N // P and b[-1] - b[-2] == N - (P - 1) * (N // P) and (N % P) != 0
    idx = [inputs.uniform_subset(rng, N, 4000) for _ in range(P)]
    val = [inputs.laplace(rng, 1e-3, 4000) for _ in range(P)]
    hp, dp = [], []
    for s in range(P):
        lo, hi = b[s], b[s + 1]
        cut = [np.searchsorted(a, (lo, hi)) for a in idx]
        si = [a[x:y] for a, (x, y) in zip(idx, cut)]
        sv = [v[x:y] for v, (x, y) in zip(val, cut)]
        if s % 12 == 0:
            say(f"[dsar] App. A partition P={P} N={N} share {s} [{lo}, {hi})")
        o = oracle.sparse_reduce_range(si, sv, N, lo, hi, delta)
        g = gpu_reduce(si, sv, N, delta, rng=(lo, hi))
        assert g["dense"] == o["dense"]
        assert_values(g["val"], o["val"], f"share {s}")
        ov = o["val"] if o["dense"] else oracle.densify((o["idx"].astype(np.int64) - lo).astype(np.uint32),
                                                          o["val"], hi - lo)
        gv = g["val"] if g["dense"] else None
        oq, osc, _ = oracle.quantize([ov], bits, seed=2000 + s, bucket=B)
        if gv is None:
            gv = to_np(S.densify(to_dev((g["idx"].astype(np.int64) - lo).astype(np.uint32)),
                                 to_dev(g["val"]), hi - lo))
        gq, gsc, _ = S.quantize_bucketed([to_dev(gv)], bits, B, 2000 + s)
        np.testing.assert_array_equal(to_np(gq[0]), oq[0], err_msg=f"share {s} codes")
        np.testing.assert_array_equal(to_np(gsc).view(np.uint32), osc.view(np.uint32))
        hp.append({"idx": None, "codes": oq[0], "scales": osc, "qbits": bits, "bucket": B, "n": hi - lo})
        dp.append({"idx": None, "codes": gq[0], "scales": gsc})
    o = oracle.concat(hp, b, N, delta)
    g = S.concat(dp, b, N, delta, qbits=bits, bucket=B)
    torch.cuda.synchronize()
    assert g["dense"] and o["dense"]
    assert_values(to_np(g["val"]), o["val"], "gathered DSAR result, App. A partition")
