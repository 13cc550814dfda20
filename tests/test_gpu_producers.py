"""Parity of the HIP producers (top-k, QSGD) and densify with the oracle.

Top-k: selected indices bit-exact (ties lowest index first), values and
residual bitwise.  QSGD: packed codes and scales bit-exact, dequantized
values bitwise (same Philox stream on both sides).  Densify: bitwise."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def gpu_topk(x, k, residual=None):
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    tx = to_dev(x)
    res = None
    if residual == "copy":
        res = torch.empty_like(tx)
    elif residual == "inplace":
        res = "inplace"
    i, v = S.topk_sparsify(tx, k, residual=res)
    torch.cuda.synchronize()
    out_res = None
    if residual == "copy":
        out_res = to_np(res)
    elif residual == "inplace":
        out_res = to_np(tx)
    return to_np(i, np.uint32), to_np(v), out_res


@pytest.mark.parametrize("residual", [None, "copy", "inplace"])
def test_topk_random(residual):
    rng = np.random.default_rng(20)
    for case in range(12):
        P = int(rng.integers(1, 9))
        N = int(rng.choice([1, 5, 1000, 4097, 70001, 300000]))
        k = int(rng.choice([0, 1, N // 1000, N // 10, N]))
        k = min(k, N)
        x = np.stack([inputs.laplace(rng, 1e-3, N) for _ in range(P)])
        if case % 3 == 1:
            x[:, ::5] = np.float32(-0.25)  # ties with sign differences
            x[:, 1::5] = np.float32(0.25)
        if case % 4 == 2:
            x[:, ::2] = 0.0
        say(f"[topk] case {case} P={P} N={N} k={k} residual={residual}")
        oi, ov, orr = oracle.topk(x, k, residual=residual is not None)
        gi, gv, gr = gpu_topk(x, k, residual)
        np.testing.assert_array_equal(gi, oi)
        np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32))
        if residual is not None:
            np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32))


def test_topk_all_equal_and_config3_scaled():
    x = np.full((3, 9000), 1.5, np.float32)
    x[1, ::2] = -1.5
    say("[topk] all equal magnitudes")
    oi, ov, _ = oracle.topk(x, 1234)
    gi, gv, _ = gpu_topk(x, 1234)
    np.testing.assert_array_equal(gi, oi)
    np.testing.assert_array_equal(gv, ov)
    c = inputs.config(3, scale_log2=4)
    d = inputs.generate(c, seed=0)
    say(f"[topk] c3/16: P={c.P} N={c.N} k={c.k}")
    oi, ov, orr = oracle.topk(d["x"], c.k, residual=True)
    gi, gv, gr = gpu_topk(d["x"], c.k, "copy")
    np.testing.assert_array_equal(gi, oi)
    np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32))
    np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32))


def test_topk_boundary_bin_at_gather_capacity():
    """Every 4096-element unit of the first row holding exactly as many
    entries in or above the k-th largest key's 11-bit bin as a unit gathers
    (32: 8 above the bin, 24 in it), one unit of the second row one more:
    the first row is settled by its gathered entries, the second by the
    extra passes over its data."""
    rng = np.random.default_rng(31)
    N, k, unit = 1 << 18, 600, 4096
    x = np.stack([inputs.laplace(rng, 1e-3, N) for _ in range(2)])
    for r in range(2):
        for u in range(N // unit):
            cnt = 33 if (r == 1 and u == 7) else 32
            pos = u * unit + rng.choice(unit, size=cnt, replace=False)
            sign = np.float32(1.0) if r == 0 else np.float32(-1.0)
            x[r, pos] = sign * np.float32(1.0)
            x[r, pos[::6]] = sign * np.float32(1.0009765625)  # same bin, a larger key
            x[r, pos[1::4][:8]] = sign * np.float32(2.0)       # above the bin
    say(f"[topk] gather capacity P=2 N={N} k={k}")
    for mode in ("copy", "inplace", None):
        oi, ov, orr = oracle.topk(x, k, residual=True)
        gi, gv, gr = gpu_topk(x, k, mode)
        np.testing.assert_array_equal(gi, oi)
        np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32))
        if mode is not None:
            np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32))


def test_topk_sampled_gather_bin_paths():
    """The gather bin comes from a sample of every 16th 256-element segment
    (N = 2^22).  Row 0: its 200 largest values sit only in sampled segments
    and k = 1000, so the sample overestimates and the row must fall back to
    the exact bin.  Row 1: 5000 large values only outside the sample, k =
    100: the estimate holds and every large value is gathered.  Row 2: plain
    Laplace values."""
    rng = np.random.default_rng(32)
    N, seg, stride = 1 << 22, 256, 16
    x = np.stack([inputs.laplace(rng, 1e-3, N) for _ in range(3)])
    sampled = np.arange(0, N // seg, stride) * seg
    x[0, rng.choice(sampled, 200, replace=False)] = np.float32(1.0)
    hidden = (np.arange(0, N // seg, stride) + 1) * seg
    x[1, rng.choice(hidden, 5000, replace=True) + rng.integers(0, seg, 5000)] = np.float32(-3.0)
    for k in (1000, 100):
        say(f"[topk] sampled gather paths N={N} k={k}")
        oi, ov, orr = oracle.topk(x, k, residual=True)
        gi, gv, gr = gpu_topk(x, k, "copy")
        np.testing.assert_array_equal(gi, oi)
        np.testing.assert_array_equal(gv.view(np.uint32), ov.view(np.uint32))
        np.testing.assert_array_equal(gr.view(np.uint32), orr.view(np.uint32))


def gpu_quantize(vals, bits, seed, want_deq=True):
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    tv = [to_dev(v if v.size else np.zeros(0, np.float32)) for v in vals]
    codes, scale, deq = S.quantize(tv, bits, seed, want_deq=want_deq)
    torch.cuda.synchronize()
    return [to_np(c) for c in codes], to_np(scale), [to_np(d) for d in deq] if want_deq else None


def assert_quant_equal(g, o, P, label):
    gq, gs, gd = g
    oq, os_, od = o
    np.testing.assert_array_equal(gs.view(np.uint32), os_.view(np.uint32), err_msg=f"{label}: scales")
    for r in range(P):
        np.testing.assert_array_equal(gq[r], oq[r], err_msg=f"{label}: codes of stream {r}")
        if gd is not None:
            np.testing.assert_array_equal(gd[r].view(np.uint32), od[r].view(np.uint32),
                                          err_msg=f"{label}: dequantized stream {r}")


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_parity(bits):
    rng = np.random.default_rng(30 + bits)
    sizes = [0, 1, 2, 3, 4, 5, 7, 8, 9, 63, 64, 65, 1000, 8191, 8192, 8193, 100003, 1 << 20]
    vals = [inputs.laplace(rng, 1e-3, n) for n in sizes]
    vals.append(np.zeros(77, np.float32))
    vals.append(np.float32(3.0) * np.ones(5, np.float32))
    seed = 0xDEADBEEF_12345678 + bits
    o = oracle.quantize(vals, bits, seed)
    # with dequantized copies the table is uploaded; without, it travels in
    # the kernels' arguments
    for want_deq in (True, False):
        say(f"[quant] bits={bits} streams={len(vals)} deq={want_deq}")
        g = gpu_quantize(vals, bits, seed, want_deq)
        assert_quant_equal(g, o, len(vals), f"deq={want_deq}")


def test_quantize_long_stream():
    # 2^23 + 5 entries: more than 1024 partial norms, so the partials' tree
    # takes two summing launches
    rng = np.random.default_rng(77)
    vals = [inputs.laplace(rng, 1e-2, (1 << 23) + 5), inputs.laplace(rng, 1e-2, 3000)]
    seed = 0x0123456789ABCDEF
    say("[quant] long stream")
    o = oracle.quantize(vals, 4, seed)
    g = gpu_quantize(vals, 4, seed, want_deq=False)
    assert_quant_equal(g, o, len(vals), "long stream")


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_short_stream_boundary(bits):
    """Streams of at most 4 x 8192 elements take norm and codes in one
    launch; the longest one at that limit and one past it (three launches),
    with streams that end inside each of the four norm blocks and on their
    edges."""
    rng = np.random.default_rng(90 + bits)
    sizes = [1, 8191, 8192, 8193, 16385, 24575, 24577, 32767]
    seed = 0xC0FFEE_0000 + bits
    for longest in (32768, 32769):
        vals = [inputs.laplace(rng, 1e-3, n) for n in sizes + [longest]]
        o = oracle.quantize(vals, bits, seed)
        for want_deq in (True, False):
            say(f"[quant] short-stream boundary: longest {longest}, bits={bits}, deq={want_deq}")
            g = gpu_quantize(vals, bits, seed, want_deq)
            assert_quant_equal(g, o, len(vals), f"longest {longest}, deq={want_deq}")


def test_quantize_config5_scaled():
    c = inputs.config(5, scale_log2=5)
    d = inputs.generate(c, seed=0)
    seed = inputs.quant_seed(0, 5)
    say(f"[quant] c5/32 P={c.P} k={c.k}")
    o = oracle.quantize(d["val"], 4, seed)
    for want_deq in (True, False):
        g = gpu_quantize(d["val"], 4, seed, want_deq)
        assert_quant_equal(g, o, c.P, f"c5/32, deq={want_deq}")


def test_densify_parity():
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    rng = np.random.default_rng(40)
    for N in (1, 100, 4096, 4097, 123457):
        for k in (0, 1, N // 7, N):
            idx = inputs.uniform_subset(rng, N, k)
            val = inputs.normal(rng, k)
            say(f"[densify] N={N} k={k}")
            want = oracle.densify(idx, val, N)
            got = S.densify(to_dev(idx), to_dev(val), N)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(to_np(got).view(np.uint32), want.view(np.uint32))
            if k:
                q, sc, deq = oracle.quantize([val], 4, seed=5)
                want_q = oracle.densify(idx, deq[0], N)
                got_q = S.densify(to_dev(idx), None, N, codes=to_dev(q[0]), scale=to_dev(sc), qbits=4)
                torch.cuda.synchronize()
                np.testing.assert_array_equal(to_np(got_q).view(np.uint32), want_q.view(np.uint32))
