"""C-ABI checks that need no GPU: the library loads, exports every entry
point include/sparcml.h declares, and rejects bad arguments on the host
before any device work (so these calls never reach the HIP runtime)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_1802_08021_amd import sparcml as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparcml.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SPARCML_API\s+[\w\s\*]+?\b(sparcml_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for name in ("sparcml_topk_sparsify", "sparcml_quantize", "sparcml_sparse_reduce",
                 "sparcml_sparse_reduce_range", "sparcml_quantize_bucketed", "sparcml_concat",
                 "sparcml_topk_bucketed", "sparcml_topk_bucketed_count", "sparcml_sparse_reduce_async",
                 "sparcml_densify", "sparcml_split_bounds", "sparcml_validate_streams",
                 "sparcml_workspace_size", "sparcml_strerror",
                 "sparcml_last_error"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    L = S.lib()
    for name in declared_symbols():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", S.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\b[TW]\s+(\S+)$", out, flags=re.M))
    assert set(declared_symbols()) <= exported
    # nothing but the ABI is exported from the library's own code
    assert all(e.startswith("sparcml_") for e in exported if "sparcml" in e)


def test_strerror_codes():
    assert S.strerror(0) == "success"
    for code in (S.EINVAL, S.ECAPACITY, S.EWORKSPACE, S.EUNSORTED, S.EHIP):
        assert S.strerror(code) and S.strerror(code) != "unknown status"
    assert S.strerror(-99) == "unknown status"


def ws_size(op, P, N, max_nnz, delta=1.0):
    n = ctypes.c_size_t(0)
    rc = S.lib().sparcml_workspace_size(op, P, N, max_nnz, delta, ctypes.byref(n))
    return rc, n.value


def test_workspace_size_queries():
    rc, n = ws_size(S.OP_REDUCE, 128, 2**27, 2**27 // 100, 0.1)
    assert rc == 0 and n > 0
    rc2, n2 = ws_size(S.OP_REDUCE, 128, 2**27, 2**27 // 10, 0.1)
    assert rc2 == 0 and n2 >= n  # larger max_nnz never needs less
    assert ws_size(S.OP_REDUCE, 0, 100, 10)[0] == S.EINVAL
    assert ws_size(S.OP_REDUCE, 3, 100, 10)[0] == S.OK  # a tree over 4 slots
    assert ws_size(S.OP_REDUCE, 257, 100, 10)[0] == S.EINVAL
    assert ws_size(S.OP_REDUCE, 512, 100, 10)[0] == S.EINVAL
    assert ws_size(S.OP_REDUCE, 4, 0, 0)[0] == S.EINVAL
    assert ws_size(S.OP_REDUCE, 4, 2**32, 1)[0] == S.EINVAL
    assert ws_size(S.OP_REDUCE, 4, 100, 10, 0.0)[0] == S.EINVAL
    assert ws_size(S.OP_TOPK, 32, 2**24, 2**24 // 1000)[0] == 0
    assert ws_size(S.OP_TOPK, 1, 10, 11)[0] == S.EINVAL
    assert ws_size(S.OP_QUANTIZE, 128, 1, 2**20)[0] == 0
    assert ws_size(S.OP_DENSIFY, 1, 10, 0)[0] == 0
    assert ws_size(99, 1, 10, 0)[0] == S.EINVAL
    assert S.lib().sparcml_workspace_size(S.OP_DENSIFY, 1, 10, 0, 1.0, None) == S.EINVAL


FAKE = 0x1000  # never dereferenced: every call below fails validation first


def streams(P, nnz=4, qbits=0, dense=0):
    arr = (S.Stream * P)()
    for r in range(P):
        arr[r] = S.Stream(FAKE, FAKE, FAKE if qbits else None, FAKE if qbits else None,
                          nnz, dense, qbits)
    return arr


def reduce_rc(P, arr, N=100, delta=0.5, out=None, ws=FAKE, ws_bytes=1 << 40):
    if out is None:
        out = S.Stream(FAKE, FAKE, None, None, 1 << 30, 0, 0)
    return S.lib().sparcml_sparse_reduce(P, arr, N, delta, ctypes.byref(out), None, None,
                                         ws, ws_bytes, None)


def test_reduce_argument_errors():
    assert reduce_rc(0, streams(1)) == S.EINVAL
    assert reduce_rc(512, streams(512)) == S.EINVAL      # beyond the supported P
    assert reduce_rc(4, streams(4), N=0) == S.EINVAL
    assert reduce_rc(4, streams(4), N=2**32) == S.EINVAL
    assert reduce_rc(4, streams(4), delta=0.0) == S.EINVAL
    assert reduce_rc(4, streams(4), delta=float("nan")) == S.EINVAL
    assert reduce_rc(4, streams(4, nnz=101)) == S.EINVAL  # nnz > N
    assert reduce_rc(4, streams(4, dense=1)) == S.EINVAL  # leaves must be sparse
    mixed = streams(4)
    mixed[2] = S.Stream(FAKE, None, FAKE, FAKE, 4, 0, 4)
    assert reduce_rc(4, mixed) == S.EINVAL                # mixed qbits
    assert reduce_rc(4, streams(4, qbits=3)) == S.EINVAL
    noscale = streams(4, qbits=4)
    noscale[1] = S.Stream(FAKE, None, FAKE, None, 4, 0, 4)
    assert reduce_rc(4, noscale) == S.EINVAL
    nullidx = streams(4)
    nullidx[0] = S.Stream(None, FAKE, None, None, 4, 0, 0)
    assert reduce_rc(4, nullidx) == S.EINVAL
    assert S.lib().sparcml_sparse_reduce(4, None, 100, 0.5, None, None, None, FAKE, 1, None) == S.EINVAL
    out = S.Stream(FAKE, None, None, None, 100, 0, 0)
    assert reduce_rc(4, streams(4), out=out) == S.EINVAL  # out->val NULL
    assert "val" in S.last_error()


def range_rc(P, arr, N=100, lo=0, hi=100, delta=0.5, out=None, ws=FAKE, ws_bytes=1 << 40):
    if out is None:
        out = S.Stream(FAKE, FAKE, None, None, 1 << 30, 0, 0)
    return S.lib().sparcml_sparse_reduce_range(P, arr, N, lo, hi, delta, ctypes.byref(out), None,
                                               None, ws, ws_bytes, None)


def test_reduce_range_argument_errors():
    assert range_rc(4, streams(4), lo=10, hi=10) == S.EINVAL   # empty range
    assert range_rc(4, streams(4), lo=20, hi=10) == S.EINVAL
    assert range_rc(4, streams(4), lo=0, hi=101) == S.EINVAL   # hi > N
    assert range_rc(4, streams(4), N=0, lo=0, hi=0) == S.EINVAL
    assert range_rc(4, streams(4), N=2**32, lo=0, hi=5) == S.EINVAL
    assert range_rc(4, streams(4, nnz=11), lo=40, hi=50) == S.EINVAL  # nnz > hi - lo
    assert "range" in S.last_error()
    assert range_rc(0, streams(1), lo=0, hi=50) == S.EINVAL
    # the capacity bound uses the range's threshold: floor(0.5 * 40) = 20 >= 16 entries
    small = S.Stream(FAKE, FAKE, None, None, 15, 0, 0)
    assert range_rc(4, streams(4), lo=30, hi=70, out=small) == S.ECAPACITY
    assert range_rc(4, streams(4), lo=30, hi=70, ws_bytes=16) == S.EWORKSPACE


def test_reduce_async_argument_errors():
    L = S.lib()
    out = S.Stream(FAKE, FAKE, None, None, 1 << 30, 0, 0)

    def rc(P=4, arr=None, N=100, lo=0, hi=100, result=FAKE, ws_bytes=1 << 40, o=out):
        return L.sparcml_sparse_reduce_async(P, streams(P) if arr is None else arr, N, lo, hi, 0.5,
                                             ctypes.byref(o) if o is not None else None, None, None,
                                             result, FAKE, ws_bytes, None)
    assert rc(result=None) == S.EINVAL
    assert rc(lo=5, hi=5) == S.EINVAL and rc(hi=101) == S.EINVAL
    assert rc(P=0, arr=streams(1)) == S.EINVAL
    assert rc(o=None) == S.EINVAL
    assert rc(ws_bytes=16) == S.EWORKSPACE
    assert rc(o=S.Stream(FAKE, FAKE, None, None, 15, 0, 0)) == S.ECAPACITY


def test_reduce_capacity_and_workspace_errors():
    # sum nnz = 16, thr = 50: capacity must be >= 16
    small = S.Stream(FAKE, FAKE, None, None, 15, 0, 0)
    assert reduce_rc(4, streams(4), out=small) == S.ECAPACITY
    # P == 1 sparse copy needs nnz_0 entries
    assert reduce_rc(1, streams(1, nnz=10), out=S.Stream(FAKE, FAKE, None, None, 9, 0, 0)) == S.ECAPACITY
    assert reduce_rc(4, streams(4), ws=None, ws_bytes=0) == S.EWORKSPACE
    assert reduce_rc(4, streams(4), ws_bytes=16) == S.EWORKSPACE


def test_topk_argument_errors():
    L = S.lib()
    assert L.sparcml_topk_sparsify(0, FAKE, 10, 1, FAKE, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_topk_sparsify(1, FAKE, 10, 11, FAKE, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_topk_sparsify(1, None, 10, 1, FAKE, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_topk_sparsify(1, FAKE, 10, 1, None, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_topk_sparsify(1, FAKE, 0, 0, FAKE, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_topk_sparsify(2, FAKE, 1000, 10, FAKE, FAKE, None, FAKE, 8, None) == S.EWORKSPACE
    # one row per grid row: more than 65535 rows is refused before any launch
    assert L.sparcml_topk_sparsify(65536, FAKE, 10, 1, FAKE, FAKE, None, FAKE, 1 << 40, None) == S.EINVAL
    assert "65535" in S.last_error()
    assert ws_size(S.OP_TOPK, 65536, 10, 1)[0] == S.EINVAL


def test_topk_bucketed_argument_errors_and_count():
    L = S.lib()
    ok = dict(P=2, g=FAKE, e=FAKE, N=1000, a=0.1, B=512, kb=4, i=FAKE, v=FAKE)

    def rc(**kw):
        a = dict(ok, **kw)
        return L.sparcml_topk_bucketed(a["P"], a["g"], a["e"], a["N"], a["a"], a["B"], a["kb"], a["i"], a["v"], None)
    assert rc(P=0) == S.EINVAL
    assert rc(N=0) == S.EINVAL
    assert rc(N=2**32) == S.EINVAL
    for b in (0, 32, 100, 8192):
        assert rc(B=b) == S.EINVAL
    assert rc(kb=0) == S.EINVAL and rc(kb=65) == S.EINVAL
    assert rc(e=None) == S.EINVAL and rc(i=None) == S.EINVAL
    assert rc(a=float("nan")) == S.EINVAL
    cnt = L.sparcml_topk_bucketed_count
    assert cnt(1000, 512, 4) == 8 and cnt(1000, 512, 500) == 500 + 488 and cnt(3, 512, 4) == 3
    assert cnt(1 << 24, 512, 4) == (1 << 24) // 128 and cnt(0, 512, 4) == 0


def test_quantize_argument_errors():
    L = S.lib()
    q = (ctypes.c_void_p * 4)(*([FAKE] * 4))
    arr = streams(4)
    assert L.sparcml_quantize(4, arr, 3, 1, ctypes.cast(q, ctypes.c_void_p), FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize(0, arr, 4, 1, ctypes.cast(q, ctypes.c_void_p), FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize(4, arr, 4, 1, None, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize(4, arr, 4, 1, ctypes.cast(q, ctypes.c_void_p), None, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize(4, streams(4, qbits=4), 4, 1, ctypes.cast(q, ctypes.c_void_p), FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize(4, arr, 4, 1, ctypes.cast(q, ctypes.c_void_p), FAKE, None, FAKE, 8, None) == S.EWORKSPACE
    # more streams than grid rows
    big = streams(65536)
    qb = ctypes.cast((ctypes.c_void_p * 65536)(*([FAKE] * 65536)), ctypes.c_void_p)
    assert L.sparcml_quantize(65536, big, 4, 1, qb, FAKE, None, FAKE, 1 << 40, None) == S.EINVAL
    assert ws_size(S.OP_QUANTIZE, 65536, 1, 10)[0] == S.EINVAL


def test_quantize_counter_limit():
    """Element j of a stream draws from Philox counter word j >> 2, which is
    32 bits wide: a stream of 2^34 entries uses every counter once, a longer
    one would repeat draws and is refused on the host."""
    L = S.lib()
    q = ctypes.cast((ctypes.c_void_p * 2)(FAKE, FAKE), ctypes.c_void_p)
    ok = streams(2, nnz=1 << 34)
    bad = streams(2, nnz=(1 << 34) + 1)
    # at the limit validation passes and only the (too small) workspace fails
    assert L.sparcml_quantize(2, ok, 4, 1, q, FAKE, None, FAKE, 8, None) == S.EWORKSPACE
    assert L.sparcml_quantize(2, bad, 4, 1, q, FAKE, None, FAKE, 1 << 40, None) == S.EINVAL
    assert "2^34" in S.last_error()
    assert L.sparcml_quantize_bucketed(2, bad, 4, 1024, 1, q, FAKE, None, FAKE, 1 << 40, None) == S.EINVAL
    # the highest element of a maximal stream uses counter word 2^32 - 1
    assert ((1 << 34) - 1) >> 2 == 2**32 - 1


def test_split_bounds_follow_appendix_a():
    """App. A: every node but the last gets floor(N/P) indices, the last the
    remaining N - (P-1) floor(N/P)."""
    for P, N in ((48, (1 << 20) + 12345), (128, 1 << 27), (7, 100), (5, 3), (1, 9), (65535, 2**32 - 1)):
        b = S.split_bounds(P, N)
        assert len(b) == P + 1 and b[0] == 0 and b[-1] == N
        sizes = [b[s + 1] - b[s] for s in range(P)]
        assert all(x == N // P for x in sizes[:-1])
        assert sizes[-1] == N - (P - 1) * (N // P)
    b = (ctypes.c_uint64 * 3)()
    assert S.lib().sparcml_split_bounds(0, 10, b) == S.EINVAL
    assert S.lib().sparcml_split_bounds(65536, 10, None) == S.EINVAL
    assert S.lib().sparcml_split_bounds(2, 0, b) == S.EINVAL
    assert S.lib().sparcml_split_bounds(2, 2**32, b) == S.EINVAL
    assert S.lib().sparcml_split_bounds(2, 10, None) == S.EINVAL


def test_quantize_bucketed_argument_errors():
    L = S.lib()
    q = ctypes.cast((ctypes.c_void_p * 4)(*([FAKE] * 4)), ctypes.c_void_p)
    arr = streams(4)
    for bad in (0, 2, 3, 100, 16384):
        assert L.sparcml_quantize_bucketed(4, arr, 4, bad, 1, q, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert "bucket" in S.last_error()
    assert L.sparcml_quantize_bucketed(4, arr, 5, 1024, 1, q, FAKE, None, FAKE, 1 << 30, None) == S.EINVAL
    assert L.sparcml_quantize_bucketed(4, arr, 4, 1024, 1, q, FAKE, None, FAKE, 8, None) == S.EWORKSPACE
    assert ws_size(S.OP_QUANTIZE_BUCKETED, 4, 1, 0) == (S.OK, 256)


def concat_rc(parts, bounds, N=100, delta=0.5, bucket=0, out=None, ws=FAKE, ws_bytes=1 << 30):
    P = len(bounds) - 1
    b = (ctypes.c_uint64 * len(bounds))(*bounds)
    if out is None:
        out = S.Stream(FAKE, FAKE, None, None, 1 << 30, 0, 0)
    return S.lib().sparcml_concat(P, parts, b, N, delta, bucket, ctypes.byref(out), ws, ws_bytes, None)


def test_concat_argument_errors():
    # every call below fails validation before any device work
    sp = streams(2, nnz=4)
    assert concat_rc(sp, [1, 50, 100]) == S.EINVAL       # bounds[0] != 0
    assert concat_rc(sp, [0, 50, 99]) == S.EINVAL        # bounds[P] != N
    assert concat_rc(streams(3, nnz=4), [0, 60, 50, 100]) == S.EINVAL  # decreasing bounds
    assert concat_rc(streams(2, nnz=51), [0, 50, 100]) == S.EINVAL  # more entries than the range
    dense = streams(2, nnz=49, dense=1)
    assert concat_rc(dense, [0, 50, 100]) == S.EINVAL    # a dense part must hold its range
    assert concat_rc(sp, [0, 50, 100], N=0) == S.EINVAL
    assert concat_rc(sp, [0, 50, 100], delta=0.0) == S.EINVAL
    assert concat_rc(sp, [0, 50, 100], bucket=3) == S.EINVAL
    mixed = streams(2, nnz=4)
    mixed[1] = S.Stream(FAKE, None, FAKE, FAKE, 4, 0, 4)
    assert concat_rc(mixed, [0, 50, 100]) == S.EINVAL    # mixed qbits
    noscale = streams(2, nnz=4, qbits=4)
    noscale[0] = S.Stream(FAKE, None, FAKE, None, 4, 0, 4)
    assert concat_rc(noscale, [0, 50, 100]) == S.EINVAL
    # 8 entries, thr = 50: the result stays sparse and needs 8 output entries
    assert concat_rc(sp, [0, 50, 100], out=S.Stream(FAKE, FAKE, None, None, 7, 0, 0)) == S.ECAPACITY
    assert concat_rc(sp, [0, 50, 100], ws_bytes=8) == S.EWORKSPACE
    assert S.lib().sparcml_concat(0, sp, None, 100, 0.5, 0, None, FAKE, 1, None) == S.EINVAL


def test_densify_argument_errors():
    L = S.lib()
    s = S.Stream(FAKE, FAKE, None, None, 4, 0, 0)
    assert L.sparcml_densify(None, 10, FAKE, None) == S.EINVAL
    assert L.sparcml_densify(ctypes.byref(s), 10, None, None) == S.EINVAL
    assert L.sparcml_densify(ctypes.byref(s), 0, FAKE, None) == S.EINVAL
    big = S.Stream(FAKE, FAKE, None, None, 11, 0, 0)
    assert L.sparcml_densify(ctypes.byref(big), 10, FAKE, None) == S.EINVAL
    q = S.Stream(FAKE, None, FAKE, None, 4, 0, 4)
    assert L.sparcml_densify(ctypes.byref(q), 10, FAKE, None) == S.EINVAL
    q3 = S.Stream(FAKE, None, FAKE, FAKE, 4, 0, 3)
    assert L.sparcml_densify(ctypes.byref(q3), 10, FAKE, None) == S.EINVAL


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(S, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(S, "_lib", None)
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        S.lib()


def test_validate_argument_errors():
    L = S.lib()
    assert ws_size(S.OP_VALIDATE, 4, 1, 0)[0] == S.OK
    assert ws_size(S.OP_VALIDATE, 0, 1, 0)[0] == S.EINVAL
    assert ws_size(S.OP_VALIDATE, 65536, 1, 0)[0] == S.EINVAL

    def rc(P=4, arr=None, lo=0, hi=100, ws=FAKE, nb=1 << 20):
        return L.sparcml_validate_streams(P, streams(P) if arr is None else arr, lo, hi, ws, nb, None)
    assert rc(P=0, arr=streams(1)) == S.EINVAL
    assert L.sparcml_validate_streams(2, None, 0, 10, FAKE, 1 << 20, None) == S.EINVAL
    assert rc(lo=10, hi=10) == S.EINVAL and rc(lo=0, hi=2**32 + 1) == S.EINVAL
    assert rc(arr=streams(4, dense=1)) == S.EINVAL
    nullidx = streams(4)
    nullidx[3] = S.Stream(None, FAKE, None, None, 4, 0, 0)
    assert rc(arr=nullidx) == S.EINVAL
    assert rc(nb=8) == S.EWORKSPACE and rc(ws=None) == S.EWORKSPACE
