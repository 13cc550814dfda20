"""SparCML reference oracle -- TEST INFRASTRUCTURE ONLY.

Python (ctypes + numpy) front end of ``liboracle.so``, the plain sequential C
implementation of the SparCML definitions (arXiv 1802.08021).  Only the
tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path.

Functions follow the paper:
  * ``sparse_reduce``  -- §5.1 sparse streams, switch rule, pairwise sum;
                          §5.3.1 recursive doubling order.
  * ``sparse_reduce_range`` -- one node's share of the split phase of the
                          large-data allreduce (§5.3.2).
  * ``concat``         -- the gathered shares summed as a concatenation
                          (§5.1 case (2), §5.3.2 allgather phase, §6 dense
                          stage in QSGD buckets).
  * ``topk``           -- §2.2 Top-k sparsification, Alg. 1 error update.
  * ``topk_bucketed``  -- §8.4 k of every group of consecutive coordinates,
                          with Alg. 1's accumulate and error update.
  * ``quantize``       -- §2.2 / §6 QSGD stochastic quantization.
  * ``dequantize``, ``densify``, ``philox4x32_10``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SOURCES = [os.path.join(_HERE, "oracle.c")]


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (no contraction, no fast-math)."""
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-pthread",
           "-fPIC", "-shared", "-o", tmp] + _SOURCES + ["-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        vp = ctypes.c_void_p
        L.orc_philox4x32_10.argtypes = [u32p, u32p, u32p]
        L.orc_philox4x32_10.restype = None
        L.orc_set_threads.argtypes = [ctypes.c_int]
        L.orc_set_threads.restype = None
        L.orc_get_threads.argtypes = []
        L.orc_get_threads.restype = ctypes.c_int
        L.orc_sparse_reduce.argtypes = [
            ctypes.c_int, vp, vp, vp, ctypes.c_uint64, ctypes.c_double,
            vp, ctypes.c_uint64, vp, vp, vp, vp, vp]
        L.orc_sparse_reduce.restype = ctypes.c_int
        L.orc_topk.argtypes = [ctypes.c_int, vp, ctypes.c_uint64, ctypes.c_uint64, vp, vp, vp]
        L.orc_topk.restype = ctypes.c_int
        L.orc_quantize.argtypes = [ctypes.c_int, vp, vp, ctypes.c_int, ctypes.c_uint64, vp, vp, vp]
        L.orc_quantize.restype = ctypes.c_int
        L.orc_dequantize.argtypes = [vp, ctypes.c_float, ctypes.c_int, ctypes.c_uint64, vp]
        L.orc_dequantize.restype = ctypes.c_int
        L.orc_topk_bucketed.argtypes = [ctypes.c_int, vp, vp, ctypes.c_uint64, ctypes.c_float,
                                        ctypes.c_uint64, ctypes.c_uint64, vp, vp]
        L.orc_topk_bucketed.restype = ctypes.c_int
        L.orc_quantize_bucketed.argtypes = [ctypes.c_int, vp, vp, ctypes.c_int, ctypes.c_uint64,
                                            ctypes.c_uint64, vp, vp, vp]
        L.orc_quantize_bucketed.restype = ctypes.c_int
        L.orc_dequantize_bucketed.argtypes = [vp, vp, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, vp]
        L.orc_dequantize_bucketed.restype = ctypes.c_int
        L.orc_densify.argtypes = [vp, vp, ctypes.c_uint64, ctypes.c_uint64, vp]
        L.orc_densify.restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data if a.size else 0


def _ptr_table(arrs):
    return (ctypes.c_void_p * len(arrs))(*[_ptr(a) for a in arrs])


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block (Salmon et al., SC'11)."""
    c = (ctypes.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (ctypes.c_uint32 * 4)()
    lib().orc_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def set_threads(n: int) -> None:
    """Threads for the independent items of a call (the nodes of one tree
    level, the rows of top-k, the streams of quantization); results are the
    same bits for any count.  Default 1."""
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


class threads:
    """``with oracle.threads(n): ...`` -- n threads inside, the previous
    count restored afterwards."""

    def __init__(self, n: int):
        self.n, self.prev = int(n), None

    def __enter__(self):
        self.prev = get_threads()
        set_threads(self.n)
        return self

    def __exit__(self, *exc):
        set_threads(self.prev)
        return False


def threshold(N: int, delta: float) -> int:
    """Sparse-item threshold: floor(delta * N) in double (§5.1)."""
    return int(np.floor(np.float64(delta) * np.float64(N)))


def sparse_reduce(idx_list, val_list, N: int, delta: float):
    """Recursive-doubling sparse allreduce with the dense switch.

    Returns dict(idx, val, nnz, dense, node_nnz, node_dense); for a dense root
    ``val`` holds all N values and ``idx`` is None.
    """
    P = len(idx_list)
    idx_list = [np.ascontiguousarray(a, dtype=np.uint32) for a in idx_list]
    val_list = [np.ascontiguousarray(a, dtype=np.float32) for a in val_list]
    nnz = np.array([a.size for a in idx_list], dtype=np.uint64)
    cap = int(min(nnz.sum(), N)) if P else 0
    out_idx = np.zeros(max(cap, 1), dtype=np.uint32)
    out_val = np.zeros(N, dtype=np.float32)
    out_nnz = np.zeros(1, dtype=np.uint64)
    out_dense = np.zeros(1, dtype=np.int32)
    node_nnz = np.zeros(max(P - 1, 1), dtype=np.uint64)
    node_dense = np.zeros(max(P - 1, 1), dtype=np.uint8)
    rc = lib().orc_sparse_reduce(
        P, _ptr_table(idx_list), _ptr_table(val_list), nnz.ctypes.data, N, float(delta),
        out_idx.ctypes.data, cap, out_val.ctypes.data, out_nnz.ctypes.data,
        out_dense.ctypes.data, node_nnz.ctypes.data, node_dense.ctypes.data)
    if rc != 0:
        raise OracleError(f"orc_sparse_reduce returned {rc}")
    n = int(out_nnz[0])
    dense = bool(out_dense[0])
    return {
        "idx": None if dense else out_idx[:n].copy(),
        "val": out_val if dense else out_val[:n].copy(),
        "nnz": n,
        "dense": dense,
        "node_nnz": node_nnz[: P - 1].copy(),
        "node_dense": node_dense[: P - 1].copy(),
    }


def sparse_reduce_range(idx_list, val_list, N: int, lo: int, hi: int, delta: float):
    """One node's share of the split phase of the large-data (split-allgather)
    allreduce, §5.3.2: the node responsible for the index range [lo, hi)
    reduces the part of every rank's stream that falls in it.  The share is
    the reduction of those parts as a vector of hi - lo coordinates (index
    lo + i at i): threshold floor(delta * (hi - lo)), recursive-doubling
    association as in ``sparse_reduce``.  Entries outside [lo, hi) are
    dropped.  A sparse root's ``idx`` holds absolute indices; a dense root's
    ``val`` holds hi - lo values."""
    if not (0 <= lo < hi <= N):
        raise OracleError("need 0 <= lo < hi <= N")
    parts_i, parts_v = [], []
    for a, v in zip(idx_list, val_list):
        a = np.asarray(a, dtype=np.uint64)
        keep = (a >= lo) & (a < hi)
        parts_i.append((a[keep] - lo).astype(np.uint32))
        parts_v.append(np.asarray(v, dtype=np.float32)[keep])
    res = sparse_reduce(parts_i, parts_v, hi - lo, delta)
    if not res["dense"]:
        res["idx"] = (res["idx"].astype(np.uint64) + lo).astype(np.uint32)
    return res


def part_values(part) -> np.ndarray:
    """Stored values of one part: fp32 as given, or QSGD codes dequantized
    with one scale (``bucket`` 0) or one per ``bucket`` entries (§6)."""
    if part.get("qbits", 0):
        n = part["n"]
        return dequantize(part["codes"], part["scales"] if part.get("bucket", 0) else part["scales"][0],
                          part["qbits"], n, bucket=part.get("bucket", 0))
    return np.asarray(part["val"], dtype=np.float32)


def concat(parts, bounds, N: int, delta: float):
    """Sum of P vectors with disjoint index ranges, part s covering
    [bounds[s], bounds[s+1]) -- the gathered shares of the split-allgather
    allreduce (§5.3.2).  Disjoint index sets make the sum a concatenation
    (§5.1, case (2)).  A part is sparse (``idx`` absolute, ascending, in its
    range; values) or dense (its range's values, ``idx`` None), with fp32
    values or QSGD codes (§6).  The result is dense if a part is dense or
    the parts hold more than thr = floor(delta * N) entries together (the
    representation rule of §5.1); then every index without an entry is
    +0.0.  Returns dict(idx, val, nnz, dense)."""
    P = len(parts)
    if len(bounds) != P + 1 or bounds[0] != 0 or bounds[-1] != N or any(
            bounds[s] > bounds[s + 1] for s in range(P)):
        raise OracleError("bounds must rise from 0 to N")
    total = 0
    any_dense = False
    for s, part in enumerate(parts):
        lo, hi = bounds[s], bounds[s + 1]
        if part["idx"] is None:
            any_dense = True
            if len(part_values(part)) != hi - lo:
                raise OracleError(f"dense part {s} must hold {hi - lo} values")
        else:
            a = np.asarray(part["idx"], dtype=np.int64)
            if a.size and (a[0] < lo or a[-1] >= hi or np.any(np.diff(a) <= 0)):
                raise OracleError(f"part {s}: indices must ascend inside [{lo}, {hi})")
            total += a.size
    thr = threshold(N, delta)
    if any_dense or total > thr:
        out = np.zeros(N, dtype=np.float32)
        for s, part in enumerate(parts):
            v = part_values(part)
            if part["idx"] is None:
                out[bounds[s]: bounds[s + 1]] = v
            else:
                out[np.asarray(part["idx"], dtype=np.int64)] = v
        return {"idx": None, "val": out, "nnz": N, "dense": True}
    idx = [np.asarray(p["idx"], dtype=np.uint32) for p in parts]
    val = [part_values(p) for p in parts]
    return {"idx": np.concatenate(idx) if idx else np.zeros(0, np.uint32),
            "val": np.concatenate(val) if val else np.zeros(0, np.float32),
            "nnz": total, "dense": False}


def topk(x: np.ndarray, k: int, residual: bool = False):
    """Exact per-row top-k by magnitude of x[P, N] by a full sort."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    P, N = x.shape
    out_idx = np.zeros((P, max(k, 1)), dtype=np.uint32)
    out_val = np.zeros((P, max(k, 1)), dtype=np.float32)
    res = x.copy() if residual else None
    rc = lib().orc_topk(P, x.ctypes.data, N, k, out_idx.ctypes.data, out_val.ctypes.data,
                        res.ctypes.data if residual else None)
    if rc != 0:
        raise OracleError(f"orc_topk returned {rc}")
    return out_idx[:, :k].copy(), out_val[:, :k].copy(), res


def scale_counts(sizes, bucket: int):
    """Scales per stream: ceil(n / bucket), or 1 when bucket == 0."""
    return [(n + bucket - 1) // bucket if bucket else 1 for n in sizes]


def bucketed_count(N: int, bucket: int, kb: int) -> int:
    """Entries per rank of the bucketed top-k: min(kb, len) per bucket."""
    nb = (N + bucket - 1) // bucket
    return (nb - 1) * kb + min(kb, N - (nb - 1) * bucket)


def topk_bucketed(eps: np.ndarray, grad, alpha: float, bucket: int, kb: int):
    """Alg. 1's error-feedback step with bucketed selection (§8.4): acc =
    eps + alpha * grad in fp32 (grad None: acc = eps); from each bucket of
    ``bucket`` consecutive coordinates the kb largest magnitudes.  Returns
    (idx [P, K], val [P, K], new eps [P, N])."""
    e = np.ascontiguousarray(eps, dtype=np.float32).copy()
    P, N = e.shape
    g = None if grad is None else np.ascontiguousarray(grad, dtype=np.float32)
    K = bucketed_count(N, bucket, kb)
    out_idx = np.zeros((P, max(K, 1)), dtype=np.uint32)
    out_val = np.zeros((P, max(K, 1)), dtype=np.float32)
    rc = lib().orc_topk_bucketed(P, None if g is None else g.ctypes.data, e.ctypes.data, N,
                                 ctypes.c_float(alpha), bucket, kb, out_idx.ctypes.data,
                                 out_val.ctypes.data)
    if rc != 0:
        raise OracleError(f"orc_topk_bucketed returned {rc}")
    return out_idx[:, :K].copy(), out_val[:, :K].copy(), e


def quantize(val_list, bits: int, seed: int, bucket: int = 0):
    """QSGD per stream (bucket = 0: one scale per stream) or in buckets of
    ``bucket`` consecutive entries (§6).  Returns (codes list, flat scales,
    dequantized list); stream r's scales follow those of streams 0..r-1."""
    P = len(val_list)
    val_list = [np.ascontiguousarray(a, dtype=np.float32) for a in val_list]
    nnz = np.array([a.size for a in val_list], dtype=np.uint64)
    per_byte = 8 // bits
    q = [np.zeros(max((a.size + per_byte - 1) // per_byte, 1), dtype=np.uint8) for a in val_list]
    deq = [np.zeros(max(a.size, 1), dtype=np.float32) for a in val_list]
    scale = np.zeros(max(sum(scale_counts([a.size for a in val_list], bucket)), 1), dtype=np.float32)
    rc = lib().orc_quantize_bucketed(P, _ptr_table(val_list), nnz.ctypes.data, bits, bucket,
                                     seed & (2**64 - 1), _ptr_table(q), scale.ctypes.data,
                                     _ptr_table(deq))
    if rc != 0:
        raise OracleError(f"orc_quantize_bucketed returned {rc}")
    scale = scale[: sum(scale_counts([a.size for a in val_list], bucket))]
    nb = [(a.size + per_byte - 1) // per_byte for a in val_list]
    return ([qq[:n].copy() for qq, n in zip(q, nb)], scale,
            [d[: a.size].copy() for d, a in zip(deq, val_list)])


def dequantize(q: np.ndarray, scale, bits: int, n: int, bucket: int = 0) -> np.ndarray:
    """Values of n packed codes: one scale (bucket = 0) or scales[j // bucket]."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    out = np.zeros(max(n, 1), dtype=np.float32)
    if bucket:
        sc = np.ascontiguousarray(scale, dtype=np.float32)
        rc = lib().orc_dequantize_bucketed(_ptr(q), _ptr(sc), bits, bucket, n, out.ctypes.data)
    else:
        rc = lib().orc_dequantize(_ptr(q), ctypes.c_float(float(np.float32(scale))), bits, n,
                                  out.ctypes.data)
    if rc != 0:
        raise OracleError(f"orc_dequantize returned {rc}")
    return out[:n].copy()


def densify(idx: np.ndarray, val: np.ndarray, N: int) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.uint32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    out = np.zeros(N, dtype=np.float32)
    rc = lib().orc_densify(_ptr(idx), _ptr(val), idx.size, N, out.ctypes.data)
    if rc != 0:
        raise OracleError(f"orc_densify returned {rc}")
    return out


def topk_by_threshold(x: np.ndarray, k: int):
    """Exact per-row top-k with the same selection as topk (magnitude key =
    the float's bits without the sign, larger first; equal keys by smaller
    index; result in index order), found from the k-th largest key by a
    partition instead of a full sort -- for rows too long to sort quickly.
    §2.2 (top-k sparsification)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    P, N = x.shape
    out_idx = np.zeros((P, k), dtype=np.uint32)
    out_val = np.zeros((P, k), dtype=np.float32)
    if k == 0:
        return out_idx, out_val
    for r in range(P):
        key = x[r].view(np.uint32) & np.uint32(0x7FFFFFFF)
        kth = np.partition(key, N - k)[N - k]
        above = np.nonzero(key > kth)[0]
        ties = np.nonzero(key == kth)[0][: k - above.size]
        sel = np.sort(np.concatenate([above, ties])).astype(np.uint32)
        out_idx[r] = sel
        out_val[r] = x[r][sel]
    return out_idx, out_val
