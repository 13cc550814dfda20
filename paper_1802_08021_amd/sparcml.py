"""Python binding of libsparcml.so (the gfx950 SparCML C ABI, include/sparcml.h).

Argument marshalling only: torch tensors supply device memory and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no fallback path -- if the library is missing or the
device is not usable, calls raise.

Index tensors are int32 holding the uint32 bit patterns of the ABI.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libsparcml.so")

OK, EINVAL, ECAPACITY, EWORKSPACE, EUNSORTED, EHIP = 0, -1, -2, -3, -4, -5
OP_TOPK, OP_QUANTIZE, OP_REDUCE, OP_DENSIFY, OP_QUANTIZE_BUCKETED, OP_CONCAT, OP_VALIDATE = 1, 2, 3, 4, 5, 6, 7


class Stream(ctypes.Structure):
    """Mirror of ``sparcml_stream``."""
    _fields_ = [
        ("idx", ctypes.c_void_p),
        ("val", ctypes.c_void_p),
        ("qval", ctypes.c_void_p),
        ("qscale", ctypes.c_void_p),
        ("nnz", ctypes.c_uint64),
        ("is_dense", ctypes.c_uint32),
        ("qbits", ctypes.c_uint32),
    ]


class SparcmlError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} ({status}): {last_error()}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsparcml.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_1802_08021_amd.build` "
            "(there is no CPU fallback)")
    L = ctypes.CDLL(LIB_PATH)
    vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
    L.sparcml_workspace_size.argtypes = [i32, i32, u64, u64, ctypes.c_double, ctypes.POINTER(ctypes.c_size_t)]
    L.sparcml_workspace_size.restype = i32
    L.sparcml_topk_sparsify.argtypes = [i32, vp, u64, u64, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparcml_topk_sparsify.restype = i32
    L.sparcml_topk_bucketed.argtypes = [i32, vp, vp, u64, ctypes.c_float, u64, u64, vp, vp, vp]
    L.sparcml_topk_bucketed.restype = i32
    L.sparcml_topk_bucketed_count.argtypes = [u64, u64, u64]
    L.sparcml_topk_bucketed_count.restype = u64
    L.sparcml_quantize.argtypes = [i32, ctypes.POINTER(Stream), i32, u64, vp, vp, vp, vp,
                                   ctypes.c_size_t, vp]
    L.sparcml_quantize.restype = i32
    L.sparcml_quantize_bucketed.argtypes = [i32, ctypes.POINTER(Stream), i32, u64, u64, vp, vp, vp, vp,
                                            ctypes.c_size_t, vp]
    L.sparcml_quantize_bucketed.restype = i32
    L.sparcml_sparse_reduce.argtypes = [i32, ctypes.POINTER(Stream), u64, ctypes.c_double,
                                        ctypes.POINTER(Stream), vp, vp, vp, ctypes.c_size_t, vp]
    L.sparcml_sparse_reduce.restype = i32
    L.sparcml_sparse_reduce_range.argtypes = [i32, ctypes.POINTER(Stream), u64, u64, u64, ctypes.c_double,
                                              ctypes.POINTER(Stream), vp, vp, vp, ctypes.c_size_t, vp]
    L.sparcml_sparse_reduce_range.restype = i32
    L.sparcml_sparse_reduce_async.argtypes = [i32, ctypes.POINTER(Stream), u64, u64, u64, ctypes.c_double,
                                              ctypes.POINTER(Stream), vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.sparcml_sparse_reduce_async.restype = i32
    L.sparcml_sparse_reduce_async_noalloc.argtypes = [i32, ctypes.POINTER(Stream), u64, u64, u64,
                                                      ctypes.c_double, ctypes.POINTER(Stream), vp, vp, vp, vp]
    L.sparcml_sparse_reduce_async_noalloc.restype = i32
    L.sparcml_concat.argtypes = [i32, ctypes.POINTER(Stream), ctypes.POINTER(u64), u64, ctypes.c_double, u64,
                                 ctypes.POINTER(Stream), vp, ctypes.c_size_t, vp]
    L.sparcml_concat.restype = i32
    L.sparcml_validate_streams.argtypes = [i32, ctypes.POINTER(Stream), u64, u64, vp, ctypes.c_size_t, vp]
    L.sparcml_validate_streams.restype = i32
    L.sparcml_split_bounds.argtypes = [i32, u64, ctypes.POINTER(u64)]
    L.sparcml_split_bounds.restype = i32
    L.sparcml_densify.argtypes = [ctypes.POINTER(Stream), u64, vp, vp]
    L.sparcml_densify.restype = i32
    L.sparcml_timing_enable.argtypes = [i32]
    L.sparcml_timing_enable.restype = i32
    L.sparcml_timing_read.argtypes = [i32, ctypes.POINTER(ctypes.c_float)]
    L.sparcml_timing_read.restype = i32
    L.sparcml_strerror.argtypes = [i32]
    L.sparcml_strerror.restype = ctypes.c_char_p
    L.sparcml_last_error.argtypes = []
    L.sparcml_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


TIMER_REDUCE_PASS, TIMER_REDUCE_WRITE, TIMER_REDUCE_SLOW = 0, 1, 2
TIMER_QUANT_NORM, TIMER_QUANT_CODES, TIMER_TOPK_SELECT, TIMER_TOPK_WRITE, TIMER_DENSIFY = 3, 4, 5, 6, 7
TIMER_CONCAT, TIMER_TOPK_BUCKETED, TIMER_REDUCE_MERGE = 8, 9, 10


def timing_enable(on: bool) -> None:
    lib().sparcml_timing_enable(1 if on else 0)


def timing_read(group: int):
    """Mean duration (ms) of a kernel group's launches since timing was
    enabled, or None."""
    ms = ctypes.c_float(0.0)
    rc = lib().sparcml_timing_read(group, ctypes.byref(ms))
    return float(ms.value) if rc == OK else None


def strerror(status: int) -> str:
    return lib().sparcml_strerror(status).decode()


def last_error() -> str:
    return lib().sparcml_last_error().decode()


def _check(rc: int, where: str) -> None:
    if rc != OK:
        raise SparcmlError(rc, where)


def workspace_size(op: int, P: int, N: int, max_nnz: int, delta: float = 1.0) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().sparcml_workspace_size(op, P, N, max_nnz, float(delta), ctypes.byref(n)),
           "sparcml_workspace_size")
    return int(n.value)


# ---------------------------------------------------------------------------
# torch-facing helpers (device memory and streams only)

def _torch():
    import torch
    return torch


def _stream_ptr(device) -> int:
    torch = _torch()
    return int(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t) -> int:
    return int(t.data_ptr()) if t is not None and t.numel() else 0


def _require_cuda(t, name: str):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def alloc_workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def topk_sparsify(x, k: int, residual=None, ws=None):
    """Per-row top-k by magnitude of x[P, N] (fp32).  residual: None, "inplace"
    (x itself becomes the residual) or a [P, N] fp32 tensor.
    Returns (idx int32 [P, k], val fp32 [P, k])."""
    torch = _torch()
    _require_cuda(x, "x")
    if x.dtype != torch.float32 or x.dim() != 2:
        raise ValueError("x must be a 2-D float32 tensor")
    P, N = x.shape
    idx = torch.empty((P, max(k, 1)), dtype=torch.int32, device=x.device)
    val = torch.empty((P, max(k, 1)), dtype=torch.float32, device=x.device)
    res_ptr = 0
    if isinstance(residual, str):
        if residual != "inplace":
            raise ValueError("residual must be None, 'inplace' or a tensor")
        res_ptr = _ptr(x)
    elif residual is not None:
        _require_cuda(residual, "residual")
        res_ptr = _ptr(residual)
    nbytes = workspace_size(OP_TOPK, P, N, k)
    if ws is None or ws.numel() < nbytes:
        ws = alloc_workspace(nbytes, x.device)
    _check(lib().sparcml_topk_sparsify(P, _ptr(x), N, k, _ptr(idx), _ptr(val), res_ptr,
                                        _ptr(ws), ws.numel(), _stream_ptr(x.device)),
           "sparcml_topk_sparsify")
    return idx[:, :k], val[:, :k]


class TopkBucketedCall:
    """Repeated bucketed top-k with error feedback (§8.4, Alg. 1) of fixed
    device rows: eps [P, N] is updated in place; idx / val [P, K]."""

    def __init__(self, eps, grad, alpha: float, bucket: int, kb: int):
        torch = _torch()
        _require_cuda(eps, "eps")
        if eps.dim() != 2 or not eps.is_contiguous() or eps.dtype != torch.float32:
            raise ValueError("eps must be a contiguous fp32 [P, N] tensor")
        if grad is not None and (grad.shape != eps.shape or not grad.is_contiguous()
                                 or grad.dtype != torch.float32):
            raise ValueError("grad must be a contiguous fp32 tensor shaped like eps")
        self.P, self.N = eps.shape
        self.eps, self.grad = eps, grad
        self.alpha, self.bucket, self.kb = float(alpha), bucket, kb
        self.K = int(lib().sparcml_topk_bucketed_count(self.N, bucket, kb))
        self.idx = torch.empty((self.P, max(self.K, 1)), dtype=torch.int32, device=eps.device)
        self.val = torch.empty((self.P, max(self.K, 1)), dtype=torch.float32, device=eps.device)

    def run(self) -> None:
        _check(lib().sparcml_topk_bucketed(self.P, _ptr(self.grad), _ptr(self.eps), self.N, self.alpha,
                                           self.bucket, self.kb, _ptr(self.idx), _ptr(self.val),
                                           _stream_ptr(self.eps.device)), "sparcml_topk_bucketed")


def topk_bucketed(eps, grad, alpha: float, bucket: int, kb: int):
    """acc = eps + alpha * grad; the kb largest magnitudes of every bucket of
    ``bucket`` coordinates; eps <- acc with them zeroed (in place).  Returns
    (idx [P, K] int32, val [P, K] fp32)."""
    c = TopkBucketedCall(eps, grad, alpha, bucket, kb)
    c.run()
    return c.idx[:, : c.K], c.val[:, : c.K]


def quantize(vals, bits: int, seed: int, want_deq: bool = False, ws=None):
    """QSGD of each fp32 tensor in ``vals``.  Returns (codes list of uint8
    tensors, scales fp32 [P], dequantized list or None)."""
    return _quantize(vals, bits, seed, want_deq, ws, 0)


def quantize_bucketed(vals, bits: int, bucket: int, seed: int, want_deq: bool = False, ws=None):
    """QSGD in buckets of ``bucket`` entries (§6).  Returns (codes list,
    flat scales fp32 -- stream r's ceil(n_r / bucket) after those of streams
    0..r-1 --, dequantized list or None)."""
    return _quantize(vals, bits, seed, want_deq, ws, bucket)


def _quantize(vals, bits, seed, want_deq, ws, bucket):
    torch = _torch()
    P = len(vals)
    dev = vals[0].device
    per = 8 // bits
    arr = (Stream * P)()
    codes, deqs = [], []
    for r, v in enumerate(vals):
        _require_cuda(v, f"vals[{r}]")
        n = v.numel()
        arr[r] = Stream(None, _ptr(v), None, None, n, 0, 0)
        codes.append(torch.empty(max((n + per - 1) // per, 1), dtype=torch.uint8, device=dev))
        if want_deq:
            deqs.append(torch.empty(max(n, 1), dtype=torch.float32, device=dev))
    qptr = (ctypes.c_void_p * P)(*[_ptr(c) for c in codes])
    dptr = (ctypes.c_void_p * P)(*[_ptr(d) for d in deqs]) if want_deq else None
    dp = ctypes.cast(dptr, ctypes.c_void_p) if dptr else None
    if bucket:
        nscale = sum((v.numel() + bucket - 1) // bucket for v in vals)
        scale = torch.empty(max(nscale, 1), dtype=torch.float32, device=dev)
        nbytes = workspace_size(OP_QUANTIZE_BUCKETED, P, 1, 0)
    else:
        nscale = P
        scale = torch.empty(P, dtype=torch.float32, device=dev)
        nbytes = workspace_size(OP_QUANTIZE, P, 1, max(v.numel() for v in vals))
    if ws is None or ws.numel() < nbytes:
        ws = alloc_workspace(nbytes, dev)
    if bucket:
        _check(lib().sparcml_quantize_bucketed(P, arr, bits, bucket, seed & (2**64 - 1),
                                               ctypes.cast(qptr, ctypes.c_void_p), _ptr(scale), dp,
                                               _ptr(ws), ws.numel(), _stream_ptr(dev)),
               "sparcml_quantize_bucketed")
    else:
        _check(lib().sparcml_quantize(P, arr, bits, seed & (2**64 - 1), ctypes.cast(qptr, ctypes.c_void_p),
                                      _ptr(scale), dp, _ptr(ws), ws.numel(), _stream_ptr(dev)),
               "sparcml_quantize")
    nb = [(v.numel() + per - 1) // per for v in vals]
    return ([c[:m] for c, m in zip(codes, nb)], scale[:nscale],
            [d[: v.numel()] for d, v in zip(deqs, vals)] if want_deq else None)


def make_streams(idx, vals=None, codes=None, scales=None, qbits: int = 0):
    """Descriptor array for P sparse streams (fp32 values or QSGD codes)."""
    P = len(idx)
    arr = (Stream * P)()
    for r in range(P):
        _require_cuda(idx[r], f"idx[{r}]")
        n = idx[r].numel()
        if qbits:
            arr[r] = Stream(_ptr(idx[r]), None, _ptr(codes[r]), int(scales[r].data_ptr()), n, 0, qbits)
        else:
            arr[r] = Stream(_ptr(idx[r]), _ptr(vals[r]), None, None, n, 0, 0)
    return arr


def sparse_reduce(idx, vals, N: int, delta: float, codes=None, scales=None, qbits: int = 0,
                  node_info: bool = False, ws=None, out_idx=None, out_val=None):
    """Sum of P sparse streams in recursive-doubling order with the dense
    switch.  ``scales`` is a device fp32 tensor [P] (one scale per stream)
    when ``qbits`` != 0.  Returns dict(idx, val, nnz, dense, node_nnz,
    node_dense); ``idx`` is None for a dense root."""
    return _reduce(idx, vals, N, None, delta, codes, scales, qbits, node_info, ws, out_idx, out_val)


def sparse_reduce_range(idx, vals, N: int, lo: int, hi: int, delta: float, codes=None, scales=None,
                        qbits: int = 0, node_info: bool = False, ws=None, out_idx=None, out_val=None):
    """One share of the split phase: the sum of P streams whose indices lie
    in [lo, hi), reduced as a vector of hi - lo (threshold floor(delta *
    (hi - lo))).  A dense root's ``val`` holds hi - lo values (index lo + i
    at i); a sparse root's ``idx`` holds absolute indices."""
    return _reduce(idx, vals, N, (lo, hi), delta, codes, scales, qbits, node_info, ws, out_idx, out_val)


def _reduce(idx, vals, N, rng, delta, codes, scales, qbits, node_info, ws, out_idx, out_val):
    torch = _torch()
    P = len(idx)
    dev = idx[0].device
    if qbits:
        scale_views = [scales[r: r + 1] for r in range(P)]
        arr = make_streams(idx, codes=codes, scales=scale_views, qbits=qbits)
    else:
        arr = make_streams(idx, vals)
    nnz = [t.numel() for t in idx]
    R = N if rng is None else rng[1] - rng[0]
    thr = int(float(delta) * float(R) // 1)
    cap = max(1, min(thr, sum(nnz)) if P > 1 else max(nnz[0], 1))
    if out_idx is None:
        out_idx = torch.empty(cap, dtype=torch.int32, device=dev)
    if out_val is None:
        out_val = torch.empty(R, dtype=torch.float32, device=dev)
    out = Stream(_ptr(out_idx), _ptr(out_val), None, None, out_idx.numel(), 0, 0)
    node_nnz = node_dense = None
    if node_info and P > 1:
        node_nnz = torch.empty(P - 1, dtype=torch.int64, device=dev)
        node_dense = torch.empty(P - 1, dtype=torch.uint8, device=dev)
    nbytes = workspace_size(OP_REDUCE, P, R, min(max(nnz), R), delta)
    if ws is None or ws.numel() < nbytes:
        ws = alloc_workspace(nbytes, dev)
    if rng is None:
        rc = lib().sparcml_sparse_reduce(P, arr, N, float(delta), ctypes.byref(out), _ptr(node_nnz),
                                         _ptr(node_dense), _ptr(ws), ws.numel(), _stream_ptr(dev))
        _check(rc, "sparcml_sparse_reduce")
    else:
        rc = lib().sparcml_sparse_reduce_range(P, arr, N, rng[0], rng[1], float(delta), ctypes.byref(out),
                                               _ptr(node_nnz), _ptr(node_dense), _ptr(ws), ws.numel(),
                                               _stream_ptr(dev))
        _check(rc, "sparcml_sparse_reduce_range")
    n = int(out.nnz)
    dense = bool(out.is_dense)
    return {
        "idx": None if dense else out_idx[:n],
        "val": out_val if dense else out_val[:n],
        "nnz": n,
        "dense": dense,
        "node_nnz": node_nnz,
        "node_dense": node_dense,
    }


class ConcatCall:
    """Repeated concatenation of P parts with disjoint index ranges (the
    gathered shares of the split-allgather allreduce) into fixed outputs.
    ``parts``: dicts with ``idx`` (device int32 tensor, or None for a dense
    part) and ``val`` (fp32) or ``codes`` + ``scales`` (QSGD, ``qbits``)."""

    def __init__(self, parts, bounds, N: int, delta: float, qbits: int = 0, bucket: int = 0):
        torch = _torch()
        self.P = len(parts)
        self.N, self.delta, self.bucket = N, float(delta), bucket
        self.dev = None
        self.arr = (Stream * self.P)()
        total = 0
        for p, part in enumerate(parts):
            n = bounds[p + 1] - bounds[p] if part["idx"] is None else part["idx"].numel()
            ref = part["codes"] if qbits else part["val"]
            _require_cuda(ref, f"parts[{p}]")
            self.dev = ref.device
            self.arr[p] = Stream(None if part["idx"] is None else _ptr(part["idx"]),
                                 None if qbits else _ptr(part["val"]),
                                 _ptr(part["codes"]) if qbits else None,
                                 _ptr(part["scales"]) if qbits else None,
                                 n, 1 if part["idx"] is None else 0, qbits)
            total += 0 if part["idx"] is None else n
        self.bounds = (ctypes.c_uint64 * (self.P + 1))(*[int(b) for b in bounds])
        self.out_idx = torch.empty(max(total, 1), dtype=torch.int32, device=self.dev)
        self.out_val = torch.empty(N, dtype=torch.float32, device=self.dev)
        self.ws = alloc_workspace(workspace_size(OP_CONCAT, self.P, N, 0), self.dev)
        self.out = Stream(_ptr(self.out_idx), _ptr(self.out_val), None, None, self.out_idx.numel(), 0, 0)
        self._keep = parts

    def run(self):
        """Returns (nnz, dense)."""
        self.out.nnz = self.out_idx.numel()
        _check(lib().sparcml_concat(self.P, self.arr, self.bounds, self.N, self.delta, self.bucket,
                                    ctypes.byref(self.out), _ptr(self.ws), self.ws.numel(),
                                    _stream_ptr(self.dev)), "sparcml_concat")
        return int(self.out.nnz), bool(self.out.is_dense)


def concat(parts, bounds, N: int, delta: float, qbits: int = 0, bucket: int = 0):
    """Concatenation of parts with disjoint index ranges (see ConcatCall).
    Returns dict(idx, val, nnz, dense); ``idx`` is None for a dense result."""
    c = ConcatCall(parts, bounds, N, delta, qbits, bucket)
    n, dense = c.run()
    return {"idx": None if dense else c.out_idx[:n], "val": c.out_val if dense else c.out_val[:n],
            "nnz": n, "dense": dense}


def validate_streams(idx, lo: int, hi: int):
    """Check that every index tensor (device int32 holding uint32 indices)
    ascends strictly inside [lo, hi).  Returns (True, "") or (False, the
    library's message naming the first offending stream and position)."""
    P = len(idx)
    arr = (Stream * P)()
    for r, t in enumerate(idx):
        _require_cuda(t, f"idx[{r}]")
        arr[r] = Stream(_ptr(t), None, None, None, t.numel(), 0, 0)
    ws = alloc_workspace(workspace_size(OP_VALIDATE, P, 1, 0), idx[0].device)
    rc = lib().sparcml_validate_streams(P, arr, lo, hi, _ptr(ws), ws.numel(), _stream_ptr(idx[0].device))
    if rc == EUNSORTED:
        return False, last_error()
    _check(rc, "sparcml_validate_streams")
    return True, ""


def split_bounds(P: int, N: int):
    """Bounds of the P index ranges of the split phase (App. A's rule:
    floor(N/P) indices per node, the rest to the last).  List of P + 1."""
    b = (ctypes.c_uint64 * (P + 1))()
    _check(lib().sparcml_split_bounds(P, N, b), "sparcml_split_bounds")
    return [int(v) for v in b]


def densify(idx, val, N: int, codes=None, scale=None, qbits: int = 0):
    """Dense fp32[N] of one sparse stream (values or QSGD codes)."""
    torch = _torch()
    dev = idx.device
    if qbits:
        s = Stream(_ptr(idx), None, _ptr(codes), int(scale.data_ptr()), idx.numel(), 0, qbits)
    else:
        s = Stream(_ptr(idx), _ptr(val), None, None, idx.numel(), 0, 0)
    out = torch.empty(N, dtype=torch.float32, device=dev)
    _check(lib().sparcml_densify(ctypes.byref(s), N, _ptr(out), _stream_ptr(dev)), "sparcml_densify")
    return out


# ---------------------------------------------------------------------------
# Prepared calls: descriptors and buffers built once, each run() is a single
# C-ABI call (used by the benchmark so that Python marshalling stays out of
# the timed loop).

class QuantizeCall:
    """Repeated QSGD of fixed device arrays into fixed code buffers
    (``bucket`` > 0: buckets of that many entries, flat scales)."""

    def __init__(self, vals, codes, scale, bits: int, seed: int, deq=None, bucket: int = 0):
        self.P = len(vals)
        self.bits, self.seed, self.bucket = bits, seed & (2**64 - 1), bucket
        self.dev = vals[0].device
        self.arr = (Stream * self.P)()
        for r, v in enumerate(vals):
            _require_cuda(v, f"vals[{r}]")
            self.arr[r] = Stream(None, _ptr(v), None, None, v.numel(), 0, 0)
        self.qptr = (ctypes.c_void_p * self.P)(*[_ptr(c) for c in codes])
        self.dptr = (ctypes.c_void_p * self.P)(*[_ptr(d) for d in deq]) if deq else None
        self.scale = scale
        if bucket:
            nbytes = workspace_size(OP_QUANTIZE_BUCKETED, self.P, 1, 0)
        else:
            nbytes = workspace_size(OP_QUANTIZE, self.P, 1, max(v.numel() for v in vals))
        self.ws = alloc_workspace(nbytes, self.dev)
        self._keep = (vals, codes, deq)

    def run(self) -> None:
        dp = ctypes.cast(self.dptr, ctypes.c_void_p) if self.dptr else None
        qp = ctypes.cast(self.qptr, ctypes.c_void_p)
        if self.bucket:
            _check(lib().sparcml_quantize_bucketed(
                self.P, self.arr, self.bits, self.bucket, self.seed, qp, _ptr(self.scale), dp,
                _ptr(self.ws), self.ws.numel(), _stream_ptr(self.dev)), "sparcml_quantize_bucketed")
        else:
            _check(lib().sparcml_quantize(
                self.P, self.arr, self.bits, self.seed, qp, _ptr(self.scale), dp,
                _ptr(self.ws), self.ws.numel(), _stream_ptr(self.dev)), "sparcml_quantize")


class ReduceCall:
    """Repeated sparse reduce of fixed device streams into fixed outputs."""

    def __init__(self, idx, N: int, delta: float, vals=None, codes=None, scales=None,
                 qbits: int = 0, node_info: bool = False, lo: int | None = None, hi: int | None = None):
        """``lo``, ``hi``: reduce the index range [lo, hi) (the split-phase
        share) instead of the whole vector."""
        self.P = len(idx)
        self.N, self.delta = N, float(delta)
        self.rng = None if lo is None else (int(lo), int(hi))
        R = N if self.rng is None else self.rng[1] - self.rng[0]
        self.dev = idx[0].device
        torch = _torch()
        if qbits:
            self.arr = make_streams(idx, codes=codes, scales=[scales[r: r + 1] for r in range(self.P)],
                                    qbits=qbits)
        else:
            self.arr = make_streams(idx, vals)
        nnz = [t.numel() for t in idx]
        thr = int(self.delta * float(R) // 1)
        cap = max(1, min(thr, sum(nnz)) if self.P > 1 else max(nnz[0], 1))
        self.out_idx = torch.empty(cap, dtype=torch.int32, device=self.dev)
        self.out_val = torch.empty(R, dtype=torch.float32, device=self.dev)
        self.node_nnz = self.node_dense = None
        if node_info and self.P > 1:
            self.node_nnz = torch.empty(self.P - 1, dtype=torch.int64, device=self.dev)
            self.node_dense = torch.empty(self.P - 1, dtype=torch.uint8, device=self.dev)
        nbytes = workspace_size(OP_REDUCE, self.P, R, min(max(nnz), R), self.delta)
        self.ws = alloc_workspace(nbytes, self.dev)
        self.out = Stream(_ptr(self.out_idx), _ptr(self.out_val), None, None, self.out_idx.numel(), 0, 0)
        self._keep = (idx, vals, codes, scales)

    def run_async(self):
        """Enqueue the reduction without waiting (capturable in a HIP
        graph); the root header lands in ``self.result`` (device int64 [2]:
        nnz, dense flag in the low word of the second)."""
        if not hasattr(self, "result"):
            torch = _torch()
            self.result = torch.zeros(2, dtype=torch.int64, device=self.dev)
        self.out.nnz = self.out_idx.numel()
        lo, hi = self.rng if self.rng is not None else (0, self.N)
        _check(lib().sparcml_sparse_reduce_async(
            self.P, self.arr, self.N, lo, hi, self.delta, ctypes.byref(self.out), _ptr(self.node_nnz),
            _ptr(self.node_dense), _ptr(self.result), _ptr(self.ws), self.ws.numel(),
            _stream_ptr(self.dev)), "sparcml_sparse_reduce_async")

    def run_async_noalloc(self):
        """run_async through the allocation-free entry point (the library's
        fixed scratch array instead of ``self.ws``)."""
        if not hasattr(self, "result"):
            torch = _torch()
            self.result = torch.zeros(2, dtype=torch.int64, device=self.dev)
        self.out.nnz = self.out_idx.numel()
        lo, hi = self.rng if self.rng is not None else (0, self.N)
        _check(lib().sparcml_sparse_reduce_async_noalloc(
            self.P, self.arr, self.N, lo, hi, self.delta, ctypes.byref(self.out), _ptr(self.node_nnz),
            _ptr(self.node_dense), _ptr(self.result), _stream_ptr(self.dev)),
            "sparcml_sparse_reduce_async_noalloc")

    def result_header(self):
        """(nnz, dense) from ``self.result`` (synchronizes); raises if the
        header's reserved word reports an incomplete reduction."""
        r = self.result.cpu()
        flags = (int(r[1]) >> 32) & 0xFFFFFFFF
        if flags & 2:
            raise RuntimeError("sparse_reduce_async: the merge path met streams that do not ascend; "
                               "the outputs are incomplete")
        if flags:
            raise RuntimeError("sparse_reduce_async: a segment of the merge path gave up waiting for its "
                               "predecessors' sizes; the outputs are incomplete")
        return int(r[0]), bool(int(r[1]) & 0xFFFFFFFF)

    def run(self):
        """Returns (nnz, dense)."""
        self.out.nnz = self.out_idx.numel()
        if self.rng is None:
            _check(lib().sparcml_sparse_reduce(
                self.P, self.arr, self.N, self.delta, ctypes.byref(self.out), _ptr(self.node_nnz),
                _ptr(self.node_dense), _ptr(self.ws), self.ws.numel(), _stream_ptr(self.dev)),
                "sparcml_sparse_reduce")
        else:
            _check(lib().sparcml_sparse_reduce_range(
                self.P, self.arr, self.N, self.rng[0], self.rng[1], self.delta, ctypes.byref(self.out),
                _ptr(self.node_nnz), _ptr(self.node_dense), _ptr(self.ws), self.ws.numel(),
                _stream_ptr(self.dev)), "sparcml_sparse_reduce_range")
        return int(self.out.nnz), bool(self.out.is_dense)


class TopkCall:
    """Repeated top-k of a fixed device matrix into fixed outputs."""

    def __init__(self, x, k: int, residual=None):
        torch = _torch()
        _require_cuda(x, "x")
        self.x, self.k = x, k
        self.P, self.N = x.shape
        self.idx = torch.empty((self.P, max(k, 1)), dtype=torch.int32, device=x.device)
        self.val = torch.empty((self.P, max(k, 1)), dtype=torch.float32, device=x.device)
        self.res_ptr = _ptr(residual) if residual is not None else 0
        nbytes = workspace_size(OP_TOPK, self.P, self.N, k)
        self.ws = alloc_workspace(nbytes, x.device)
        self._keep = residual

    def run(self) -> None:
        _check(lib().sparcml_topk_sparsify(
            self.P, _ptr(self.x), self.N, self.k, _ptr(self.idx), _ptr(self.val), self.res_ptr,
            _ptr(self.ws), self.ws.numel(), _stream_ptr(self.x.device)), "sparcml_topk_sparsify")
