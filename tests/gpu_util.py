"""Helpers shared by the GPU parity tests: move seeded numpy inputs to the
device, call the HIP path through the C ABI binding, and compare with the
oracle at the bar the tests state (indices / nnz / decisions / codes
bit-exact; fp32 values within 1e-6 relative + 1e-7 absolute and, by
construction of the kernels, bitwise equal)."""
import sys

import numpy as np

RTOL, ATOL = 1e-6, 1e-7


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def torch_dev():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device")
    return torch, torch.device("cuda:0")


def to_dev(a: np.ndarray):
    torch, dev = torch_dev()
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def to_np(t, dtype=None) -> np.ndarray:
    a = t.detach().cpu().numpy()
    if dtype is not None:
        a = a.view(dtype)
    return a


def gpu_reduce(idx, val, N, delta, qbits=0, codes=None, scales=None, ws=None, rng=None):
    """HIP sparse reduce through the C ABI; ``rng`` = (lo, hi) calls the
    range entry point."""
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    ti = [to_dev(a) for a in idx]
    tv = None if qbits else [to_dev(v) for v in val]
    kw = dict(codes=codes, scales=scales, qbits=qbits, node_info=True, ws=ws)
    if rng is None:
        r = S.sparse_reduce(ti, tv, N, delta, **kw)
    else:
        r = S.sparse_reduce_range(ti, tv, N, rng[0], rng[1], delta, **kw)
    torch.cuda.synchronize()
    P = len(idx)
    return {
        "dense": r["dense"],
        "nnz": r["nnz"],
        "idx": None if r["dense"] else to_np(r["idx"], np.uint32).copy(),
        "val": to_np(r["val"]).copy(),
        "node_nnz": to_np(r["node_nnz"]).astype(np.uint64) if P > 1 else np.zeros(0, np.uint64),
        "node_dense": to_np(r["node_dense"]) if P > 1 else np.zeros(0, np.uint8),
    }


def assert_values(got: np.ndarray, want: np.ndarray, what: str = "values") -> None:
    assert got.shape == want.shape, (what, got.shape, want.shape)
    np.testing.assert_allclose(got, want, rtol=RTOL, atol=ATOL, err_msg=what)
    same = got.view(np.uint32) == want.view(np.uint32)
    if not same.all():
        bad = np.nonzero(~same)[0][:10]
        raise AssertionError(f"{what}: {int((~same).sum())} values differ bitwise, e.g. at {bad}: "
                             f"{got[bad]} vs {want[bad]}")


def assert_reduce_equal(g: dict, o: dict, label: str = "") -> None:
    assert g["dense"] == o["dense"], (label, "root representation")
    assert g["nnz"] == o["nnz"], (label, "root nnz", g["nnz"], o["nnz"])
    np.testing.assert_array_equal(g["node_dense"].astype(np.uint8), o["node_dense"].astype(np.uint8),
                                  err_msg=f"{label} node decisions")
    np.testing.assert_array_equal(g["node_nnz"], o["node_nnz"].astype(np.uint64),
                                  err_msg=f"{label} node nnz")
    if g["dense"]:
        assert_values(g["val"], o["val"], f"{label} dense root")
    else:
        np.testing.assert_array_equal(g["idx"], o["idx"], err_msg=f"{label} root indices")
        assert_values(g["val"], o["val"], f"{label} sparse root values")
