"""Parity of the bucketed top-k with error feedback (§8.4, Alg. 1) through
the C ABI with the CPU oracle: selected indices bit-exact, selected values
and the updated error bitwise.  Cases span one- to 64-entry lanes (buckets
of 64..4096), kb from 1 to 64, ragged last buckets, rows whose length is not
a multiple of 4 (unaligned rows), ties at zero, no gradient, and the c3
shape (N = 2^24, buckets of 512, 4 per bucket)."""
import numpy as np
import pytest

import oracle
from paper_1802_08021_amd import inputs
from gpu_util import assert_values, say, to_dev, to_np, torch_dev

pytestmark = pytest.mark.gpu


def check(eps, grad, alpha, bucket, kb, label):
    from paper_1802_08021_amd import sparcml as S
    torch, dev = torch_dev()
    P, N = eps.shape
    say(f"[topk_buckets] {label}: P={P} N={N} B={bucket} kb={kb} alpha={alpha} grad={grad is not None}")
    oi, ov, oe = oracle.topk_bucketed(eps, grad, alpha, bucket, kb)
    te = to_dev(eps)
    tg = None if grad is None else to_dev(grad)
    gi, gv = S.topk_bucketed(te, tg, alpha, bucket, kb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(gi, np.uint32), oi, err_msg=f"{label} indices")
    assert_values(to_np(gv).ravel(), ov.ravel(), f"{label} values")
    assert_values(to_np(te).ravel(), oe.ravel(), f"{label} error")


@pytest.mark.parametrize("bucket", [64, 128, 256, 512, 1024, 2048, 4096])
def test_sizes_and_ragged_buckets(bucket):
    rng = np.random.default_rng(500 + bucket)
    for N in (1, 63, bucket - 1, bucket, bucket + 1, 3 * bucket + 5, 40001):
        for kb in sorted({1, 4, min(bucket, 64)}):
            P = 3
            eps = inputs.laplace(rng, 1.0, P * N).reshape(P, N)
            grad = inputs.normal(rng, P * N).reshape(P, N)
            check(eps, grad, 0.05, bucket, kb, f"N={N}")


def test_ties_no_gradient_and_alpha_zero():
    rng = np.random.default_rng(510)
    P, N = 4, 10000
    eps = np.zeros((P, N), np.float32)
    eps[:, ::7] = 1.0
    eps[:, ::11] = -1.0  # equal magnitudes everywhere: lowest index wins
    check(eps, None, 1.0, 512, 4, "ties, no gradient")
    grad = inputs.normal(rng, P * N).reshape(P, N)
    check(eps, grad, 0.0, 64, 8, "alpha 0")
    check(np.zeros((P, N), np.float32), None, 1.0, 256, 16, "all zero")


def test_c3_shape():
    """N = 2^24 rows, buckets of 512, 4 per bucket (the paper's setting):
    four rows checked in full against the oracle; 32 rows of 2^20 too."""
    rng = np.random.default_rng(511)
    c = inputs.config(3)
    for P, N in ((4, c.N), (c.P, 1 << 20)):
        eps = inputs.laplace(rng, 1e-3, P * N).reshape(P, N)
        grad = inputs.laplace(rng, 1e-3, P * N).reshape(P, N)
        check(eps, grad, 0.1, 512, 4, f"c3 shape P={P}")
