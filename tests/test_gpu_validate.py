"""sparcml_validate_streams through the C ABI: well-formed streams pass;
crafted defects -- a duplicate, a descending pair, an index at or above hi,
an index below lo -- are reported as SPARCML_EUNSORTED with the first
offending stream and position (lowest stream, then lowest position).  The
expected verdicts come from the definition (strictly ascending, inside
[lo, hi)) checked with numpy on the host."""
import re

import numpy as np
import pytest

from paper_1802_08021_amd import inputs
from gpu_util import say, to_dev, torch_dev

pytestmark = pytest.mark.gpu


def host_first_bad(idx, lo, hi):
    for r, a in enumerate(idx):
        a = a.astype(np.int64)
        bad = (a < lo) | (a >= hi)
        bad[1:] |= a[1:] <= a[:-1]
        if bad.any():
            return r, int(np.nonzero(bad)[0][0])
    return None


def run(idx, lo, hi, label):
    from paper_1802_08021_amd import sparcml as S
    torch_dev()
    say(f"[validate] {label}: P={len(idx)} [{lo}, {hi})")
    ok, msg = S.validate_streams([to_dev(a if a.size else np.zeros(1, np.uint32))[: a.size] for a in idx], lo, hi)
    want = host_first_bad(idx, lo, hi)
    if want is None:
        assert ok, (label, msg)
    else:
        assert not ok, label
        m = re.search(r"stream (\d+), position (\d+)", msg)
        assert m and (int(m.group(1)), int(m.group(2))) == want, (label, msg, want)


def test_well_formed_streams_pass():
    rng = np.random.default_rng(950)
    idx = [inputs.uniform_subset(rng, 1 << 20, int(k)) for k in rng.integers(0, 5000, size=24)]
    run(idx, 0, 1 << 20, "uniform")
    run([np.zeros(0, np.uint32)] * 3, 0, 10, "empty")
    top = [np.array([2**32 - 3, 2**32 - 2, 2**32 - 1], np.uint32)]
    run(top, 2**32 - 5, 2**32, "top of the index space")


@pytest.mark.parametrize("defect", ["duplicate", "descending", "at_hi", "below_lo"])
def test_defects_are_reported(defect):
    rng = np.random.default_rng(951)
    lo, hi = 1000, 1 << 21
    idx = [(inputs.uniform_subset(rng, hi - lo, 3000).astype(np.int64) + lo).astype(np.uint32) for _ in range(12)]
    for r, pos in ((7, 1500), (3, 2999), (3, 10)):  # two defects in stream 3: the lower position counts
        a = idx[r].astype(np.int64)
        if defect == "duplicate":
            a[pos] = a[pos - 1]
        elif defect == "descending":
            a[pos], a[pos - 1] = a[pos - 1], a[pos]
        elif defect == "at_hi":
            a[pos] = hi + (pos % 3)
        else:
            a[pos] = lo - 1 - (pos % 5)
        idx[r] = a.astype(np.uint32)
    run(idx, lo, hi, defect)


def test_many_and_long_streams():
    rng = np.random.default_rng(952)
    idx = [inputs.uniform_subset(rng, 1 << 16, 50) for _ in range(300)]
    run(idx, 0, 1 << 16, "300 streams, well formed")
    idx[257] = idx[257].copy()
    idx[257][49] = idx[257][48]
    run(idx, 0, 1 << 16, "300 streams, stream 257 bad")
    long = [inputs.uniform_subset(rng, 1 << 26, 1 << 22)]
    run(long, 0, 1 << 26, "4M entries, well formed")
    long[0] = long[0].copy()
    long[0][-1] = long[0][-2]
    run(long, 0, 1 << 26, "4M entries, last bad")
