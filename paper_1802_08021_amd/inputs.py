"""Seeded synthetic inputs shaped like SparCML's gradient workloads.

This module only draws inputs; it holds none of the method's arithmetic
(no merging, summing, selection or quantization).  Both the HIP path's tests
and benchmark and the CPU oracle consume what it returns.

Recipes (stand-ins for the paper's synthetic micro-benchmarks, §8.1: "k
indices out of N selected uniformly at random at each node and assigned a
random value", and for the top-k densities of its DNN runs, §8.3-8.4):

  c1  P=4,   N=2^16, k=64          uniform sorted indices, N(0,1) values, delta 0.5
  c2  P=16,  N=2^20, k=1024        uniform indices, Laplace(0,1e-3) values, delta 0.25
  c3  P=32,  N=2^24, k=N//1000     dense Laplace(0,1e-3) rows, 1% of coordinates
                                   (drawn per rank) scaled by 100; top-k then reduce,
                                   delta 0.25
  c4  P=64,  N=2^26, k=N//200      Zipf(1.1) draws with replacement, values > N
                                   rejected, mapped through one seeded pseudorandom
                                   bijection of [0,N) shared by all ranks, kept in
                                   first-occurrence order until k distinct; N(0,1)
                                   values, delta 0.1
  c5  P=128, N=2^27, k=N//100      uniform indices, Laplace(0,1e-3) values, QSGD 4-bit
                                   with per-rank L2 scale, delta 0.1

Every rank's generator is numpy PCG64 seeded by SeedSequence([BASE, seed, cfg,
rank]) with BASE = 20180222; ``scale_log2`` shrinks N (and k in proportion)
for tests while keeping P and the value distributions.
"""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor
from dataclasses import dataclass

import numpy as np

BASE = 20180222


@dataclass(frozen=True)
class Config:
    name: str
    cfg: int
    P: int
    N: int
    k: int
    delta: float
    kind: str        # "uniform", "topk", "zipf"
    values: str      # "normal", "laplace"
    qbits: int = 0   # QSGD bits for the values (0 = fp32)


def _k_of(cfg: int, N: int) -> int:
    return {1: 64 * N // 65536, 2: 1024 * N // 2**20, 3: N // 1000, 4: N // 200, 5: N // 100}[cfg]


def config(cfg: int, scale_log2: int = 0, N: int | None = None) -> Config:
    """Config ``cfg`` (1..5) at full size, or with N shrunk by 2^scale_log2
    (or set explicitly); k follows N with the config's density, at least 1."""
    base = {
        1: (4, 2**16, 0.5, "uniform", "normal", 0),
        2: (16, 2**20, 0.25, "uniform", "laplace", 0),
        3: (32, 2**24, 0.25, "topk", "laplace", 0),
        4: (64, 2**26, 0.1, "zipf", "normal", 0),
        5: (128, 2**27, 0.1, "uniform", "laplace", 4),
    }[cfg]
    P, Nfull, delta, kind, values, qbits = base
    n = int(N) if N is not None else Nfull >> scale_log2
    k = max(1, _k_of(cfg, n))
    return Config(f"c{cfg}", cfg, P, n, k, delta, kind, values, qbits)


def rng_for(seed: int, cfg: int, rank: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([BASE, seed, cfg, rank])))


def quant_seed(seed: int, cfg: int) -> int:
    """Seed handed to the stochastic quantizer (its own counter-based RNG)."""
    return (BASE * 1000 + cfg + (seed << 40)) & (2**64 - 1)


def laplace(rng: np.random.Generator, b: float, n: int) -> np.ndarray:
    """Laplace(0, b) by inverse CDF, as fp32, never -0.0."""
    u = rng.random(n) - 0.5
    a = np.minimum(2.0 * np.abs(u), 1.0 - 2.0**-53)
    x = (-b) * np.sign(u) * np.log1p(-a)
    return (x.astype(np.float32) + np.float32(0.0))


def normal(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.standard_normal(n, dtype=np.float32) + np.float32(0.0)


def uniform_subset(rng: np.random.Generator, N: int, k: int) -> np.ndarray:
    """Uniformly random k-subset of [0, N), sorted ascending, uint32.

    Draws with replacement and deduplicates (every m-subset is then equally
    likely), then keeps a uniform k-subset of the distinct values."""
    if k > N:
        raise ValueError("k > N")
    if k == 0:
        return np.zeros(0, dtype=np.uint32)
    if 8 * k > N:
        return np.sort(rng.permutation(N)[:k]).astype(np.uint32)
    got = np.zeros(0, dtype=np.int64)
    while got.size < k:
        need = k - got.size
        draw = rng.integers(0, N, size=need + 4 * int(np.sqrt(need)) + 32, dtype=np.int64)
        got = np.unique(np.concatenate([got, draw]))
    if got.size > k:
        keep = np.sort(rng.choice(got.size, size=k, replace=False))
        got = got[keep]
    return got.astype(np.uint32)


def _mix_rounds(seed: int, cfg: int):
    r = rng_for(seed, cfg, 0x7FFF_0000)
    return [(int(r.integers(0, 2**62)) | 1, int(r.integers(0, 2**62))) for _ in range(4)]


def bijection(x: np.ndarray, N: int, rounds) -> np.ndarray:
    """Seeded pseudorandom bijection of [0, N): keyed odd-multiply / add /
    xor-shift rounds on ceil(log2 N) bits, cycle-walked back into [0, N)."""
    b = max(1, int(np.ceil(np.log2(N))))
    mask = np.uint64((1 << b) - 1)
    sh = np.uint64(max(1, b // 2))

    def f(v):
        v = v.astype(np.uint64)
        for mul, add in rounds:
            v = (v * np.uint64(mul & ((1 << b) - 1) | 1) + np.uint64(add)) & mask
            v = v ^ (v >> sh)
        return v

    y = f(x)
    bad = y >= np.uint64(N)
    while bad.any():
        y[bad] = f(y[bad])
        bad = y >= np.uint64(N)
    return y


def _zipf_indices(rng, N: int, k: int, rounds) -> np.ndarray:
    """First k distinct values of Zipf(1.1) draws (<= N) mapped through the
    shared bijection; returned sorted ascending as uint32."""
    if k > N:
        raise ValueError("k > N")
    draws = np.zeros(0, dtype=np.int64)
    batch = max(4 * k, 4096)
    while True:
        z = rng.zipf(1.1, size=batch)
        draws = np.concatenate([draws, z[z <= N]])
        uniq, first = np.unique(draws, return_index=True)
        if uniq.size >= k:
            break
        if uniq.size == N:
            break
    order = np.argsort(first, kind="stable")[:k]
    vals = uniq[order] - 1
    mapped = bijection(vals.astype(np.uint64), N, rounds)
    return np.sort(mapped).astype(np.uint32)


def _rank_job(args):
    c, seed, r = args
    rng = rng_for(seed, c.cfg, r)
    if c.kind == "topk":
        x = laplace(rng, 1e-3, c.N)
        o = uniform_subset(rng, c.N, c.N // 100)
        x[o] = x[o] * np.float32(100.0)
        return x
    if c.kind == "zipf":
        idx = _zipf_indices(rng, c.N, c.k, _mix_rounds(seed, c.cfg))
    else:
        idx = uniform_subset(rng, c.N, c.k)
    vals = normal(rng, idx.size) if c.values == "normal" else laplace(rng, 1e-3, idx.size)
    return idx, vals


def _map(jobs, workers):
    if workers <= 1 or len(jobs) <= 1:
        return [_rank_job(j) for j in jobs]
    import multiprocessing as mp
    with ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("fork")) as ex:
        return list(ex.map(_rank_job, jobs))


def default_workers() -> int:
    return max(1, min(16, (os.cpu_count() or 1)))


def generate(c: Config, seed: int = 0, workers: int | None = None):
    """Inputs of config ``c``.

    kind "topk": returns {"x": fp32[P, N]}.
    otherwise:   returns {"idx": [uint32 sorted], "val": [fp32]} per rank.
    """
    workers = default_workers() if workers is None else workers
    jobs = [(c, seed, r) for r in range(c.P)]
    if c.kind == "topk":
        rows = _map(jobs, workers if c.N >= 2**20 else 1)
        return {"x": np.stack(rows)}
    out = _map(jobs, workers if c.P * c.k >= 2**18 else 1)
    return {"idx": [o[0] for o in out], "val": [o[1] for o in out]}


# ---------------------------------------------------------------------------
# Hand-shaped streams for edge cases (tests only need these shapes; no
# arithmetic of the method lives here).

def streams_from_sets(sets, N: int, seed: int = 0, dist: str = "normal"):
    """Streams whose index sets are the given iterables; random values."""
    rng = rng_for(seed, 99, 0)
    idx, val = [], []
    for s in sets:
        a = np.unique(np.asarray(list(s), dtype=np.int64)).astype(np.uint32)
        if a.size and int(a[-1]) >= N:
            raise ValueError("index out of range")
        idx.append(a)
        val.append(normal(rng, a.size) if dist == "normal" else laplace(rng, 1e-3, a.size))
    return idx, val
