#!/usr/bin/env python3
"""Benchmark of the SparCML hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5]

A step is one pass of the hot path over one batch of synthetic input held
in HBM.  The headline workload is c5, the largest configuration: 128 ranks x
1,342,177 uniform indices of N = 2^27 with Laplace(0, 1e-3) values, QSGD
4-bit quantization (per-rank L2 scale, Philox) followed by the
recursive-doubling sparse reduce with fused dequantization and the dense
switch (delta = 0.1).  value = reduce input nnz per second of step time.

Besides the headline line the JSON carries:
  roofline      the dominant kernel's algorithmic bytes per launch over its
                average duration (HIP events on the launch stream, recorded
                by the library during the timed steps), against 8 TB/s;
                traffic = measured HBM bytes per launch from rocprofv3
                FETCH_SIZE/WRITE_SIZE runs (profiles/), or null when the
                kernel source changed since they were taken;
  cpu_baseline  one step of the workload run by the CPU oracle on the same
                host inputs: value on all usable host threads (the
                oracle's independent items spread over them, same bits as
                one thread), with the single-thread time beside it; every
                per_config entry carries the same as cpu_oracle;
  ms_per_step   the K timed steps, during which the library records HIP
                events around its kernels (the durations the roofline uses);
  ms_per_step_no_events  the same K steps just before, without those events;
  cold_ms_per_step  the step with the 256 MB Infinity Cache evicted first
                (median of 5);
  seeds         the step over seeds s..s+4 (fresh inputs): per-seed ms,
                median and quartiles;
  copy_ceiling  a plain 1 GiB device copy's bandwidth, the streaming ceiling;
  parts         the producer (QSGD or top-k) and the reduce apart: summed
                kernel time and input rate of each;
  per_config    the other configurations, each with ms_per_step from steps
                without the library's kernel events (at tens of microseconds
                per step their records are a visible share) and
                ms_per_step_with_kernel_events from the steps whose kernel
                durations are reported (c1..c4; c3 = top-k then reduce,
                with the top-k input elements per second), each timed
                after at least 0.3 s of warm-up steps, and the split-phase
                share of c4 and c5 (index range 0 of App. A's P-way
                partition, every rank's stream restricted to it: one node's
                reduction in the split-allgather allreduce), c4/p48: c4
                with 48 ranks (App. A's step in front), c3/bucketed: c3
                with Alg. 1's
                error feedback and 4 of every 512 coordinates selected
                (§8.4), and c5/dsar: one node's compute
                in DSAR with the QSGD dense stage (its share reduced, the
                dense share quantized 4-bit in buckets of 1024, all P
                gathered shares decoded into the full vector).

Only one GPU is used; --gpus above 1 exits with a message.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse-reduce input nnz/s + achieved HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c5", choices=["c1", "c2", "c3", "c4", "c5"])
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-per-config", action="store_true")
    p.add_argument("--configs", default=None,
                   help="comma-separated per-config workloads to run (others and the seed sweep skipped)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="only run a plain 1 GiB device copy (3 times): the reference for "
                        "scaling rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes")
    return p.parse_args()


def calibrate_copy(torch) -> int:
    x = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0").fill_(1.0)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    log("copied 1 GiB three times")
    return 0


def copy_ceiling(torch, reps=5):
    """A plain 1 GiB device copy (torch copy_): bytes read + written over its
    time, the bandwidth a streaming kernel can reach on this device."""
    x = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0").fill_(1.0)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        y.copy_(x)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / reps
    gbs = 2 * (1 << 30) / (ms * 1e-3) / 1e9
    del x, y
    return {"GB/s": gbs, "frac_of_peak": gbs / HBM_PEAK_GBS, "bytes": 2 << 30, "ms": ms}


def time_cold(w, n, torch):
    """Steps with the 256 MB Infinity Cache evicted first (a 512 MB buffer is
    written before each); median ms of the step alone."""
    flush = torch.empty(1 << 27, dtype=torch.float32, device="cuda:0")
    times = []
    for _ in range(n):
        flush.fill_(0.0)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record()
        w.step()
        end.record()
        torch.cuda.synchronize()
        times.append(start.elapsed_time(end))
    del flush
    return float(np.median(times))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def arena(arrays, dtype, torch, dev, align=64):
    """One device allocation holding every rank's array, each slice starting
    on a 256-byte boundary; returns (arena, per-rank views)."""
    offs, tot = [], 0
    for a in arrays:
        offs.append(tot)
        tot += (a.size + align - 1) // align * align
    host = np.zeros(max(tot, 1), dtype=arrays[0].dtype)
    for a, o in zip(arrays, offs):
        host[o: o + a.size] = a
    dev_arena = torch.from_numpy(host).to(dev)
    return dev_arena, [dev_arena[o: o + a.size] for a, o in zip(arrays, offs)]


def empty_arena(sizes, dtype, torch, dev, align=256):
    offs, tot = [], 0
    for n in sizes:
        offs.append(tot)
        tot += (max(n, 1) + align - 1) // align * align
    t = torch.empty(max(tot, 1), dtype=dtype, device=dev)
    return t, [t[o: o + n] for n, o in zip(sizes, offs)]


class Workload:
    """Device-resident inputs, prepared calls and byte accounting of one config."""

    def __init__(self, name, cfg, seed, torch, dev, share=None, bucketed=None, keep_host=False):
        """``share`` = (s, S): the s-th of S index ranges of the config's
        vector (App. A's partition: floor(N/S) indices each, the rest to the
        last), each rank's stream restricted to it (one node's work in the
        split phase of the large-data allreduce)."""
        from paper_1802_08021_amd import inputs
        from paper_1802_08021_amd import sparcml as S
        self.name, self.c = name, cfg
        self.seed, self.bucketed = seed, bucketed
        c = cfg
        t0 = time.time()
        d = inputs.generate(c, seed)
        log(f"{name}: generated inputs in {time.time() - t0:.1f}s")
        self.d_host = d if keep_host else None  # for the CPU oracle leg
        rng = {}
        self.R = c.N
        if share is not None:
            assert c.kind != "topk"
            lo, hi = S.split_bounds(share[1], c.N)[share[0]: share[0] + 2]  # App. A's partition
            keep = [(a >= lo) & (a < hi) for a in d["idx"]]
            d = {"idx": [a[m] for a, m in zip(d["idx"], keep)], "val": [v[m] for v, m in zip(d["val"], keep)]}
            rng = {"lo": lo, "hi": hi}
            self.R = hi - lo
            if keep_host:
                self.d_host = d
        self.groups = [S.TIMER_REDUCE_PASS, S.TIMER_REDUCE_SLOW, S.TIMER_REDUCE_WRITE, S.TIMER_REDUCE_MERGE]
        self.kernel_bytes = {}
        if c.kind == "topk" and bucketed:
            # Alg. 1 with §8.4's selection: acc = eps + alpha * grad, kb of
            # every bucket; eps starts at zero and carries over between steps
            B, kb = bucketed
            x = torch.from_numpy(d["x"]).to(dev)
            del d
            eps = torch.zeros_like(x)
            self.topk = S.TopkBucketedCall(eps, x, 0.1, B, kb)
            K = self.topk.K
            idx = [self.topk.idx[r, :K] for r in range(c.P)]
            vals = [self.topk.val[r, :K] for r in range(c.P)]
            self.nnz = c.P * K
            self.reduce = S.ReduceCall(idx, c.N, c.delta, vals=vals)
            self.groups += [S.TIMER_TOPK_BUCKETED]
            # grad read, eps read and written, K pairs written per rank
            self.kernel_bytes[S.TIMER_TOPK_BUCKETED] = c.P * c.N * 12 + c.P * K * 8
            self._steps = [self.topk.run, self.reduce.run_async]
            self.topk_step_bytes = self.kernel_bytes[S.TIMER_TOPK_BUCKETED]
            self._keep = (x, eps)
        elif c.kind == "topk":
            x = torch.from_numpy(d["x"]).to(dev)
            del d
            self.topk_step_bytes = c.P * c.N * 4 + c.P * c.k * 8
            self.topk = S.TopkCall(x, c.k)
            idx = [self.topk.idx[r] for r in range(c.P)]
            vals = [self.topk.val[r] for r in range(c.P)]
            self.nnz = c.P * c.k
            self.reduce = S.ReduceCall(idx, c.N, c.delta, vals=vals)
            self.groups += [S.TIMER_TOPK_SELECT, S.TIMER_TOPK_WRITE]
            # compulsory bytes: one read of x (the sampled histogram and the
            # gather pass), the k selected pairs written (from the gathered
            # entries); any re-read shows as lost bandwidth
            self.kernel_bytes[S.TIMER_TOPK_SELECT] = c.P * c.N * 4
            self.kernel_bytes[S.TIMER_TOPK_WRITE] = c.P * c.k * 8
            self._steps = [self.topk.run, self.reduce.run_async]
        else:
            self.nnz = sum(a.size for a in d["idx"])
            _, idx = arena([a.view(np.int32) for a in d["idx"]], None, torch, dev)
            if c.qbits:
                _, vals = arena(d["val"], None, torch, dev)
                per = 8 // c.qbits
                code_bytes = [(a.size + per - 1) // per for a in d["idx"]]
                _, codes = empty_arena(code_bytes, torch.uint8, torch, dev)
                scale = torch.empty(c.P, dtype=torch.float32, device=dev)
                self.quant = S.QuantizeCall(vals, codes, scale, c.qbits, inputs.quant_seed(seed, c.cfg))
                self.reduce = S.ReduceCall(idx, c.N, c.delta, codes=codes, scales=scale, qbits=c.qbits, **rng)
                self.groups += [S.TIMER_QUANT_NORM, S.TIMER_QUANT_CODES]
                cb = sum(code_bytes)
                self.kernel_bytes[S.TIMER_QUANT_NORM] = self.nnz * 4
                self.kernel_bytes[S.TIMER_QUANT_CODES] = self.nnz * 4 + cb
                self.in_bytes = self.nnz * 4 + cb
                self.quant_bytes = self.nnz * 4 + cb
                self._steps = [self.quant.run, self.reduce.run_async]
            else:
                _, vals = arena(d["val"], None, torch, dev)
                self.reduce = S.ReduceCall(idx, c.N, c.delta, vals=vals, **rng)
                self.in_bytes = self.nnz * 8
                self.quant_bytes = 0
                self._steps = [self.reduce.run_async]
        self.rng = rng
        d = None

    def step(self):
        """One step, enqueued without waiting; header() reads its root."""
        for f in self._steps:
            f()

    def header(self):
        return self.reduce.result_header()

    def finish_bytes(self, root_nnz, dense):
        """Algorithmic bytes once the root representation is known."""
        from paper_1802_08021_amd import sparcml as S
        c = self.c
        out_bytes = self.R * 4 if dense else root_nnz * 8
        if c.kind == "topk":
            red_in = self.nnz * 8
        else:
            red_in = self.in_bytes
        # first tile pass: reads the streams; a dense root is written there
        self.kernel_bytes[S.TIMER_REDUCE_PASS] = red_in + (self.R * 4 if dense else 0)
        if not dense:
            self.kernel_bytes[S.TIMER_REDUCE_WRITE] = red_in + out_bytes
        # small-data path: the streams read once, the root written once
        self.kernel_bytes[S.TIMER_REDUCE_MERGE] = red_in + out_bytes
        if c.kind == "topk":
            self.step_bytes = self.topk_step_bytes + red_in + out_bytes
        else:
            self.step_bytes = self.quant_bytes + red_in + out_bytes


class DsarWorkload:
    """One node's compute in the split-allgather allreduce with QSGD on the
    dense stage (DSAR, §5.3.2 and §6), on c5's streams in fp32: the node's
    share (index range 0 of App. A's P-way partition) reduced over the P ranks'
    sub-streams, the dense share quantized in buckets, and the P gathered
    quantized shares decoded into the full vector.  The other nodes' shares
    (their own work) are prepared once, untimed."""

    def __init__(self, name, cfg, seed, torch, dev, bits=4, bucket=1024, keep_host=False):
        from paper_1802_08021_amd import inputs
        from paper_1802_08021_amd import sparcml as S
        self.name, self.c = name, cfg
        c = cfg
        t0 = time.time()
        d = inputs.generate(c, seed)
        log(f"{name}: generated inputs in {time.time() - t0:.1f}s")
        P, N = c.P, c.N
        self.bits, self.bucket = bits, bucket
        b = S.split_bounds(P, N)  # App. A: floor(N/P) per node, the rest to the last
        self.bounds = b
        _, idx = arena([a.view(np.int32) for a in d["idx"]], None, torch, dev)
        _, vals = arena(d["val"], None, torch, dev)
        # sub-stream of rank r for share s: a slice of the sorted stream
        cuts = [np.searchsorted(a, b) for a in d["idx"]]
        per = 8 // bits
        codes, scales, keep = [], [], []
        self.nnz = 0
        for sh in range(P):
            si = [idx[r][int(cuts[r][sh]): int(cuts[r][sh + 1])] for r in range(P)]
            sv = [vals[r][int(cuts[r][sh]): int(cuts[r][sh + 1])] for r in range(P)]
            red = S.ReduceCall(si, N, c.delta, vals=sv, lo=b[sh], hi=b[sh + 1])
            R = b[sh + 1] - b[sh]
            cq = torch.empty((R + per - 1) // per, dtype=torch.uint8, device=dev)
            sc = torch.empty((R + bucket - 1) // bucket, dtype=torch.float32, device=dev)
            qc = S.QuantizeCall([red.out_val], [cq], sc, bits, inputs.quant_seed(seed, c.cfg) + sh,
                                bucket=bucket)
            if sh == 0:
                self.reduce, self.quant = red, qc
                self.nnz = sum(int(cuts[r][1] - cuts[r][0]) for r in range(P))
                self.R = R
            else:
                _, dense = red.run()
                assert dense, "a DSAR share is expected to be dense"
                qc.run()
                keep.append(red.out_val)
                red = qc = None
            codes.append(cq)
            scales.append(sc)
        torch.cuda.synchronize()
        parts = [{"idx": None, "codes": cq, "scales": sc} for cq, sc in zip(codes, scales)]
        self.concat = S.ConcatCall(parts, b, N, c.delta, qbits=bits, bucket=bucket)
        self._keep = (idx, vals, codes, scales)
        self.groups = [S.TIMER_REDUCE_PASS, S.TIMER_REDUCE_SLOW, S.TIMER_QUANT_CODES, S.TIMER_CONCAT]
        nsc = (N + bucket - 1) // bucket
        self.kernel_bytes = {
            S.TIMER_REDUCE_PASS: self.nnz * 8 + self.R * 4,
            S.TIMER_QUANT_CODES: self.R * 4 + self.R * bits // 8 + (self.R // bucket) * 4,
            S.TIMER_CONCAT: N * bits // 8 + nsc * 4 + N * 4,
        }
        self.step_bytes = sum(self.kernel_bytes.values())
        self.seed = seed
        self.d_host = d if keep_host else None
        self._steps = [self.reduce.run_async, self.quant.run, self._gather]
        self._last = None

    def step(self):
        for f in self._steps:
            f()

    def _gather(self):
        self._last = self.concat.run()  # decided on the host: (nnz, dense)

    def header(self):
        return self._last

    def finish_bytes(self, root_nnz, dense):
        pass


def time_steps(w, K, W, torch, warm_s=0.0):
    """W untimed steps (continued until warm_s seconds have passed, so that
    clocks have ramped after an idle gap), then K timed steps."""
    from paper_1802_08021_amd import sparcml as S
    t0 = time.perf_counter()
    done = 0
    while done < W or time.perf_counter() - t0 < warm_s:
        w.step()
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    # the same K steps without the library's kernel events (their records
    # are extra packets on the stream, visible at microsecond step times)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(K):
        w.step()
    end.record()
    torch.cuda.synchronize()
    ms_plain = start.elapsed_time(end) / K
    # the timed steps: kernel durations from the library's events around
    # every launch of these steps, read once afterwards
    S.timing_enable(True)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record()
    for _ in range(K):
        w.step()
    end.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - wall0) * 1e3 / K
    durs = {g: S.timing_read(g) for g in w.groups}
    S.timing_enable(False)
    ms = start.elapsed_time(end) / K
    nnz, dense = w.header()
    w.finish_bytes(nnz, dense)
    w.ms_plain = ms_plain
    return ms, wall, {g: v for g, v in durs.items() if v is not None}, nnz, dense


GROUP_NAMES = {0: "reduce_tiles", 1: "reduce_write", 2: "reduce_slow", 3: "qsgd_norm",
               4: "qsgd_codes", 5: "topk_select", 6: "topk_write", 7: "densify", 8: "concat",
               9: "topk_bucketed", 10: "reduce_merge"}


# the sources each kernel group is built from (a change of code in them
# invalidates its measured traffic)
GROUP_SOURCES = {
    "reduce_tiles": ("reduce.hip", "qsgd_device.h", "internal.h"),
    "reduce_write": ("reduce.hip", "qsgd_device.h", "internal.h"),
    "reduce_slow": ("reduce.hip", "qsgd_device.h", "internal.h"),
    "reduce_merge": ("merge.hip", "qsgd_device.h", "internal.h"),
    "qsgd_norm": ("quant.hip", "internal.h"),
    "qsgd_codes": ("quant.hip", "internal.h"),
    "topk_select": ("topk.hip", "internal.h"),
    "topk_write": ("topk.hip", "internal.h"),
    "topk_bucketed": ("topk_buckets.hip", "internal.h"),
    "concat": ("concat.hip", "qsgd_device.h", "internal.h"),
    "densify": ("densify.hip", "qsgd_device.h", "internal.h"),
}


def source_hash(group: str = "reduce_tiles") -> str:
    """sha256 of a kernel group's sources without comments and blank lines
    (a change of code, not of wording, invalidates measured traffic)."""
    h = hashlib.sha256()
    for f in GROUP_SOURCES[group]:
        with open(os.path.join(ROOT, "paper_1802_08021_amd", "csrc", f)) as fh:
            for line in fh:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def traffic_for(kernel: str, workload: str):
    """Measured HBM bytes per launch of a kernel group on a workload, from
    the committed rocprofv3 FETCH_SIZE/WRITE_SIZE runs (profiles/), only
    while the group's sources are unchanged since they were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    for e in t.get("entries", []):
        if e.get("kernel") == kernel and e.get("workload") == workload:
            if kernel in GROUP_SOURCES and e.get("source_sha256") == source_hash(kernel):
                return e.get("bytes_per_launch")
            return None
    return None


def oracle_threads() -> int:
    """Threads for the oracle's parallel leg: the CPUs this process may run
    on, capped by OMP_NUM_THREADS when that is set (the host share of one
    GPU)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(1, n)


def _mean_seconds(fn, min_s):
    """fn() repeated until min_s seconds have passed (at least once): mean."""
    reps, t0 = 0, time.perf_counter()
    while True:
        fn()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return dt / reps


def oracle_step_times(w, threads):
    """One step of workload ``w`` run by the CPU oracle on the workload's own
    host inputs, with the oracle's independent items (tree-level nodes,
    top-k rows, quantized streams) on 1 and on ``threads`` threads; the
    results are the same bits either way.  Where a single-thread step would
    take minutes (top-k over 32 rows of 2^24) only some rows are selected and
    the time is scaled to all P rows.  Returns (single_s, multi_s, sample)."""
    import oracle
    from paper_1802_08021_amd import inputs
    c, d = w.c, w.d_host
    if isinstance(w, DsarWorkload):
        return _oracle_dsar(w, threads)
    if c.kind == "topk":
        x = d["x"]
        P = x.shape[0]
        if w.bucketed:
            B, kb = w.bucketed

            def select(rows):
                return oracle.topk_bucketed(np.zeros_like(x[:rows]), x[:rows], 0.1, B, kb)[:2]
        else:
            def select(rows):
                return oracle.topk(x[:rows], c.k)[:2]
        one_rows = 1
        with oracle.threads(threads):
            t0 = time.perf_counter()
            idx, val = select(P)
            t_sel_multi = time.perf_counter() - t0
        with oracle.threads(1):
            t0 = time.perf_counter()
            select(one_rows)
            t_sel_one = (time.perf_counter() - t0) * P / one_rows
        il, vl = [idx[r] for r in range(P)], [val[r] for r in range(P)]
        times = []
        for th in (1, threads):
            with oracle.threads(th):
                times.append(_mean_seconds(lambda: oracle.sparse_reduce(il, vl, c.N, c.delta), 0.2))
        sample = (f"selection: all {P} rows on {threads} threads, {one_rows} row on one thread "
                  f"(scaled by {P}); reduce: the whole input")
        return t_sel_one + times[0], t_sel_multi + times[1], sample
    idx, val = d["idx"], d["val"]
    qseed = inputs.quant_seed(w.seed, c.cfg)
    lo, hi = w.rng.get("lo"), w.rng.get("hi")

    def step():
        deq = oracle.quantize(val, c.qbits, qseed)[2] if c.qbits else val
        if lo is None:
            oracle.sparse_reduce(idx, deq, c.N, c.delta)
        else:
            oracle.sparse_reduce_range(idx, deq, c.N, lo, hi, c.delta)
    times = []
    for th in (1, threads):
        with oracle.threads(th):
            times.append(_mean_seconds(step, 0.2))
    return times[0], times[1], "the whole input" + (", quantize + reduce" if c.qbits else "")


def _oracle_dsar(w, threads):
    """DSAR node step: share 0 reduced (fp32), quantized in buckets, and the
    P quantized shares decoded into the full vector.  The other P - 1 shares
    are stand-ins of the right sizes (random codes, unit scales): the decode
    does the same work for any codes."""
    import oracle
    from paper_1802_08021_amd import inputs
    c, d = w.c, w.d_host
    b = w.bounds
    P, N = c.P, c.N
    lo, hi = b[0], b[1]
    cut = [int(np.searchsorted(a, hi)) for a in d["idx"]]
    si = [a[:n] for a, n in zip(d["idx"], cut)]
    sv = [v[:n] for v, n in zip(d["val"], cut)]
    rng = np.random.default_rng(7)
    per = 8 // w.bits
    others = []
    for s in range(1, P):
        R = b[s + 1] - b[s]
        others.append({"idx": None, "qbits": w.bits, "bucket": w.bucket, "n": R,
                       "codes": rng.integers(0, 256, size=(R + per - 1) // per, dtype=np.uint8),
                       "scales": np.ones((R + w.bucket - 1) // w.bucket, np.float32)})
    qseed = inputs.quant_seed(w.seed, c.cfg)

    def step():
        red = oracle.sparse_reduce_range(si, sv, N, lo, hi, c.delta)
        q, sc, _ = oracle.quantize([red["val"]], w.bits, qseed, bucket=w.bucket)
        mine = {"idx": None, "qbits": w.bits, "bucket": w.bucket, "n": hi - lo, "codes": q[0], "scales": sc}
        oracle.concat([mine] + others, b, N, c.delta)
    times = []
    for th in (1, threads):
        with oracle.threads(th):
            times.append(_mean_seconds(step, 0.2))
    return times[0], times[1], (f"share [0, {hi}) reduced and quantized; the other {P - 1} shares' codes "
                                "random stand-ins of their sizes; the decode runs on one thread in both legs")


def oracle_leg(w, threads):
    """The CPU oracle's time for one step of ``w``, single-thread and on
    ``threads`` threads, as step times and input rates."""
    one, multi, sample = oracle_step_times(w, threads)
    return {"kind": "oracle", "threads": threads, "ms_per_step": multi * 1e3,
            "input_nnz_per_s": w.nnz / multi, "single_thread_ms_per_step": one * 1e3,
            "single_thread_input_nnz_per_s": w.nnz / one, "sample": sample}


def describe(c) -> str:
    q = f", QSGD {c.qbits}-bit" if c.qbits else ""
    kind = {"uniform": "uniform indices", "zipf": "Zipf(1.1) permuted indices",
            "topk": "top-k of dense Laplace rows"}[c.kind]
    return f"{c.name}: P={c.P}, N={c.N}, k={c.k}, {kind}{q}, delta={c.delta}"


def main() -> int:
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the reduction; runs on more than one GPU "
              "are not implemented (use --gpus 1).", file=sys.stderr)
        return 2
    import torch
    from paper_1802_08021_amd import inputs, sparcml as S
    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        return 2
    if args.calibrate_copy:
        return calibrate_copy(torch)
    S.lib()
    dev = torch.device("cuda:0")

    head_cfg = inputs.config(int(args.workload[1]))
    w = Workload(args.workload, head_cfg, args.seed, torch, dev, keep_host=not args.no_cpu_baseline)
    ms, wall, kdur, root_nnz, dense = time_steps(w, args.steps, args.warmup, torch)
    w_ms_plain = w.ms_plain
    log(f"{args.workload}: {ms:.3f} ms/step (wall {wall:.3f}), kernels {kdur}")
    value = w.nnz / (ms * 1e-3)
    step_gbs = w.step_bytes / (ms * 1e-3) / 1e9

    # dominant kernel and its roofline
    dom = max(kdur, key=lambda g: kdur[g])
    dom_bytes = w.kernel_bytes.get(dom)
    achieved = dom_bytes / (kdur[dom] * 1e-3) / 1e9 if dom_bytes else None
    roofline = {
        "bound": "hbm",
        "kernel": GROUP_NAMES[dom],
        "achieved": achieved,
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": achieved / HBM_PEAK_GBS if achieved else None,
        "traffic": traffic_for(GROUP_NAMES[dom], args.workload),
        "bytes_per_launch": dom_bytes,
        "avg_ms": kdur[dom],
    }
    kernels = {GROUP_NAMES[g]: {"avg_ms": v, "bytes": w.kernel_bytes.get(g),
                                "GB/s": (w.kernel_bytes[g] / (v * 1e-3) / 1e9) if w.kernel_bytes.get(g) else None,
                                "traffic": traffic_for(GROUP_NAMES[g], args.workload)}
               for g, v in kdur.items()}

    # the step's producer and reduce apart (kernel timers; launches between
    # kernels not included), each with its input rate
    def group_ms(gs):
        return sum(kdur.get(g, 0.0) for g in gs)
    prod = [S.TIMER_QUANT_NORM, S.TIMER_QUANT_CODES, S.TIMER_TOPK_SELECT, S.TIMER_TOPK_WRITE]
    red = [S.TIMER_REDUCE_PASS, S.TIMER_REDUCE_SLOW, S.TIMER_REDUCE_WRITE, S.TIMER_REDUCE_MERGE]
    parts = {"reduce": {"kernel_ms": group_ms(red), "input_nnz_per_s": w.nnz / (group_ms(red) * 1e-3)}}
    if group_ms(prod):
        pn = w.nnz if head_cfg.qbits else head_cfg.P * head_cfg.N
        parts["producer"] = {"kind": "qsgd" if head_cfg.qbits else "topk", "kernel_ms": group_ms(prod),
                             "input_elems_per_s": pn / (group_ms(prod) * 1e-3)}
    cold_ms = time_cold(w, 5, torch)
    log(f"{args.workload}: cold (Infinity Cache evicted) {cold_ms:.3f} ms/step")
    cpu = None
    threads = oracle_threads()
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle on the workload (1 and {threads} threads)")
        leg = oracle_leg(w, threads)
        cpu = {"value": leg["input_nnz_per_s"], "unit": "nnz/s", "cores": threads, "kind": "oracle",
               "sample": f"{leg['sample']}; one step of {describe(head_cfg)}, "
                         f"{leg['ms_per_step'] / 1e3:.2f} s on {threads} threads",
               "single_thread": {"value": leg["single_thread_input_nnz_per_s"], "cores": 1,
                                 "seconds": leg["single_thread_ms_per_step"] / 1e3},
               "host": f"{cpu_model()}, {os.cpu_count()} logical CPUs, {threads} usable"}
        log(f"oracle: {leg['ms_per_step']:.0f} ms on {threads} threads, "
            f"{leg['single_thread_ms_per_step']:.0f} ms on one")
    w = None
    torch.cuda.empty_cache()

    # the same step over further seeds (fresh inputs): median and quartiles
    seeds = None
    if not args.no_per_config and args.configs is None:
        per_seed = [ms]
        for sd in range(args.seed + 1, args.seed + 5):
            sw = Workload(args.workload, head_cfg, sd, torch, dev)
            sms = time_steps(sw, 10, 2, torch, warm_s=0.3)[0]
            per_seed.append(sms)
            sw = None
            torch.cuda.empty_cache()
        q25, q50, q75 = np.percentile(per_seed, [25, 50, 75])
        seeds = {"seeds": list(range(args.seed, args.seed + 5)), "ms_per_step": per_seed,
                 "median_ms": float(q50), "q25_ms": float(q25), "q75_ms": float(q75)}
        log(f"{args.workload}: over 5 seeds median {q50:.3f} ms (IQR {q25:.3f}-{q75:.3f})")
    ceiling = copy_ceiling(torch)
    log(f"copy ceiling {ceiling['GB/s']:.0f} GB/s")

    per_config = {}
    if not args.no_per_config:
        for name in ("c1", "c2", "c3", "c4", "c5", "c3/bucketed", "c4/p48", "c4/share", "c5/share",
                     "c5/dsar"):
            if name == args.workload or (args.configs is not None and name not in args.configs.split(",")):
                continue
            c = inputs.config(int(name[1]))
            if name.endswith("/p48"):  # a rank count that is not a power of two
                c = dataclasses.replace(c, P=48)
            share = (0, c.P) if name.endswith("/share") else None
            keep = not args.no_cpu_baseline
            if name.endswith("/dsar"):
                pw = DsarWorkload(name, c, args.seed, torch, dev, keep_host=keep)
            else:
                pw = Workload(name, c, args.seed, torch, dev, share=share,
                              bucketed=(512, 4) if name.endswith("/bucketed") else None, keep_host=keep)
            pms, pwall, pk, pn, pd = time_steps(pw, max(5, args.steps // 2), 2, torch, warm_s=0.3)
            desc = describe(c) + (f"; split-phase share [{pw.reduce.rng[0]}, {pw.reduce.rng[1]}) "
                                  f"(1 of {c.P})" if share else "")
            if name.endswith("/bucketed"):
                desc = (describe(c) + "; Alg. 1 error feedback (acc = eps + 0.1 grad) with 4 of every "
                        f"512 coordinates ({pw.topk.K} per rank) in place of the global top-k")
            if name.endswith("/dsar"):
                desc = (f"{c.name} streams in fp32 (P={c.P}, N={c.N}, k={c.k}, delta={c.delta}): "
                        f"share [0, {pw.R}) reduced, QSGD {pw.bits}-bit in buckets of {pw.bucket}, "
                        f"{c.P} quantized shares decoded into N")
            per_config[name] = {
                "workload": desc, "ms_per_step": pw.ms_plain, "input_nnz_per_s": pw.nnz / (pw.ms_plain * 1e-3),
                "ms_per_step_with_kernel_events": pms,
                "cold_ms_per_step": time_cold(pw, 3, torch),
                "step_GB/s": pw.step_bytes / (pw.ms_plain * 1e-3) / 1e9,
                "step_frac_of_hbm_peak": pw.step_bytes / (pw.ms_plain * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "root_nnz": pn, "root_dense": pd,
                "kernels": {GROUP_NAMES[g]: {"avg_ms": v, "GB/s": (pw.kernel_bytes[g] / (v * 1e-3) / 1e9)
                                             if pw.kernel_bytes.get(g) else None,
                                             "traffic": traffic_for(GROUP_NAMES[g], name)} for g, v in pk.items()},
            }
            if c.kind == "topk":
                tk = sum(pk.get(g, 0.0) for g in (S.TIMER_TOPK_SELECT, S.TIMER_TOPK_WRITE,
                                                  S.TIMER_TOPK_BUCKETED))
                per_config[name]["topk_input_elems_per_s"] = c.P * c.N / (tk * 1e-3) if tk else None
            if keep:
                leg = oracle_leg(pw, threads)
                per_config[name]["cpu_oracle"] = leg
                log(f"{name}: oracle {leg['ms_per_step']:.1f} ms on {threads} threads, "
                    f"{leg['single_thread_ms_per_step']:.1f} ms on one")
            log(f"{name}: {pw.ms_plain:.3f} ms/step ({pms:.3f} with kernel events)")
            pw = None
            torch.cuda.empty_cache()

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "nnz/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_no_events": w_ms_plain,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": describe(head_cfg), "P": head_cfg.P, "N": head_cfg.N, "k": head_cfg.k,
                   "delta": head_cfg.delta, "qbits": head_cfg.qbits, "seed": args.seed,
                   "root_nnz": root_nnz, "root_dense": dense},
        "step_GB/s": step_gbs,
        "roofline": roofline,
        "kernels": kernels,
        "parts": parts,
        "cpu_baseline": cpu,
        "wall_ms_per_step": wall,
        "cold_ms_per_step": cold_ms,
        "seeds": seeds,
        "copy_ceiling": ceiling,
        "per_config": per_config,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
