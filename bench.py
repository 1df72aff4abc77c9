#!/usr/bin/env python3
"""YOSO attention forward + backward throughput on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
    codes_q = hash(Q), codes_k = hash(K)       (yoso_hash, twice)
    Y = forward(codes, V)                      (yoso_forward)
    dQ, dK, dV = backward(codes, Q, K, V, dY)  (yoso_backward)
for every (batch, head) of the workload (default: 16 x 2 heads, n = 4096, d = 64,
m = 32 hashes of tau = 8 bits, fp32).  Inputs are resident in HBM before the
timed region; W warm-up steps are followed by K timed steps bracketed by device
synchronisation.  The timed steps replay the step captured once into a HIP graph
(the same kernels on the same inputs, without host launch gaps; `execution`
says which mode ran, and `eager_ms_per_step` gives the eager time as well).
One JSON line is printed on stdout.

Per-kernel durations come from HIP events that the library records around each
of its launches on the launch stream (yoso_timing_enable); the roofline object
describes the kernel with the largest total time.  For the dQ, dK pair kernel that
is a matrix-unit roofline (3d multiply-adds per colliding pair, at the matrix
peak of the input type: fp32, or bf16 for bf16 inputs), with its HBM figures
alongside.  The CPU baseline is the fp64
oracle, timed on this machine's host cores on a stated sample of heads.

The `configs` object repeats the step measurement (graph replay, fewer steps for
the long sequences) for each of the five workloads, with the dominant kernel's
roofline and a bounded oracle sample; `yoso_star` times the *YOSO backward on
the bench workload.
"""
from __future__ import annotations

import argparse
import concurrent.futures
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "YOSO attention fwd+bwd tokens/sec at n=4096,d=64,m=32,tau=8; % HBM roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense fp16/bf16 matrix peak
FP32_PEAK_TFLOPS = 157.3        # MI355X fp32 (matrix or vector) peak
# fp32 vector instructions without packed math: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12


def kernel_algorithmic(w, kernel: str):
    """Algorithmic bytes one launch of `kernel` must move (each launch covers every head):
      hash_kernel    reads one of Q, K                                  n*d*e per head
      table_kernel   forward: reads V, writes Y; dV: reads dY, writes dV  2*n*d*e
      pass_kernel    reads Q, K, V, dY (both the dQ and the dK pass)      4*n*d*e
      reduce_kernel  writes one of dQ, dK                               n*d*e
    Everything else these kernels move (codes, per-hash partial rows, re-reads of
    rows for every hash) is implementation traffic and is not credited."""
    nde = w.n * w.d * w.elem_bytes
    per_head = {"hash_kernel": nde, "table_kernel": 2 * nde, "pass_kernel": 4 * nde,
                "reduce_kernel": nde}.get(kernel)
    if per_head is None:
        return None
    return per_head * w.bh


def bucket_work(qc, kc, tau: int, t: int):
    """Work of the backward's two forms, from the codes on the host, summed over
    heads and hashes: (pairs, pair_form_pairs, table_form_rows).  `pairs` counts the
    colliding (query, key) pairs, sum of count_q * count_k over (head, hash, bucket);
    buckets with count_q * count_k > t (count_q + count_k) take the table form and
    contribute count_q + count_k rows, the others their pairs."""
    import numpy as np
    B = 1 << tau
    q = qc.cpu().numpy().astype(np.int64) & (B - 1)  # [bh, n_q, m]
    k = kc.cpu().numpy().astype(np.int64) & (B - 1)  # [bh, n_k, m]
    bh, _, m = q.shape
    unit = (np.arange(bh)[:, None, None] * m + np.arange(m)[None, None, :]) * B
    hq = np.bincount((unit + q).ravel(), minlength=bh * m * B)
    hk = np.bincount((unit + k).ravel(), minlength=bh * m * B)
    prod = hq * hk
    tab = prod > t * (hq + hk)
    return int(prod.sum()), int(prod[~tab].sum()), int((hq + hk)[tab].sum())


# upper bounds of the bucket-size classes of bucket_load's histogram (rows of one
# side in one (head, hash, bucket)); the last class is everything above
LOAD_CLASSES = (16, 64, 256, 1024)


def bucket_load(qc, kc, tau: int):
    """How the rows fall into buckets, from the codes on the host: per side the mean
    rows per (head, hash, bucket) (n / 2^tau), the largest bucket and their ratio, and
    the share of rows in buckets of each size class (up to 16, 64, 256, 1024 rows, and
    more)."""
    import numpy as np
    B = 1 << tau
    out = {}
    for side, c in (("queries", qc), ("keys", kc)):
        x = c.cpu().numpy().astype(np.int64) & (B - 1)  # [bh, n, m]
        bh, n, m = x.shape
        unit = (np.arange(bh)[:, None, None] * m + np.arange(m)[None, None, :]) * B
        cnt = np.bincount((unit + x).ravel(), minlength=bh * m * B)
        mean = n / B
        rows = np.zeros(len(LOAD_CLASSES) + 1)
        lo = 0
        for i, hi in enumerate(LOAD_CLASSES + (None,)):
            sel = (cnt > lo) if hi is None else ((cnt > lo) & (cnt <= hi))
            rows[i] = cnt[sel].sum()
            lo = hi if hi is not None else lo
        total = max(rows.sum(), 1)
        labels = [f"<={hi}" for hi in LOAD_CLASSES] + [f">{LOAD_CLASSES[-1]}"]
        out[side] = {"mean_rows": round(mean, 3), "max_rows": int(cnt.max()) if cnt.size else 0,
                     "max_over_mean": round(float(cnt.max()) / mean, 2) if cnt.size and mean > 0 else None,
                     "row_share_by_bucket_rows": {lab: round(float(r / total), 4) for lab, r in zip(labels, rows)}}
    return out


COPY_BYTES = 256 << 20


def source_digest(files) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# Kernel -> the sources its code comes from (the traffic figure is void once they change).
_PAIRS = ["paper_2111_09714_amd/csrc/pairs.hip", "paper_2111_09714_amd/csrc/common.h"]
KERNEL_SOURCES = {
    "hash_kernel": ["paper_2111_09714_amd/csrc/hash.hip", "paper_2111_09714_amd/csrc/common.h"],
    "table_kernel": ["paper_2111_09714_amd/csrc/tables.hip", "paper_2111_09714_amd/csrc/common.h"],
    **{k: _PAIRS for k in ("codes_t_kernel", "sort_kernel", "absmax_kernel", "split_kernel", "pass_kernel", "bucket_kernel",
                           "reduce_kernel", "dense_kernel", "dense_sum_kernel", "dense_fwd_kernel")},
}


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from its committed counter summary
    (profiles/<kernel>_<workload>_traffic.md), or None when there is none or the
    kernel's sources have changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.startswith("- `"):
                key, _, val = line[3:].partition("`:")
                fields[key.strip()] = val.strip().strip("`")
    if fields.get("source_digest") != source_digest(KERNEL_SOURCES[kernel]):
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, inp, heads, min_wall: float = 10.0):
    """Time the oracle (hash + forward + backward) on `heads`, one head per thread,
    repeating the sample until `min_wall` seconds have been spent (at most 30 s)."""
    import oracle
    oracle._load()
    threads = min(len(os.sched_getaffinity(0)), len(heads))

    def one(h):
        oracle.run_all(inp, w.m, w.tau, heads=slice(h, h + 1))

    # repeat the sample until about 10 s of wall time have been spent (at most 30 s)
    reps, wall = 0, 0.0
    with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as ex:
        while reps == 0 or (wall < min_wall and wall * (reps + 1) / reps < 30.0):
            t0 = time.perf_counter()
            list(ex.map(one, heads))
            wall += time.perf_counter() - t0
            reps += 1
    step_equiv = wall / reps * w.bh / len(heads)
    return {
        "value": w.tokens / step_equiv,
        "unit": "tokens/s",
        "cores": threads,
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": f"{len(heads)} of {w.bh} heads of the same workload (hash+forward+backward, fp64 C oracle, "
                  f"one head per thread), {reps} repetitions in {wall:.2f} s wall, scaled by {w.bh}/{len(heads)}",
    }


STEP_KERNELS = ("hash_kernel", "table_kernel", "codes_t_kernel", "sort_kernel", "absmax_kernel", "split_kernel",
                "pass_kernel",
                "bucket_kernel",
                "reduce_kernel", "dense_kernel", "dense_sum_kernel", "dense_fwd_kernel", "zero_kernel")


def make_step(Y, torch, w, inp, dev):
    """Device tensors of workload `w` and the step (hash Q, hash K, forward, backward)."""
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    t = {s: torch.from_numpy(inp[s]).to(dev).to(tdt).contiguous() for s in ("q", "k", "v", "dy")}
    t["R"] = torch.from_numpy(inp["R"]).to(dev)
    t["qc"] = torch.empty((w.bh, w.n, w.m), dtype=torch.int16, device=dev)
    t["kc"] = torch.empty_like(t["qc"])
    t["y"] = torch.empty_like(t["q"])
    t["dq"], t["dk"], t["dv"] = torch.empty_like(t["q"]), torch.empty_like(t["k"]), torch.empty_like(t["v"])
    t["ws_f"] = Y.workspace(Y.OP_FORWARD, t["q"], w.m, w.tau)
    t["ws_b"] = Y.workspace(Y.OP_BACKWARD, t["q"], w.m, w.tau)

    def step(s):
        Y.yoso_hash(t["q"], t["R"], w.m, w.tau, t["qc"], s)
        Y.yoso_hash(t["k"], t["R"], w.m, w.tau, t["kc"], s)
        Y.yoso_forward(t["qc"], t["kc"], t["v"], w.m, w.tau, t["y"], t["ws_f"], s)
        Y.yoso_backward(t["qc"], t["kc"], t["q"], t["k"], t["v"], t["dy"], w.m, w.tau, t["dq"], t["dk"], t["dv"],
                        t["ws_b"], s)
    return t, step


def time_step(Y, torch, step, steps, warmup):
    """(eager ms per step, per-kernel timings, graph-replay ms per step, execution mode)."""
    stream = torch.cuda.current_stream()
    # per-kernel durations: eager steps with the library's HIP-event timer on
    Y.yoso_timing_enable(4 * (steps + warmup) + 8)
    for _ in range(warmup):
        step(stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        step(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    eager_ms_per_step = start.elapsed_time(stop) / steps
    kernels = {}
    for name in STEP_KERNELS:
        tot, n = Y.yoso_timing_query(name)
        if n:
            kernels[name] = {"launches_per_step": n / steps, "avg_us": 1000.0 * tot / n,
                             "share_of_step": tot / (eager_ms_per_step * steps)}
    Y.yoso_timing_enable(0)

    # The timed run: the step captured once into a HIP graph (stream capture; the
    # library enqueues kernels only) and replayed: the same kernels on the same
    # inputs, without the host's launch gaps.  Eager steps if capture fails.
    execution = "hip_graph"
    try:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step(side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(torch.cuda.current_stream())
        torch.cuda.synchronize()
        run = graph.replay
    except Exception as exc:  # report and time eagerly
        execution = f"eager (graph capture failed: {type(exc).__name__})"
        run = lambda: step(stream)  # noqa: E731
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(steps):
        run()
    stop.record(stream)
    torch.cuda.synchronize()
    return eager_ms_per_step, kernels, start.elapsed_time(stop) / steps, execution


def dominant_roofline(w, kernels, qc, kc):
    """Roofline of the kernel with the largest time per step: HBM for the streaming
    kernels, the matrix peak of the input type for the dQ/dK kernels (3d multiply-adds
    per colliding pair, 2d^2 per table row and side, counted exactly from the codes)
    with their HBM figures alongside."""
    dominant = max(kernels, key=lambda kname: kernels[kname]["avg_us"] * kernels[kname]["launches_per_step"])
    alg = kernel_algorithmic(w, dominant)
    avg_s = kernels[dominant]["avg_us"] * 1e-6
    roofline = None
    if alg is not None:
        achieved = alg / avg_s / 1e9
        roofline = {"kernel": dominant, "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                    "algorithmic_bytes_per_launch": alg, "avg_launch_us": round(kernels[dominant]["avg_us"], 2)}
    # A contraction is priced at the matrix peak of its own input type: fp32 inputs
    # against the fp32 peak (they run as three fp16 products), bf16 inputs against
    # the dense bf16/fp16 peak (bf16 values are exact fp16 operands there).
    peak = FP16_MFMA_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    if dominant in ("pass_kernel", "bucket_kernel"):
        # dQ, dK are dense per-bucket contractions, bound by the matrix units.
        # Pair form (pass_kernel): per colliding (query, key) pair 3d multiply-adds
        # (dy.v once, then its share of dQ and of dK).  Table form (bucket_kernel): per
        # row of a table bucket and side 2 d^2 (its share of M = sum a' b^T, then its
        # row of a^T M).  Both counted exactly from this step's codes.
        import paper_2111_09714_amd as Y
        pairs, pair_form, table_rows = bucket_work(qc, kc, w.tau, Y.yoso_backward_table_threshold())
        flops = 6 * w.d * pair_form if dominant == "pass_kernel" else 4 * w.d * w.d * table_rows
        tf = flops / avg_s / 1e12
        hbm = roofline
        roofline = {"kernel": dominant, "bound": "mfma", "achieved": round(tf, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(tf / peak, 4), "traffic": None,
                    "algorithmic_flops_per_launch": flops, "colliding_pairs_per_launch": pairs,
                    "pair_form_pairs_per_launch": pair_form, "table_form_rows_per_launch": table_rows,
                    "avg_launch_us": round(kernels[dominant]["avg_us"], 2)}
        if hbm is not None:
            roofline["hbm"] = {"achieved": hbm["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": hbm["frac"], "algorithmic_bytes_per_launch": alg}
    if dominant == "dense_kernel":
        # short sequences: dQ, dK and dV as dense blocks over every (query, key) pair,
        # 5 d multiply-adds per pair (dy.v once for each of the two sides, then its
        # shares of dQ, dK and the count-weighted dV)
        flops = 10 * w.d * w.n * w.n * w.bh
        tf = flops / avg_s / 1e12
        roofline = {"kernel": dominant, "bound": "mfma", "achieved": round(tf, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(tf / peak, 4), "traffic": None,
                    "algorithmic_flops_per_launch": flops, "avg_launch_us": round(kernels[dominant]["avg_us"], 2)}
    if roofline is not None:
        roofline["traffic"] = measured_traffic(dominant, w.name)
    return roofline


# Steps and warm-up steps per workload in the `configs` object (the long
# sequences take tens of milliseconds per step).
CONFIG_STEPS = {"single_head_n512": (20, 5), "bert_base_n512": (10, 3), "lra_n4096": (10, 3),
                "skewed_n16384": (4, 1), "bf16_n32768": (4, 1)}


def measure_configs(Y, torch, dev, cpu: bool):
    """The step on every workload: graph-replayed time, tokens/s, HBM fraction, the
    dominant kernel's roofline, the kernel table, and the oracle on a sample of heads."""
    from workloads import WORKLOADS, make_inputs
    out = {}
    for name, (steps, warmup) in CONFIG_STEPS.items():
        w = WORKLOADS[name]
        inp = make_inputs(w)
        t, step = make_step(Y, torch, w, inp, dev)
        _, kernels, ms, execution = time_step(Y, torch, step, steps, warmup)
        alg = 11 * w.n * w.d * w.elem_bytes * w.bh
        entry = {"config": {"batch": w.batch, "heads": w.heads, "seq_len": w.n, "tau": w.tau, "hashes": w.m,
                            "dtype": w.dtype, "inputs": w.dist},
                 "steps": steps, "ms_per_step": round(ms, 4), "execution": execution,
                 "tokens_per_s": round(w.tokens / (ms * 1e-3), 1),
                 "hbm_roofline_frac": round(alg / (ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
                 "roofline": dominant_roofline(w, kernels, t["qc"], t["kc"]),
                 "bucket_load": bucket_load(t["qc"], t["kc"], w.tau),
                 "kernels": {kn: {"launches_per_step": round(kv["launches_per_step"], 2),
                                  "avg_us": round(kv["avg_us"], 2)} for kn, kv in kernels.items()}}
        del t, step
        torch.cuda.empty_cache()
        if cpu:
            # one oracle pass over as many heads as there are cores (at most the head
            # count; long sequences: 4 heads), scaled to all heads
            cores = len(os.sched_getaffinity(0))
            nh = min(w.bh, cores, 4 if w.n > 4096 else cores)
            entry["cpu_baseline"] = cpu_baseline(w, inp, list(range(nh)), min_wall=0.0)
        out[name] = entry
        del inp
    return out


SCALING_N = (1024, 2048, 4096, 8192, 16384, 32768)


def scaling_timing(Y, torch, dev, reps: int = 5):
    """Time per token against sequence length at fixed heads, tau and m (Table 1:
    the forward is linear in n; the backward, pairs per bucket growing with n, is
    linear where the buckets take the table form): hash of Q and K, forward and
    backward on 8 heads (4 x 2), tau = 8, m = 32, fp32, Gaussian inputs, each timed
    with events around `reps` eager calls after one warm-up call."""
    from workloads import Workload, make_inputs
    rows = []
    for n in SCALING_N:
        w = Workload(f"scaling_n{n}", 4, 2, n, 64, 8, 32, "f32", "gauss", 2111_09714 + n)
        inp = make_inputs(w)
        q, k, v, dy = (torch.from_numpy(inp[s]).to(dev) for s in ("q", "k", "v", "dy"))
        R = torch.from_numpy(inp["R"]).to(dev)
        qc = torch.empty((w.bh, n, w.m), dtype=torch.int16, device=dev)
        kc = torch.empty_like(qc)
        y, dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        wsf = Y.workspace(Y.OP_FORWARD, q, w.m, w.tau)
        wsb = Y.workspace(Y.OP_BACKWARD, q, w.m, w.tau)
        calls = {"hash_ms": lambda: (Y.yoso_hash(q, R, w.m, w.tau, qc), Y.yoso_hash(k, R, w.m, w.tau, kc)),
                 "forward_ms": lambda: Y.yoso_forward(qc, kc, v, w.m, w.tau, y, wsf),
                 "backward_ms": lambda: Y.yoso_backward(qc, kc, q, k, v, dy, w.m, w.tau, dq, dk, dv, wsb)}
        row = {"n": n}
        for key, call in calls.items():
            call()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                call()
            b.record()
            torch.cuda.synchronize()
            row[key] = round(a.elapsed_time(b) / reps, 4)
        tokens = w.batch * n
        for key in ("hash_ms", "forward_ms", "backward_ms"):
            row[key.replace("_ms", "_ns_per_token")] = round(row[key] * 1e6 / tokens, 2)
        rows.append(row)
        del q, k, v, dy, R, qc, kc, y, dq, dk, dv, wsf, wsb, inp
        torch.cuda.empty_cache()
    return {"heads": 8, "batch": 4, "tau": 8, "hashes": 32, "dtype": "f32", "inputs": "gauss", "rows": rows}


def star_timing(Y, torch, w, t, stream):
    """*YOSO's backward (yoso_backward_star) on the bench workload, outside the timed
    step: its pair kernel runs over the m*tau derived hashes (pairs whose codes agree
    on all bits but at most one); 8d flops per derived pair (s = dy.v and x = q.k,
    then the dQ and the dK share)."""
    import numpy as np
    ws = Y.workspace(Y.OP_BACKWARD_STAR, t["q"], w.m, w.tau)
    dq, dk, dv = torch.empty_like(t["q"]), torch.empty_like(t["k"]), torch.empty_like(t["v"])
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def call():
        Y.yoso_backward_star(t["qc"], t["kc"], t["q"], t["k"], t["v"], t["dy"], w.m, w.tau, dq, dk, dv, ws, stream)

    call()
    torch.cuda.synchronize()
    Y.yoso_timing_enable(64)
    start.record(stream)
    for _ in range(3):
        call()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / 3
    tot, n = Y.yoso_timing_query("pass_star_kernel")
    Y.yoso_timing_enable(0)
    # pairs of the derived hashes (code minus bit t), counted from the codes
    B = 1 << (w.tau - 1)
    qc = t["qc"].cpu().numpy().astype(np.int64) & ((1 << w.tau) - 1)
    kc = t["kc"].cpu().numpy().astype(np.int64) & ((1 << w.tau) - 1)
    bh, _, m = qc.shape
    unit = (np.arange(bh)[:, None, None] * m + np.arange(m)[None, None, :]) * B
    pairs = 0
    for bit in range(w.tau):
        low = (1 << bit) - 1
        qd = ((qc >> (bit + 1)) << bit) | (qc & low)
        kd = ((kc >> (bit + 1)) << bit) | (kc & low)
        hq = np.bincount((unit + qd).ravel(), minlength=bh * m * B)
        hk = np.bincount((unit + kd).ravel(), minlength=bh * m * B)
        pairs += int((hq * hk).sum())
    del ws, dq, dk, dv
    out = {"ms_per_backward": round(ms, 3), "derived_pairs": pairs}
    if n:
        avg_s = tot / n * 1e-3
        tf = 8 * w.d * pairs / avg_s / 1e12
        out["pass_star_kernel"] = {"avg_us": round(avg_s * 1e6, 1), "bound": "mfma", "achieved": round(tf, 2),
                                   "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                                   "frac": round(tf / FP32_PEAK_TFLOPS, 4),
                                   "algorithmic_flops_per_launch": 8 * w.d * pairs}
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="lra_n4096")
    ap.add_argument("--cpu-heads", type=int, default=-1, help="heads in the oracle sample (-1: all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the per-workload `configs` object")
    ap.add_argument("--parts", default="star,l2,yoso_e,fast_hash,scaling",
                    help="measurements besides the step (comma list of star, l2, yoso_e, fast_hash, scaling; 'none' "
                         "for none), "
                         "e.g. to profile the step's kernels alone")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run a plain 256 MiB device copy (read + write) three times, "
                         "so that a counter run sees a kernel of known traffic")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the (batch, head) units of YOSO attention are independent, so N GPUs would each run "
              "this same kernel sequence on BH/N heads with no communication.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2111_09714_amd as Y
    from workloads import WORKLOADS, make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    w = WORKLOADS[args.workload]
    inp = make_inputs(w)
    dev = torch.device("cuda:0")
    t, step = make_step(Y, torch, w, inp, dev)
    q, k, v, dy, qc, kc = (t[s] for s in ("q", "k", "v", "dy", "qc", "kc"))
    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    eager_ms_per_step, kernels, ms_per_step, execution = time_step(Y, torch, step, args.steps, args.warmup)
    roofline = dominant_roofline(w, kernels, qc, kc)
    parts = {p.strip() for p in args.parts.split(",") if p.strip()}
    star = star_timing(Y, torch, w, t, stream) if "star" in parts else None

    # the l2 row normalisation (N-YOSO output / Q, K prologue) on this workload's Q
    # rows, outside the timed step: HBM-bound, algorithmic bytes = rows read + written
    l2 = {}
    qn, dqn = torch.empty_like(q), torch.empty_like(q)
    l2_reps = 10 if "l2" in parts else 0
    Y.yoso_timing_enable(64)
    for _ in range(3 if l2_reps else 0):
        Y.yoso_l2_normalize(q, qn, stream)
        Y.yoso_l2_normalize_backward(q, dy, dqn, stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    for _ in range(l2_reps):
        Y.yoso_l2_normalize(q, qn, stream)
        Y.yoso_l2_normalize_backward(q, dy, dqn, stream)
    torch.cuda.synchronize()
    row_bytes = w.d * w.elem_bytes
    for name, per_row in (("l2norm_kernel", 2 * row_bytes), ("l2norm_bwd_kernel", 3 * row_bytes)):
        tot, n = Y.yoso_timing_query(name)
        if n:
            avg_s = tot / n * 1e-3
            gbs = per_row * w.bh * w.n / avg_s / 1e9
            l2[name] = {"avg_us": round(avg_s * 1e6, 2), "bound": "hbm", "achieved": round(gbs, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "algorithmic_bytes_per_launch": per_row * w.bh * w.n}
    Y.yoso_timing_enable(0)
    del qn, dqn

    # YOSO-E (exact expectation, O(n^2 d)) on the same inputs, outside the timed step:
    # MFMA-bound dense tiles.  Algorithmic fp32 flops per head: forward 4 n_q n_k d (Q K^T
    # and P V), backward 14 n_q n_k d (cosines and G twice, dV, dK, dQ); each is run as
    # three fp16 products.
    expect = {}
    ye = torch.empty_like(q)
    dqe, dke, dve = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    e_reps = 3 if "yoso_e" in parts else 0
    Y.yoso_timing_enable(64)
    if e_reps:
        Y.yoso_expectation_forward(q, k, v, w.tau, ye, stream)
        Y.yoso_expectation_backward(q, k, v, dy, w.tau, dqe, dke, dve, stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    for _ in range(e_reps):
        Y.yoso_expectation_forward(q, k, v, w.tau, ye, stream)
        Y.yoso_expectation_backward(q, k, v, dy, w.tau, dqe, dke, dve, stream)
    torch.cuda.synchronize()
    nnd = float(w.n) * w.n * w.d * w.bh
    for name, flops in (("expect_fwd_kernel", 4 * nnd), ("expect_bwd_kv_kernel", 8 * nnd),
                        ("expect_bwd_q_kernel", 6 * nnd)):
        tot, n = Y.yoso_timing_query(name)
        if n:
            avg_s = tot / n * 1e-3
            tf = flops / avg_s / 1e12
            expect[name] = {"avg_us": round(avg_s * 1e6, 1), "bound": "mfma", "achieved": round(tf, 1),
                            "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / FP32_PEAK_TFLOPS, 4),
                            "fp16_mfma_util": round(3 * tf / FP16_MFMA_PEAK_TFLOPS, 4),
                            "algorithmic_flops_per_launch": flops}
    Y.yoso_timing_enable(0)
    del ye, dqe, dke, dve

    # The fast hash (Sec. 3.2 "Speed-up") on this workload's Q and K, outside the timed
    # step: fast_hash_kernel applies the Walsh-Hadamard rotations row by row and is
    # bound by fp32 VALU issue.  Its ALU peak counts one instruction per lane and
    # clock (no packed fp32): 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz.  Per row and
    # rotation the algorithm needs 3 * 64 * 6 = 1152 butterfly operations.  The
    # expansion of the rotations into hyperplanes (for the dense hash kernel) is
    # timed as well.
    fast = {}
    signs = torch.from_numpy(inp["signs"].view(np.int64)).to(dev)
    Rf = torch.empty((w.d, w.m * w.tau), dtype=torch.float32, device=dev)
    Y.yoso_timing_enable(64)
    for it in range(11 if "fast_hash" in parts else 0):
        if it == 1:
            torch.cuda.synchronize()
            Y.yoso_timing_reset()
        Y.yoso_fast_hash(q, signs, w.m, w.tau, qc, stream)
        Y.yoso_fast_hash(k, signs, w.m, w.tau, kc, stream)
        Y.yoso_fast_hyperplanes(signs, w.m, w.tau, Rf, stream)
    torch.cuda.synchronize()
    nrot = (w.m * w.tau + 63) // 64
    ops = 1152.0 * nrot * w.bh * w.n
    for name in ("fast_hash_kernel", "fast_hyperplanes_kernel"):
        tot, n = Y.yoso_timing_query(name)
        if n:
            avg_s = tot / n * 1e-3
            fast[name] = {"avg_us": round(avg_s * 1e6, 2), "launches_per_call": n / 10}
            if name == "fast_hash_kernel":
                tops = ops / avg_s / 1e12
                fast[name].update({"bound": "alu", "achieved": round(tops, 2), "peak": VALU_PEAK_TOPS,
                                   "unit": "Top/s", "frac": round(tops / VALU_PEAK_TOPS, 4),
                                   "algorithmic_ops_per_launch": ops})
    Y.yoso_timing_enable(0)
    del signs, Rf

    if args.copy_calibration:
        # elementwise multiply by 1: one kernel reading and writing COPY_BYTES each
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()

    # measured HBM copy bandwidth (1 GiB device-to-device copy, bytes read + written,
    # median of five), the practical ceiling next to the 8 TB/s vendor figure
    csrc = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    cdst = torch.empty_like(csrc)
    copy_ms = []
    for _ in range(6):
        start.record(stream)
        cdst.copy_(csrc)
        stop.record(stream)
        torch.cuda.synchronize()
        copy_ms.append(start.elapsed_time(stop))
    copy_gbs = 2 * csrc.numel() * 4 / (sorted(copy_ms[1:])[2] * 1e-3) / 1e9
    del csrc, cdst

    tokens_per_s = w.tokens / (ms_per_step * 1e-3)
    alg_step_bytes = 11 * w.n * w.d * w.elem_bytes * w.bh
    hbm_frac = alg_step_bytes / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9)
    copy_frac = alg_step_bytes / (ms_per_step * 1e-3) / (copy_gbs * 1e9)

    cpu = None
    if not args.no_cpu_baseline:
        nh = w.bh if args.cpu_heads < 0 else min(args.cpu_heads, w.bh)
        cpu = cpu_baseline(w, inp, list(range(nh)))

    out = {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "heads": w.heads, "seq_len": w.n, "head_dim": w.d,
                   "tau": w.tau, "hashes": w.m, "inputs": w.dist},
        "execution": execution,
        "eager_ms_per_step": round(eager_ms_per_step, 5),
        "hbm_roofline_frac": round(hbm_frac, 4),
        "hbm_copy_GBs": round(copy_gbs, 1),
        "hbm_roofline_frac_of_copy": round(copy_frac, 4),
        "algorithmic_bytes_per_step": alg_step_bytes,
        "roofline": roofline,
        "bucket_load": bucket_load(qc, kc, w.tau),
        "kernels": {kn: {kk: round(vv, 3) for kk, vv in kv.items()} for kn, kv in kernels.items()},
        "cpu_baseline": cpu,
        "l2_normalize": l2,
        "yoso_e": expect,
        "fast_hash": fast,
        "yoso_star": star,
    }
    if "scaling" in parts:
        del t, step, q, k, v, dy, qc, kc
        torch.cuda.empty_cache()
        out["scaling"] = scaling_timing(Y, torch, dev)
    if not args.no_configs:
        if "scaling" not in parts:
            del t, step, q, k, v, dy, qc, kc
        torch.cuda.empty_cache()
        out["configs"] = measure_configs(Y, torch, dev, cpu=not args.no_cpu_baseline)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
