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
is a matrix-unit roofline (3d multiply-adds per colliding pair, fp32 peak), with
its HBM figures alongside.  The CPU baseline is the fp64
oracle, timed on this machine's host cores on a stated sample of heads.
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


def colliding_pairs(qc, kc, tau: int) -> int:
    """Number of (query, key) pairs that share a bucket, summed over heads and hashes:
    sum over (head, hash, bucket) of count_q * count_k, from the codes on the host."""
    import numpy as np
    B = 1 << tau
    q = qc.cpu().numpy().astype(np.int64) & (B - 1)  # [bh, n_q, m]
    k = kc.cpu().numpy().astype(np.int64) & (B - 1)  # [bh, n_k, m]
    bh, _, m = q.shape
    unit = (np.arange(bh)[:, None, None] * m + np.arange(m)[None, None, :]) * B
    hq = np.bincount((unit + q).ravel(), minlength=bh * m * B)
    hk = np.bincount((unit + k).ravel(), minlength=bh * m * B)
    return int((hq * hk).sum())


COPY_BYTES = 256 << 20


def source_digest(files) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# Kernel -> the sources its code comes from (the traffic figure is void once they change).
KERNEL_SOURCES = {
    "pass_kernel": ["paper_2111_09714_amd/csrc/pairs.hip", "paper_2111_09714_amd/csrc/common.h"],
    "table_kernel": ["paper_2111_09714_amd/csrc/tables.hip", "paper_2111_09714_amd/csrc/common.h"],
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


def cpu_baseline(w, inp, heads):
    """Time the oracle (hash + forward + backward) on `heads`, one head per thread."""
    import oracle
    oracle._load()
    threads = min(len(os.sched_getaffinity(0)), len(heads))

    def one(h):
        oracle.run_all(inp, w.m, w.tau, heads=slice(h, h + 1))

    # repeat the sample until about 10 s of wall time have been spent (at most 30 s)
    reps, wall = 0, 0.0
    with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as ex:
        while reps == 0 or (wall < 10.0 and wall * (reps + 1) / reps < 30.0):
            t0 = time.perf_counter()
            list(ex.map(one, heads))
            wall += time.perf_counter() - t0
            reps += 1
    step_equiv = wall / reps * w.bh / len(heads)
    return {
        "value": w.tokens / step_equiv,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{len(heads)} of {w.bh} heads of the same workload (hash+forward+backward, fp64 C oracle, "
                  f"one head per thread), {reps} repetitions in {wall:.2f} s wall, scaled by {w.bh}/{len(heads)}",
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="lra_n4096")
    ap.add_argument("--cpu-heads", type=int, default=-1, help="heads in the oracle sample (-1: all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = torch.device("cuda:0")
    q, k, v, dy = (torch.from_numpy(inp[s]).to(dev).to(tdt).contiguous() for s in ("q", "k", "v", "dy"))
    R = torch.from_numpy(inp["R"]).to(dev)
    qc = torch.empty((w.bh, w.n, w.m), dtype=torch.int16, device=dev)
    kc = torch.empty_like(qc)
    y = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws_f = Y.workspace(Y.OP_FORWARD, q, w.m, w.tau)
    ws_b = Y.workspace(Y.OP_BACKWARD, q, w.m, w.tau)
    stream = torch.cuda.current_stream()

    def step(s):
        Y.yoso_hash(q, R, w.m, w.tau, qc, s)
        Y.yoso_hash(k, R, w.m, w.tau, kc, s)
        Y.yoso_forward(qc, kc, v, w.m, w.tau, y, ws_f, s)
        Y.yoso_backward(qc, kc, q, k, v, dy, w.m, w.tau, dq, dk, dv, ws_b, s)

    # per-kernel durations: eager steps with the library's HIP-event timer on
    Y.yoso_timing_enable(4 * (args.steps + args.warmup) + 8)
    for _ in range(args.warmup):
        step(stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    eager_ms_per_step = start.elapsed_time(stop) / args.steps
    kernels = {}
    for name in ("hash_kernel", "table_kernel", "sort_kernel", "split_kernel", "pass_kernel", "reduce_kernel",
                 "zero_kernel"):
        tot, n = Y.yoso_timing_query(name)
        if n:
            kernels[name] = {"launches_per_step": n / args.steps, "avg_us": 1000.0 * tot / n,
                             "share_of_step": tot / (eager_ms_per_step * args.steps)}
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
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        run()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    ms_per_step = ms_total / args.steps

    dominant = max(kernels, key=lambda kname: kernels[kname]["avg_us"] * kernels[kname]["launches_per_step"])
    alg = kernel_algorithmic(w, dominant)
    avg_s = kernels[dominant]["avg_us"] * 1e-6
    roofline = None
    if alg is not None:
        achieved = alg / avg_s / 1e9
        roofline = {"kernel": dominant, "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                    "algorithmic_bytes_per_launch": alg, "avg_launch_us": round(kernels[dominant]["avg_us"], 2)}
    if dominant == "pass_kernel":
        # dQ, dK are dense per-bucket contractions, bound by the matrix units: per
        # colliding (query, key) pair 3d multiply-adds (dy.v once, then its share of
        # dQ and of dK), in fp32; the pairs are counted exactly from this step's codes
        pairs = colliding_pairs(qc, kc, w.tau)
        flops = 6 * w.d * pairs
        tf = flops / avg_s / 1e12
        hbm = roofline
        roofline = {"kernel": dominant, "bound": "mfma", "achieved": round(tf, 2), "peak": FP32_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(tf / FP32_PEAK_TFLOPS, 4), "traffic": None,
                    "algorithmic_flops_per_launch": flops, "colliding_pairs_per_launch": pairs,
                    "avg_launch_us": round(kernels[dominant]["avg_us"], 2),
                    "hbm": {"achieved": hbm["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": hbm["frac"],
                            "algorithmic_bytes_per_launch": alg}}

    if roofline is not None:
        roofline["traffic"] = measured_traffic(dominant, w.name)

    # the l2 row normalisation (N-YOSO output / Q, K prologue) on this workload's Q
    # rows, outside the timed step: HBM-bound, algorithmic bytes = rows read + written
    l2 = {}
    qn, dqn = torch.empty_like(q), torch.empty_like(q)
    Y.yoso_timing_enable(64)
    for _ in range(3):
        Y.yoso_l2_normalize(q, qn, stream)
        Y.yoso_l2_normalize_backward(q, dy, dqn, stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    for _ in range(10):
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
    Y.yoso_timing_enable(64)
    Y.yoso_expectation_forward(q, k, v, w.tau, ye, stream)
    Y.yoso_expectation_backward(q, k, v, dy, w.tau, dqe, dke, dve, stream)
    torch.cuda.synchronize()
    Y.yoso_timing_reset()
    for _ in range(3):
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
    for it in range(11):
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
        "kernels": {kn: {kk: round(vv, 3) for kk, vv in kv.items()} for kn, kv in kernels.items()},
        "cpu_baseline": cpu,
        "l2_normalize": l2,
        "yoso_e": expect,
        "fast_hash": fast,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
