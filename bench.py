#!/usr/bin/env python3
"""Throughput of the AsymSpec fused decision step on one MI355X.

One step = one call of asymspec_fuse_verify over a batch of B requests with K
drafts each (t rows 0..K and a, b rows 0..K-1 read once: (3K+1) V elements per
request).  The default workload is B=128, K=6, V=151936 bf16 (Qwen-sized
vocabulary), temperature 1, half the requests with identical drafter views.

Prints one JSON line: rows/s (B*(K+1) verified positions per second) as the
value, the achieved HBM bandwidth of the kernel against MI355X's 8 TB/s, and
the CPU oracle timed on the host as a reported baseline.

  python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload 3]
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_26004_amd import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
METRIC = "fused-verify rows/s and achieved HBM GB/s (% of peak), B=128 V=151936 bf16"


def lib_digest():
    """Digest of the library sources: traffic figures measured on other
    sources are not reported."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_26004_amd", "csrc")
    paths = sorted(os.path.join(csrc, n) for n in os.listdir(csrc) if n.endswith((".hip", ".h")))
    for p in paths + [os.path.join(ROOT, "include", "asymspec.h")]:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# ------------------------------------------------------------ CPU baseline --
_CPU_INPUTS = None


def _oracle_worker(reqs):
    import oracle as O
    x = _CPU_INPUTS
    O.fuse_verify(x.t, x.a, x.b, x.draft_tokens, x.draft_probs, x.uniforms,
                  x.temperature, requests=reqs)
    return len(reqs)


def cpu_baseline(x, max_requests):
    """The oracle over the first `max_requests` requests of the workload, in a
    fork pool over requests on the host cores; returns rows/s and cores."""
    global _CPU_INPUTS
    import multiprocessing as mp
    _CPU_INPUTS = x
    n = min(max_requests, x.B)
    cores = max(1, min(16, len(os.sched_getaffinity(0)), n))
    chunks = [list(range(i, n, cores)) for i in range(cores)]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        done = sum(pool.map(_oracle_worker, chunks))
    wall = time.perf_counter() - t0
    rows = done * (x.K + 1)
    return dict(value=rows / wall, unit="rows/s", cores=cores, kind="oracle",
                sample=f"{done} of {x.B} requests ({rows} rows) of the same workload, "
                       f"fp64 NumPy oracle, fork pool of {cores} processes, wall {wall:.2f} s")


# ------------------------------------------------------------------- main --
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--gate", action="store_true", help="also return (D, gamma_eff) per row")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-requests", type=int, default=128)
    ap.add_argument("--copies", type=int, default=2,
                    help="distinct input copies rotated between steps (cold cache)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; the step shards by "
                          "request with no communication (see DESIGN.md)", "n_gpus": args.gpus}))
        sys.exit(2)

    wl = synth.WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    x = synth.workload_inputs(args.workload)
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] generated {wl.name} in {t_gen:.1f} s", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(x, args.cpu_requests)
        print(f"[bench] cpu baseline {cpu['value']:.1f} rows/s on {cpu['cores']} cores",
              file=sys.stderr, flush=True)

    import torch
    import paper_2608_26004_amd as asp
    asp.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def dev_tensor(arr):
        if arr.dtype == np.uint16:
            return torch.from_numpy(arr.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(arr)).to(dev)

    base = [dev_tensor(v) for v in (x.t, x.a, x.b)]
    copies = [base] + [[v.clone() for v in base] for _ in range(max(0, args.copies - 1))]
    d = dev_tensor(x.draft_tokens)
    q = dev_tensor(x.draft_probs)
    u = dev_tensor(x.uniforms)
    tau = dev_tensor(x.temperature)
    B, K, V = x.B, x.K, x.V
    ws = asp.Workspace(dev)
    outs = asp.fuse_verify(*copies[0], d, q, u, tau, return_gate=args.gate, workspace=ws)
    outs = tuple(o for o in outs)

    def step(i):
        return asp.fuse_verify(*copies[i % len(copies)], d, q, u, tau, return_gate=args.gate,
                               workspace=ws, out=outs if args.gate else outs + (None,))

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(i)
        ev[i][1].record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    per = np.array([a.elapsed_time(b) for a, b in ev])
    ms_step = total_ms / args.steps
    kern_ms = float(np.mean(per))
    rows = B * (K + 1)
    nbytes = x.nbytes_read()
    achieved = nbytes / (kern_ms * 1e-3) / 1e9

    acc = outs[0].cpu().numpy()
    traffic = None
    tpath = os.path.join(ROOT, "profiles", f"traffic_{wl.name}.json")
    if os.path.exists(tpath):
        try:
            tj = json.load(open(tpath))
            if tj.get("source_digest") == lib_digest():
                traffic = tj.get("bytes_per_launch")
        except (OSError, ValueError):
            traffic = None

    res = {
        "metric": METRIC,
        "value": rows / (ms_step * 1e-3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "fp32",
        "data": "synthetic (seeded generator; stands in for the paper's datasets)",
        "config": {"workload": wl.name, "B": B, "K": K, "V": V, "rows_per_step": rows,
                   "bytes_per_step": nbytes, "gate_output": bool(args.gate),
                   "input_copies": len(copies), "mean_accept_len": float(acc.mean()),
                   "parallelism": "single GPU"},
        "hbm_GBps": achieved,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel_ms_mean": kern_ms, "kernel_ms_p10": float(np.percentile(per, 10)),
                     "kernel_ms_p90": float(np.percentile(per, 90)),
                     "bytes_per_launch": nbytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
