#!/usr/bin/env python3
"""Benchmark of the sparse-gradient hot path on one MI355X.

A step is one pass of the whole path over the workload's inputs, already
resident in HBM: for the default SpMM-gradient workload (CSR A 100,000 x
100,000 with 1M power-law nnz, B 100,000 x 64) that is the forward product
C = A B, the SDDMM gradient dA on A's pattern with the fused loss
1/2 ||C||^2, and the transposed product dB = A^T C (nsd_loss_frob_spmm).
The pattern-only preprocessing (row expansion, CSR -> CSC) is timed
separately.

Prints one JSON line with the metric (gradient nonzeros per second), the
roofline of the dominant kernel (algorithmic bytes / its average launch
duration from HIP events, against 8 TB/s), and the fp64 oracle timed on the
host as a reported CPU baseline.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="spmm", choices=["spmm", "gnn", "spmv"])
    ap.add_argument("--size", default="full")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + steps only (for rocprofv3), no JSON line")
    return ap.parse_args()


def source_digest():
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2303_07030_amd", "csrc"))):
        with open(os.path.join(ROOT, "paper_2303_07030_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    s = re.search(r"source_digest:\s*([0-9a-f]+)", text)
    if not m or not s or s.group(1) != source_digest():
        return None
    return float(m.group(1))


class Events:
    def __init__(self, torch):
        self.torch = torch

    def time(self, fn, reps):
        t = self.torch
        s, e = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(reps):
            fn()
        e.record()
        e.synchronize()
        return s.elapsed_time(e) / reps


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "design is described, not built", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2303_07030_amd import nsd, synth
    from paper_2303_07030_amd.operand import DeviceCsr

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ev = Events(torch)

    d = synth.make(args.workload, args.size)
    nrows, ncols = d["nrows"], d["ncols"]
    nnz = len(d["colind"])
    k = d.get("k", 1)

    # ---- preprocessing (pattern only), timed separately
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    A = DeviceCsr(nrows, ncols, d["rowptr"], d["colind"], d["val"], device=dev)
    torch.cuda.synchronize()
    prep_ms_incl_upload = (time.perf_counter() - t0) * 1e3
    csc_ms = ev.time(lambda: A.build_csc(), 3)

    ws = A.workspace(k)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    dA = torch.empty(nnz, dtype=torch.float32, device=dev)
    if args.workload == "spmm":
        B = torch.from_numpy(d["B"]).to(dev)
        C = torch.empty((nrows, k), dtype=torch.float32, device=dev)
        dB = torch.empty((ncols, k), dtype=torch.float32, device=dev)

        def step():
            nsd.nsd_loss_frob_spmm(A.desc, A.csc, B, k, 1.0, C, loss, dA, dB, ws)

        kernels = {
            "spmm_forward": (lambda: nsd.nsd_spmm(A.desc, B, k, C, ws),
                             4 * (3 * nnz) + 4 * (nrows + ncols) * k),
            "sddmm_grad": (lambda: nsd.nsd_sddmm(A.desc, C, B, k, 1.0, dA),
                           4 * (2 * nnz + nnz) + 4 * (nrows + ncols) * k),
            "spmm_t_grad": (lambda: nsd.nsd_spmm_t(A.desc, A.csc, C, k, 1.0, dB, ws),
                            4 * (3 * nnz + nnz) + 4 * (nrows + ncols) * k),
        }
    elif args.workload == "gnn":
        H = torch.from_numpy(d["H"]).to(dev)
        G = torch.from_numpy(d["G"]).to(dev)
        dH = torch.empty((ncols, k), dtype=torch.float32, device=dev)

        def step():
            nsd.nsd_loss_bilinear(A.desc, A.csc, H, G, k, 1.0, loss, dA, dH, ws)

        kernels = {
            "sddmm_grad": (lambda: nsd.nsd_sddmm(A.desc, G, H, k, 1.0, dA),
                           4 * (3 * nnz) + 4 * (nrows + ncols) * k),
            "spmm_t_grad": (lambda: nsd.nsd_spmm_t(A.desc, A.csc, G, k, 1.0, dH, ws),
                            4 * (4 * nnz) + 4 * (nrows + ncols) * k),
        }
    else:
        x = torch.from_numpy(d["x"]).to(dev)
        dx = torch.empty(ncols, dtype=torch.float32, device=dev)

        def step():
            nsd.nsd_loss_sum_spmv(A.desc, A.csc, x, 1.0, loss, dA, dx, ws)

        kernels = {
            "spmm_t_grad": (lambda: nsd.nsd_spmm_t(A.desc, A.csc, None, 1, 1.0, dx, ws),
                            4 * (4 * nnz) + 4 * ncols),
        }

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.profile_only:
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        return

    # ---- timed region: exactly K steps
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / args.steps

    # ---- per-kernel durations (HIP events on the launching stream)
    per_kernel = {}
    for name, (fn, algo_bytes) in kernels.items():
        fn()
        ms = ev.time(fn, max(args.steps, 20))
        per_kernel[name] = {"ms": round(ms, 5), "algo_bytes": int(algo_bytes),
                            "GBps": round(algo_bytes / (ms * 1e-3) / 1e9, 1)}
    dom = max(per_kernel, key=lambda n: per_kernel[n]["ms"])
    dk = per_kernel[dom]
    traffic = committed_traffic(dom, args.workload)
    roofline = {
        "bound": "hbm", "kernel": dom,
        "achieved": dk["GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(dk["GBps"] / HBM_PEAK_GBS, 4),
        "traffic": traffic,
    }

    # ---- the oracle on the host, a reported baseline
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, d, nnz)

    out = {
        "metric": "gradient nonzeros/sec (forward+backward)",
        "value": round(nnz / (ms_per_step * 1e-3), 1),
        "unit": "nnz/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": workload_name(args.workload, d), "nnz": nnz, "k": k,
                   "nrows": nrows, "ncols": ncols},
        "roofline": roofline,
        "kernels": per_kernel,
        "preprocess_ms": {"csr_to_csc": round(csc_ms, 4),
                          "upload_expand_csc": round(prep_ms_incl_upload, 2)},
        "cpu_baseline": cpu,
        "source_digest": source_digest(),
    }
    print(json.dumps(out))


def workload_name(w, d):
    if w == "spmm":
        return "spmm_grad_100k_1M_zipf1.1_k64"
    if w == "gnn":
        return "gnn_bilinear_2.4M_60M_zipf1.05_k256"
    return "spmv_sum_1k_10k"


def cpu_baseline(args, d, nnz):
    """The fp64 oracle, unchanged, on this host: whole passes of the same
    workload (DOK build + every output) repeated for about cpu_seconds."""
    import oracle
    nrows, ncols = d["nrows"], d["ncols"]
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(d["rowptr"]))
    k = d.get("k", 1)

    def one_pass():
        D = oracle.Dok((nrows, ncols), (rows, d["colind"]), d["val"])
        if args.workload == "spmm":
            Cr, Cm = oracle.spmm(D, d["B"], k)
            oracle.loss_half_sq(Cr, Cm)
            oracle.sddmm(D, Cr, d["B"], k, rows, d["colind"], Xmag=Cm)
            oracle.spmm_t(D, Cr, k, Gmag=Cm)
        elif args.workload == "gnn":
            oracle.loss_bilinear(D, d["G"], d["H"], k)
            oracle.sddmm(D, d["G"], d["H"], k, rows, d["colind"])
            oracle.spmm_t(D, d["G"], k)
        else:
            oracle.loss_sum_spmv(D, d["x"])
            oracle.sddmm(D, None, d["x"].reshape(-1, 1), 1, rows, d["colind"])
            oracle.spmm_t(D, None, 1)

    passes, t0 = 0, time.perf_counter()
    while True:
        one_pass()
        passes += 1
        el = time.perf_counter() - t0
        if el >= args.cpu_seconds or passes >= 1000:
            break
    per_pass = el / passes
    return {"value": round(nnz / per_pass, 1), "unit": "nnz/s", "cores": 1, "kind": "oracle",
            "sample": f"{passes} full pass(es) of the {args.workload} workload "
                      f"({nnz} nnz; DOK build + all outputs), {el:.1f} s single-threaded",
            "host_cpus_visible": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    main()
