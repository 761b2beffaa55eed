"""Benchmark of the sparse-linear hot path (SparseDNN, arXiv 2101.07948) on one MI355X.

One step = one sdnn_spmm over the whole measured layer: W 768 x 3072 fp32 at 90 %
unstructured sparsity (uniform random support), B 3072 x 4096 fp32 (batch x tokens),
bias, no activation -- C = W @ B + bias.  Inputs are resident in HBM before timing
starts; steps rotate over enough (B, C) buffer sets (>= 1 GiB) that the 256 MB
Infinity Cache cannot hold a step's operands from the previous visit.

Prints one JSON line.  Extra keys: roofline (the kernel against its bounding peak),
cpu_baseline (the CPU oracle's fp32 CSR loop on the host cores), dense comparison
kernel time, warm-cache rate.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, GB/s
# FP32 FMA issued as single (unpacked) v_fma_f32: 256 CUs x 4 SIMD x 16 lanes x 2 FLOP
# x 2.4 GHz.  Packed FP32 (157.3 TFLOP/s) is not used by this build.
ALU_PEAK_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12
PACKED_FP32_PEAK_TFLOPS = 157.3
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2101_07948_amd", "csrc", f)
                  for f in ("sdnn_kernels.hip", "sdnn_host.cpp", "sdnn_internal.h",
                            "gen_spmm_asm.py", "spmm_asm_gen.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_spmm_w0.json")


def kernel_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch from committed rocprofv3 counters, if taken on this kernel."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    return t.get("bytes_per_launch") if t.get("kernel_hash") == kernel_hash() else None


def _pmc_rows(path, counter):
    import csv
    rows = []
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") == counter:
            rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    return sorted(rows)


def summarize_pmc(fetch_csv, write_csv, N):
    """Per-launch HBM traffic of the sparse kernel from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for the calibration copy (an
    elementwise negation that reads and writes exactly K*N*4 bytes).  Only the sparse
    launches before the copy count: those are the warm-up and timed steps, each on a
    buffer set not touched since it was created."""
    K = 3072
    copy_bytes = 4.0 * K * N
    out = {"kernel_hash": kernel_hash(), "copy_bytes_each_way": copy_bytes}
    for name, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        rows = _pmc_rows(path, counter)
        copy = [(d, v) for d, k, v in rows if "elementwise" in k.lower() and "neg" in k.lower()]
        if not copy:
            raise SystemExit(f"{path}: no calibration copy dispatch")
        spmm = [v for d, k, v in rows if "spmm_panel_kernel" in k and d < copy[0][0]]
        if not spmm:
            raise SystemExit(f"{path}: no sparse-kernel dispatch before the calibration copy")
        factor = copy_bytes / (copy[0][1] * 1024.0)   # true bytes per counted byte
        out[name + "_launches"] = len(spmm)
        out[name + "_kib_counted_per_launch"] = sum(spmm) / len(spmm)
        out[name + "_copy_kib_counted"] = copy[0][1]
        out[name + "_calibration_factor"] = factor
        out[name + "_bytes_per_launch"] = sum(spmm) / len(spmm) * 1024.0 * factor
    out["bytes_per_launch"] = out["fetch_bytes_per_launch"] + out["write_bytes_per_launch"]
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
    print(json.dumps(out))


def cpu_baseline(W, B, bias, budget_s: float):
    import numpy as np
    import oracle
    out = np.empty((W.M, B.shape[1]), dtype=np.float32)
    oracle.spmm_f32(W.row_ptr, W.col_idx, W.values, W.K, B, bias, "none", out=out)  # warm-up
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.spmm_f32(W.row_ptr, W.col_idx, W.values, W.K, B, bias, "none", out=out)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 50:
            break
    per = el / reps
    return {"value": round(2.0 * W.nnz * B.shape[1] / per / 1e9, 3), "unit": "GFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"full measured layer ({W.M}x{W.K}, nnz {W.nnz}, N {B.shape[1]}), "
                      f"{reps} timed calls of the fp32 CSR loop after 1 warm-up, "
                      f"{per * 1e3:.1f} ms per call"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--N", type=int, default=4096)
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of CPU-oracle timing (0 = skip the cpu_baseline leg)")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense comparison kernel")
    ap.add_argument("--warm", action="store_true", help="reuse one buffer set (cache-warm)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after timing, run one plain elementwise copy of B (known bytes) so a "
                         "counter pass can calibrate FETCH_SIZE / WRITE_SIZE")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE) of a --calib-copy run into per-launch HBM bytes and write "
                         f"{os.path.relpath(TRAFFIC_FILE, ROOT)}")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, N=args.N)
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested); the operator "
              "shards over N with no exchange, so per-GPU throughput is the N=1 figure.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2101_07948_amd as sd
    from paper_2101_07948_amd import inputs

    dev = torch.device("cuda:0")
    w = inputs.workload("w0", N=args.N)
    L = w.layers[0]
    W, N, M, K = L.W, w.N, L.W.M, L.W.K
    plan = sd.Plan.from_csr(W)
    info = plan.info

    bytes_set = 4 * (K * N + M * N)
    nsets = 1 if args.warm else max(1, math.ceil((1 << 30) / bytes_set))
    Bs = [torch.from_numpy(w.B).to(dev)]
    for _ in range(nsets - 1):
        Bs.append(Bs[0].clone())
    Cs = [torch.empty((M, N), device=dev) for _ in range(nsets)]
    bias = torch.from_numpy(L.bias).to(dev)
    torch.cuda.synchronize()

    for i in range(args.warmup):
        plan.spmm(Bs[i % nsets], Cs[i % nsets], bias)
    torch.cuda.synchronize()

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(args.steps):
        plan.spmm(Bs[i % nsets], Cs[i % nsets], bias)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps

    flop = 2.0 * W.nnz * N
    alg_bytes = 8.0 * W.nnz + 4.0 * K * N + 4.0 * M * N + 4.0 * M
    t = ms * 1e-3
    gflops = flop / t / 1e9
    gbs = alg_bytes / t / 1e9
    t_alu = flop / (ALU_PEAK_TFLOPS * 1e12)
    t_hbm = alg_bytes / (HBM_PEAK_GBS * 1e9)
    if t_alu >= t_hbm:
        roof = {"bound": "alu", "achieved": round(flop / t / 1e12, 3),
                "peak": round(ALU_PEAK_TFLOPS, 1), "unit": "TFLOP/s",
                "frac": round(flop / t / 1e12 / ALU_PEAK_TFLOPS, 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    traffic = measured_traffic()
    roof["traffic"] = traffic
    roof["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 4)
    roof["frac_of_packed_fp32_peak"] = round(flop / t / 1e12 / PACKED_FP32_PEAK_TFLOPS, 4)
    roof["alg_bytes"] = int(alg_bytes)
    roof["flop"] = int(flop)

    if args.calib_copy:  # plain copy of known size for counter calibration
        X = torch.empty_like(Bs[0])
        torch.neg(Bs[0], out=X)
        torch.cuda.synchronize()
        del X

    # cache-warm rate on one buffer set (context only)
    warm_ms = None
    if not args.warm:
        for _ in range(5):
            plan.spmm(Bs[0], Cs[0], bias)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(50):
            plan.spmm(Bs[0], Cs[0], bias)
        e1.record()
        torch.cuda.synchronize()
        warm_ms = e0.elapsed_time(e1) / 50

    dense = None
    if not args.no_dense:
        Wd = torch.from_numpy(W.to_dense()).to(dev)
        Cd = torch.empty((M, N), device=dev)
        sd.dense_gemm(Wd, Bs[0], Cd, bias)
        torch.cuda.synchronize()
        reps = 10
        e0.record()
        for _ in range(reps):
            sd.dense_gemm(Wd, Bs[0], Cd, bias)
        e1.record()
        torch.cuda.synchronize()
        dms = e0.elapsed_time(e1) / reps
        dense = {"ms": round(dms, 4), "tflops": round(2.0 * M * K * N / (dms * 1e-3) / 1e12, 2),
                 "sparse_speedup": round(dms / ms, 2)}
        del Wd, Cd

    cpu = None
    if args.cpu_budget > 0:
        cpu = cpu_baseline(W, w.B, L.bias, args.cpu_budget)

    rec = {
        "metric": "sparse-linear GFLOP/s (2*nnz*N/t), 768x3072 W at 90% sparsity",
        "value": round(gflops, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "w0: W 768x3072 fp32, 90% uniform-random sparsity, "
                               f"B 3072x{N} fp32, bias, no activation",
                   "M": M, "K": K, "N": N, "nnz": W.nnz, "panel_rows": info["panel_rows"],
                   "rho": round(info["rho"], 4), "buffer_sets": nsets},
        "alg_GBps": round(gbs, 1),
        "roofline": roof,
        "cpu_baseline": cpu,
        "dense_kernel": dense,
        "warm_ms_per_step": None if warm_ms is None else round(warm_ms, 5),
        "kernel_hash": kernel_hash(),
    }
    print(json.dumps(rec))
    plan.close()


if __name__ == "__main__":
    main()
