"""Benchmark of the sparse-linear hot path (SparseDNN, arXiv 2101.07948) on one MI355X.

One step = one sdnn_spmm over the whole measured layer: W 768 x 3072 fp32 at 90 %
unstructured sparsity (uniform random support), B 3072 x 4096 fp32 (batch x tokens),
bias, no activation -- C = W @ B + bias.  Inputs are resident in HBM before timing
starts; steps rotate over enough (B, C) buffer sets (>= 1 GiB) that the 256 MB
Infinity Cache cannot hold a step's operands from the previous visit.

Timing: the step first runs untimed for --settle-ms of wall time (the GPU leaves its
idle clock only after some tens of milliseconds of work: the first 200 steps after an
idle spell run about 25 % slower than the steady state), then --warmup untimed steps,
then --steps timed ones between two HIP events on the launch stream.

Prints one JSON line.  Extra keys: roofline (the kernel against its bounding peak),
cpu_baseline (the CPU oracle's fp32 CSR loop on the host cores), dense comparison
kernel time, warm-cache rate.

Other modes: --suite OUT.md times every configuration (cold/warm, median and p10/p90),
the dense comparison, the row-order ablation, the chained C5 stack in both row spaces,
the sparse 3x3 convolutions, the paper-shaped kernel problems, the CPU oracle at 1/4/all
threads and the machine probes;
--summarize-pmc turns two rocprofv3 counter passes into profiles/traffic_spmm_w0.json.
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
# FP32 vector peak of MI355X: 256 CUs x 128 FP32 FMA lanes per clock x 2 FLOP x 2.4 GHz
# = 157.3 TFLOP/s.  The kernel issues unpacked v_fma_f32; the machine probe measures
# unpacked FMAs alone well above half of this figure, so it is the ceiling they are
# held to.
ALU_PEAK_TFLOPS = 256 * 128 * 2 * 2.4e9 / 1e12
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2101_07948_amd", "csrc", f)
                  for f in ("sdnn_kernels.hip", "sdnn_host.cpp", "sdnn_internal.h",
                            "gen_spmm_asm.py", "spmm_asm_gen.h")]
def traffic_file(layer: str = "w0") -> str:
    return os.path.join(ROOT, "profiles", f"traffic_spmm_{layer}.json")


def kernel_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(layer: str = "w0"):
    """HBM bytes per launch from committed rocprofv3 counters, if taken on this kernel."""
    try:
        t = json.load(open(traffic_file(layer)))
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


def summarize_pmc(fetch_csv, write_csv, K, N, layer="w0"):
    """Per-launch HBM traffic of the sparse kernel from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for the calibration copy (an
    elementwise negation that reads and writes exactly K*N*4 bytes).  Only the sparse
    launches before the copy count: those are the warm-up and timed steps, each on a
    buffer set not touched since it was created."""
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
    out["layer"] = layer
    os.makedirs(os.path.dirname(traffic_file(layer)), exist_ok=True)
    json.dump(out, open(traffic_file(layer), "w"), indent=1)
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
        if el >= budget_s or reps >= 100000:
            break
    per = el / reps
    return {"value": round(2.0 * W.nnz * B.shape[1] / per / 1e9, 3), "unit": "GFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"full measured layer ({W.M}x{W.K}, nnz {W.nnz}, N {B.shape[1]}), "
                      f"{reps} timed calls of the fp32 CSR loop after 1 warm-up "
                      f"({el:.1f} s), {per * 1e3:.1f} ms per call"}


# ---------------------------------------------------------------------------------
# Configuration suite: every workload layer (cold / warm), the dense comparison, the
# Algorithm 1 ablation, the chained C5 stack, the CPU oracle at 1 / 4 / all threads and
# the machine probes.  Writes a markdown report.

def _launch_times(fn, reps):
    """Per-launch milliseconds (an event pair around each call) and the mean over one
    event pair around all reps."""
    import torch
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(reps)]
    for i in range(reps):
        pairs[i][0].record()
        fn(i)
        pairs[i][1].record()
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in pairs)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(reps):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return per, e0.elapsed_time(e1) / reps


def _settle(fn, ms):
    """Runs fn(i) back to back for at least `ms` of wall time (untimed), so that the GPU
    is at its working clock when a timed region starts."""
    import torch
    t0, i = time.perf_counter(), 0
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(20):
            fn(i)
            i += 1
        torch.cuda.synchronize()


def _pct(sorted_vals, q):
    i = min(len(sorted_vals) - 1, max(0, int(round(q * (len(sorted_vals) - 1)))))
    return sorted_vals[i]


def _suite_layers():
    from paper_2101_07948_amd import inputs
    out = []
    def add(label, name, li, N=None, **kw):
        w = inputs.workload(name, N=N, **kw)
        out.append((label, w.layers[li], w.N))
    add("C1 256x256 90% N=64", "c1", 0)
    add("C2 768x768 90% N=1024", "c2", 0)
    add("C3 W1 3072x768 94% lognormal, N=4096, GELU", "c3", 0)
    add("C3 W2 768x3072 94% lognormal, N=4096", "c3", 1)
    add("C4 512x512 80% N=3136, ReLU", "c4", 0)
    add("C5 projection 768x768 97% grouped, N=16384", "c5", 0, num_layers=1)
    add("C5 FFN1 3072x768 97% grouped, N=16384, GELU", "c5", 4, num_layers=1)
    add("C5 FFN2 768x3072 97% grouped, N=16384", "c5", 5, num_layers=1)
    for N in (1024, 4096, 16384):
        add(f"W0 768x3072 90% N={N}", "w0", 0, N=N)
    return out


def _time_layer(plan, L, N, reps=100, warmup=10, cold=True):
    import torch
    dev = torch.device("cuda:0")
    M, K = L.W.M, L.W.K
    bytes_set = 4 * (K * N + M * N)
    nsets = min(64, max(1, math.ceil((1 << 30) / bytes_set))) if cold else 1
    Bs = [torch.randn(K, N, device=dev) for _ in range(nsets)]
    Cs = [torch.empty(M, N, device=dev) for _ in range(nsets)]
    bias = torch.from_numpy(L.bias).to(dev) if L.bias is not None else None
    fn = lambda i: plan.spmm(Bs[i % nsets], Cs[i % nsets], bias, L.epi)
    _settle(fn, 30)
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    per, mean = _launch_times(fn, reps)
    del Bs, Cs
    return per, mean, nsets


def _blas_time(Wd, B, C, reps=20):
    """Mean ms of the vendor FP32 GEMM (torch.mm into C, TF32 off): a comparator only."""
    import torch
    torch.backends.cuda.matmul.allow_tf32 = False
    fn = lambda i: torch.mm(Wd, B, out=C)
    fn(0)
    torch.cuda.synchronize()
    _, mean = _launch_times(fn, reps)
    return mean


def _packing_used(plan, N):
    """(panel height, rho) of the packing plan.spmm runs on at N, as the library reports."""
    rw = plan.launch_shape(N)["panel_rows"]
    info = plan.info
    for k in ("", "tall_", "mid_", "tallest_", "deep_"):
        if info[k + "panel_rows"] == rw:
            return rw, info[k + "rho"]
    return rw, float("nan")


def run_suite(out_path):
    import platform
    import numpy as np
    import torch
    import ctypes
    import oracle
    import paper_2101_07948_amd as sd
    from paper_2101_07948_amd import inputs

    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(0)
    cus = props.multi_processor_count
    lines = [f"# Configuration suite on {props.name} ({cus} CUs)", "",
             f"Command: `python3 bench.py --suite {os.path.relpath(out_path, ROOT)}` "
             f"(kernel hash {kernel_hash()}).", "",
             "Times are `sdnn_spmm` alone, inputs resident in HBM.  Cold: (B, C) buffer sets "
             "rotated (>= 1 GiB in total, at most 64 sets); warm: one set.  Per-launch times "
             "from an event pair around each of 100 launches after 10 warm-up launches; "
             "'mean' is one event pair around 100 back-to-back launches.  % ALU is of "
             f"{ALU_PEAK_TFLOPS:.1f} TFLOP/s (FP32 vector peak), % HBM of {HBM_PEAK_GBS:.0f} GB/s "
             "(algorithmic bytes 8 nnz + 4 KN + 4 MN + 4 M).", "",
             "## Every configuration", "",
             "Launch: panel rows x consumer waves per workgroup, tile columns, as the default "
             "plan picks them.  '256-col us': a plan fixed to 256-column tiles (tile_cols = "
             "256, four packings), cold mean.  'tuned': after sdnn_plan_tune at this N, cold "
             "mean and the shape it recorded.", "",
             "| layer | nnz | launch | rho | cold median us (p10-p90) | cold mean us | "
             "warm median us | GFLOP/s (cold mean) | % ALU | alg GB/s | % HBM | 256-col us | "
             "tuned us (shape) |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    timed = {}
    for label, L, N in _suite_layers():
        W = L.W
        with sd.Plan.from_csr(W) as plan:
            rw, rho = _packing_used(plan, N)
            sh = plan.launch_shape(N)
            per, mean, nsets = _time_layer(plan, L, N)
            wper, _, _ = _time_layer(plan, L, N, cold=False)
            tsh = plan.tune(N, torch.randn(W.K, N, device=dev), torch.empty(W.M, N, device=dev))
            _, tmean, _ = _time_layer(plan, L, N)
        with sd.Plan.from_csr(W, tile_cols=256) as plan:
            _, mean256, _ = _time_layer(plan, L, N)
        flop = 2.0 * W.nnz * N
        ab = 8.0 * W.nnz + 4.0 * W.K * N + 4.0 * W.M * N + 4.0 * W.M
        t = mean * 1e-3
        timed[label] = mean
        lines.append(f"| {label} | {W.nnz} | {rw} x {sh['waves']}, {sh['tile_cols']} | {rho:.2f} | "
                     f"{_pct(per, .5)*1e3:.1f} "
                     f"({_pct(per, .1)*1e3:.1f}-{_pct(per, .9)*1e3:.1f}) | {mean*1e3:.1f} | "
                     f"{_pct(wper, .5)*1e3:.1f} | {flop/t/1e9:.0f} | "
                     f"{100*flop/t/1e12/ALU_PEAK_TFLOPS:.1f} | {ab/t/1e9:.0f} | "
                     f"{100*ab/t/1e9/HBM_PEAK_GBS:.1f} | {mean256*1e3:.1f} | {tmean*1e3:.1f} "
                     f"({tsh['panel_rows']} x {tsh['waves']}, {tsh['tile_cols']}) |")
        print(lines[-1], flush=True)

    lines += ["", "## Dense comparison: the library's FP32 GEMM kernel (same layouts and epilogue) "
              "and the vendor BLAS (torch.mm, FP32, TF32 off; GEMM only)", "",
              "| layer | dense us | dense-equivalent TFLOP/s | % of FP32 peak | "
              "sparse speedup | BLAS us | BLAS TFLOP/s | speedup over BLAS |",
              "|---|---|---|---|---|---|---|---|"]
    for label, L, N in _suite_layers():
        if not (label.startswith("C2") or label.startswith("C3 W1") or label == "W0 768x3072 90% N=4096"):
            continue
        W = L.W
        Wd = torch.from_numpy(W.to_dense()).to(dev)
        B = torch.randn(W.K, N, device=dev)
        C = torch.empty(W.M, N, device=dev)
        bias = torch.from_numpy(L.bias).to(dev) if L.bias is not None else None
        fn = lambda i: sd.dense_gemm(Wd, B, C, bias, L.epi)
        fn(0)
        torch.cuda.synchronize()
        _, dmean = _launch_times(fn, 10)
        bmean = _blas_time(Wd, B, C)
        tf = 2.0 * W.M * W.K * N / (dmean * 1e-3) / 1e12
        btf = 2.0 * W.M * W.K * N / (bmean * 1e-3) / 1e12
        lines.append(f"| {label} | {dmean*1e3:.1f} | {tf:.1f} | {100*tf/ALU_PEAK_TFLOPS:.1f} | "
                     f"{dmean/timed[label]:.2f}x | {bmean*1e3:.1f} | {btf:.1f} | "
                     f"{bmean/timed[label]:.2f}x |")
        print(lines[-1], flush=True)
        del Wd, B, C

    orders = (0, 1, 2, 3, 4, 5)
    lines += ["", "## Row order ablation: identity (permute = 0), Algorithm 1 (1), panel-"
              "balancing (2), panel-union greedy (3), MinHash clustering (4), bin-then-"
              "greedy (5), each with panels of consecutive rows of its order (grouping = "
              "order), against the library's default (Algorithm 1's permutation, balanced "
              "panels); cold mean; rho of the packing the call runs on", "",
              "| layer | " + " | ".join(f"rho {k}" for k in orders) + " | " +
              " | ".join(f"us {k}" for k in orders) + " | default us | speedup of Algorithm 1 "
              "over identity |",
              "|---|" + "---|" * (2 * len(orders) + 2)]
    for label, L, N in _suite_layers():
        if not (label.startswith("C2") or label.startswith("C3") or label.startswith("C5")
                or label == "W0 768x3072 90% N=4096"):
            continue
        res = {}
        for perm in orders:
            with sd.Plan.from_csr(L.W, permute=perm, grouping="order") as plan:
                _, rho = _packing_used(plan, N)
                _, mean, _ = _time_layer(plan, L, N, reps=50)
            res[perm] = (rho, mean)
        with sd.Plan.from_csr(L.W) as plan:
            _, dmean, _ = _time_layer(plan, L, N, reps=50)
        lines.append(f"| {label} | " + " | ".join(f"{res[k][0]:.2f}" for k in orders) + " | "
                     + " | ".join(f"{res[k][1]*1e3:.1f}" for k in orders) + " | "
                     f"{dmean*1e3:.1f} | {res[0][1]/res[1][1]:.2f}x |")
        print(lines[-1], flush=True)

    # the whole C5 stack, chained on the GPU's own activations
    w = inputs.workload("c5")
    t0 = time.perf_counter()
    plans = [sd.Plan.from_csr(L.W) for L in w.layers]
    prep_s = time.perf_counter() - t0
    X0 = torch.randn(w.layers[0].W.K, w.N, device=dev)
    biases = [None if L.bias is None else torch.from_numpy(L.bias).to(dev) for L in w.layers]
    acts = {768: [torch.empty(768, w.N, device=dev) for _ in range(2)],
            3072: [torch.empty(3072, w.N, device=dev)]}
    def forward(_i):
        X, flip = X0, 0
        for L, plan, b in zip(w.layers, plans, biases):
            if L.W.M == 3072:
                Y = acts[3072][0]
            else:
                Y = acts[768][flip]
                flip ^= 1
            plan.spmm(X, Y, b, L.epi)
            X = Y
    forward(0)
    torch.cuda.synchronize()
    _, fmean = _launch_times(forward, 5)
    flop = sum(2.0 * L.W.nnz * w.N for L in w.layers)
    # the same forward captured once as a HIP graph and replayed (the calls allocate nothing
    # and never synchronise); each replay is checked against the eager result bit for bit
    eager_out = acts[768][(sum(1 for L in w.layers if L.W.M != 3072) - 1) % 2].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        forward(0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        forward(0)
    graph_ok = True
    for _ in range(3):
        graph.replay()
        torch.cuda.synchronize()
        last = acts[768][(sum(1 for L in w.layers if L.W.M != 3072) - 1) % 2]
        graph_ok &= bool(torch.equal(last, eager_out))
    _, gmean = _launch_times(lambda _i: graph.replay(), 5)
    del graph
    for p_ in plans:
        p_.close()
    # the same chain in permuted space: every activation stays in its producer's row
    # order and the next plan takes that order as in_perm (the last writes the original)
    plans, prev = [], None
    for i, L in enumerate(w.layers):
        last = i == len(w.layers) - 1
        plans.append(sd.Plan.from_csr(L.W, out_permuted=not last, in_perm=prev))
        prev = None if last else plans[-1].perm
    forward(0)
    torch.cuda.synchronize()
    _, pmean = _launch_times(forward, 5)
    for p_ in plans:
        p_.close()
    lines += ["", "## C5: 12 encoder layers x 6 sparse products, chained (N = 16384)", "",
              f"* {len(w.layers)} products, {flop/1e9:.1f} GFLOP per forward; "
              f"{fmean:.2f} ms per forward = {flop/(fmean*1e-3)/1e12:.1f} TFLOP/s "
              f"(mean of 5 forwards after one warm-up, activations stay on the GPU).",
              f"* Captured once as a HIP graph and replayed: {gmean:.2f} ms per forward = "
              f"{flop/(gmean*1e-3)/1e12:.1f} TFLOP/s (every replay equal to the eager forward "
              f"bit for bit: {'yes' if graph_ok else 'NO'}).",
              f"* In permuted space (each activation left in its producer's Algorithm 1 row "
              f"order, the next plan built with in_perm): {pmean:.2f} ms per forward "
              f"= {flop/(pmean*1e-3)/1e12:.1f} TFLOP/s.",
              f"* Preparation of the {len(w.layers)} plans (validation, Algorithm 1, panel grouping, "
              f"five packings and the 128-column stream, upload): {prep_s:.2f} s on the host."]
    print("\n".join(lines[-4:]), flush=True)

    # sparse 3x3 convolutions shaped like the paper's benchmark (Sec. 4.1): IC, OC in
    # 32..256, images 7..56, padding 1, 90 / 95 %; 16 images per call on the GPU
    lines += ["", "## Sparse 3x3 convolution (stride 1, padding 1), 16 images per call", "",
              "Filters uniform-random at the stated sparsity; input (IC, H, W, 16).  Dense: "
              "the library's comparison GEMM, and the vendor BLAS (torch.mm, FP32), on the "
              "dense filters times a materialised im2col matrix (building it is not timed).", "",
              "| OC x IC, image | sparsity | nnz | us (cold mean) | GFLOP/s | % ALU | "
              "K-split us (auto) | dense us | speedup | BLAS us | speedup over BLAS (best call) |",
              "|---|---|---|---|---|---|---|---|---|---|---|"]
    for OC, IC, HW in ((64, 64, 56), (128, 128, 28), (256, 256, 14), (256, 256, 7)):
        for sp in (0.9, 0.95):
            L = inputs.conv_layer(OC, IC, HW, HW, 16, sp, layer=OC + HW)
            N = HW * HW * 16
            nsets = min(64, max(1, math.ceil((1 << 30) / (4 * (IC + OC) * N))))
            Xs = [torch.from_numpy(L.X).to(dev)] + [torch.randn(IC, HW, HW, 16, device=dev)
                                                     for _ in range(nsets - 1)]
            Cs = [torch.empty(OC, HW, HW, 16, device=dev) for _ in range(nsets)]
            bias = torch.from_numpy(L.bias).to(dev)
            with sd.Plan.from_csr(L.F) as plan:
                fn = lambda i: plan.conv3x3(Xs[i % nsets], Cs[i % nsets], bias)
                _settle(fn, 30)
                _, mean = _launch_times(fn, 100)
            nch = -(-L.F.K // 32)
            with sd.Plan.from_csr(L.F, split_chunks=max(1, -(-nch // 24))) as plan:
                ws = torch.empty(max(plan.workspace_floats(N), 1), device=dev)
                fn = lambda i: plan.conv3x3_split(Xs[i % nsets], Cs[i % nsets], bias, workspace=ws)
                _settle(fn, 30)
                _, smean = _launch_times(fn, 100)
                del ws
            Xp = np.pad(L.X, ((0, 0), (1, 1), (1, 1), (0, 0)))
            cols = np.stack([Xp[:, ky:ky + HW, kx:kx + HW, :] for ky in range(3) for kx in range(3)],
                            axis=1).reshape(IC * 9, N)
            Bd = torch.from_numpy(np.ascontiguousarray(cols)).to(dev)
            Wd = torch.from_numpy(L.F.to_dense()).to(dev)
            Cd = torch.empty(OC, N, device=dev)
            dfn = lambda i: sd.dense_gemm(Wd, Bd, Cd, bias)
            dfn(0)
            torch.cuda.synchronize()
            _, dmean = _launch_times(dfn, 10)
            bmean = _blas_time(Wd, Bd, Cd)
            flop = 2.0 * L.F.nnz * N
            best = min(mean, smean)
            lines.append(f"| {OC} x {IC}, {HW}x{HW} | {int(sp*100)} % | {L.F.nnz} | {mean*1e3:.1f} | "
                         f"{flop/(mean*1e-3)/1e9:.0f} | {100*flop/(mean*1e-3)/1e12/ALU_PEAK_TFLOPS:.1f} | "
                         f"{smean*1e3:.1f} | {dmean*1e3:.1f} | {dmean/mean:.2f}x | {bmean*1e3:.1f} | "
                         f"{bmean/best:.2f}x |")
            print(lines[-1], flush=True)
            del Xs, Cs, Bd, Wd, Cd

    # K-split calls on the grids that leave CUs idle: runs of a tile's K-segments get
    # their own workgroups (plans with split_chunks), and a reduction kernel forms C
    counts = (2, 4, 8)
    lines += ["", "## K-split calls (sdnn_spmm_split / sdnn_conv3x3_split) on small grids", "",
              "Unsplit: the plain call on a plain plan.  Split: a plan with about 16-24 "
              "K-segments (split_chunks = S chunks of 32 rows each), called with the "
              "library's choice of workgroups along K (auto: the cost model) and with forced "
              "counts, on the tile width the launch picks; 'tuned': after sdnn_plan_tune at "
              "this N (products only), which also times every count on both tile widths "
              "(workgroups along K, tile columns); cold means of 50 launches, reduction "
              "included.", "",
              "| problem | column tiles x panels | unsplit us | S | auto us | " +
              " | ".join(f"{k} along K us" for k in counts) + " | auto speedup | tuned us |",
              "|---|---|---|---|---|" + "---|" * len(counts) + "---|---|"]
    split_cases = [("W0 768x3072 90% N=1024", inputs.workload("w0", N=4).layers[0].W, 1024, None),
                   ("W0 768x3072 90% N=4096", inputs.workload("w0", N=4).layers[0].W, 4096, None),
                   ("C2 768x768 90% N=1024", inputs.workload("c2", N=4).layers[0].W, 1024, None),
                   ("S 2048 90% N=256", inputs.s_layer(2048, 2048, 0.9).W, 256, None),
                   ("S 2048 70% N=128", inputs.s_layer(2048, 2048, 0.7).W, 128, None),
                   ("S 1024 90% N=256", inputs.s_layer(1024, 1024, 0.9).W, 256, None),
                   ("conv 256 x 256, 14x14", None, 14, 256),
                   ("conv 256 x 256, 7x7", None, 7, 256),
                   ("conv 512 x 512, 7x7", None, 7, 512)]
    for label, W, n_or_hw, ch in split_cases:
        if ch is None:
            N = n_or_hw
            B = torch.randn(W.K, N, device=dev)
            C = torch.empty(W.M, N, device=dev)
            call = lambda p, ws, k: (lambda i: p.spmm(B, C) if ws is None else
                                     p.spmm_split(B, C, workspace=ws, splits=k))
        else:
            HW = n_or_hw
            L = inputs.conv_layer(ch, ch, HW, HW, 16, 0.9, layer=ch + HW)
            W, N = L.F, HW * HW * 16
            X = torch.from_numpy(L.X).to(dev)
            C = torch.empty(ch, HW, HW, 16, device=dev)
            call = lambda p, ws, k: (lambda i: p.conv3x3(X, C) if ws is None else
                                     p.conv3x3_split(X, C, workspace=ws, splits=k))
        nch = -(-W.K // 32)
        S = max(1, -(-nch // 24)) if nch >= 48 else max(1, nch // 16)
        def timed_mean(p, ws, k=0):
            fn = call(p, ws, k)
            _settle(fn, 30)
            return _launch_times(fn, 50)[1]
        with sd.Plan.from_csr(W) as plan:
            base = timed_mean(plan, None)
            rw, _ = _packing_used(plan, N)
            tile = plan.launch_shape(N)["tile_cols"] if ch is None else 256
        grid = f"{-(-N // tile)} x {-(-W.M // rw)} ({rw}-row, {tile}-col)"
        with sd.Plan.from_csr(W, split_chunks=S) as plan:
            ws = torch.empty(max(plan.workspace_floats(N), 1), device=dev)
            auto = timed_mean(plan, ws, 0)
            forced = [timed_mean(plan, ws, k) for k in counts]
            segs = plan.info["splits"]
            tuned = "-"
            if ch is None:
                plan.tune(N, B, C)
                tuned = f"{timed_mean(plan, ws, 0)*1e3:.1f} ({plan.split_runs(N)} along K)"
        lines.append(f"| {label} | {grid} | {base*1e3:.1f} | {S} ({segs} seg) | {auto*1e3:.1f} | " +
                     " | ".join(f"{t_*1e3:.1f}" for t_ in forced) + f" | {base/auto:.2f}x | {tuned} |")
        print(lines[-1], flush=True)
        del C

    # the paper's kernel problems (Sec. 4.1): square M = K from 256 to 2048, 70-95 %
    # sparse by magnitude threshold of a Gaussian matrix, three batch widths
    lines += ["", "## Paper-shaped kernel problems (Sec. 4.1): M = K, Gaussian magnitude threshold", "",
              "Each cell: sparse GFLOP/s (cold mean of 50 launches) and, in brackets, the speedup "
              "over the library's dense kernel and over the vendor BLAS (torch.mm, FP32) on a "
              "dense W of the same shape.", "",
              "| M = K | N | " + " | ".join(f"{int(sp*100)} %" for sp in inputs.S_SPARSITIES) +
              " | dense TFLOP/s | BLAS TFLOP/s |",
              "|---|---|" + "---|" * len(inputs.S_SPARSITIES) + "---|---|"]
    for MK in (256, 512, 1024, 2048):
        for N in (128, 512, 2048):
            B = torch.randn(MK, N, device=dev)
            C = torch.empty(MK, N, device=dev)
            Wd = torch.randn(MK, MK, device=dev)
            dfn = lambda i: sd.dense_gemm(Wd, B, C)
            dfn(0)
            torch.cuda.synchronize()
            _, dmean = _launch_times(dfn, 10)
            bmean = _blas_time(Wd, B, C)
            cells = []
            for sp in inputs.S_SPARSITIES:
                L = inputs.s_layer(MK, MK, sp)
                with sd.Plan.from_csr(L.W) as plan:
                    _, mean, _ = _time_layer(plan, L, N, reps=50)
                cells.append(f"{2.0 * L.W.nnz * N / (mean * 1e-3) / 1e9:.0f} "
                             f"({dmean / mean:.1f}x, {bmean / mean:.1f}x)")
            lines.append(f"| {MK} | {N} | " + " | ".join(cells) +
                         f" | {2.0 * MK * MK * N / (dmean * 1e-3) / 1e12:.1f} | "
                         f"{2.0 * MK * MK * N / (bmean * 1e-3) / 1e12:.1f} |")
            print(lines[-1], flush=True)
            del B, C, Wd

    # CPU oracle (fp32 CSR loop) at 1, 4 and all threads on W0 at N = 4096
    wl = inputs.workload("w0")
    L = wl.layers[0]
    cpu_model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                cpu_model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    lines += ["", f"## CPU oracle (fp32 CSR loop, OpenMP over rows) on W0, N = 4096", "",
              f"Host: {cpu_model}; {avail} CPUs available to the process "
              f"({platform.machine()}).  Median of 5 calls after 1 warm-up.", "",
              "| threads | ms per call | GFLOP/s | GPU speedup (cold mean) |", "|---|---|---|---|"]
    out = np.empty((L.W.M, wl.N), dtype=np.float32)
    default_threads = oracle.num_threads()
    for T in sorted({1, 4, default_threads}):
        oracle.set_num_threads(T)
        oracle.spmm_f32(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, wl.B, L.bias, "none", out=out)
        ts = []
        for _ in range(5):
            t0 = time.perf_counter()
            oracle.spmm_f32(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, wl.B, L.bias, "none", out=out)
            ts.append(time.perf_counter() - t0)
        med = sorted(ts)[2]
        gf = 2.0 * L.W.nnz * wl.N / med / 1e9
        lines.append(f"| {T} | {med*1e3:.1f} | {gf:.1f} | "
                     f"{med/(timed['W0 768x3072 90% N=4096']*1e-3):.0f}x |")
        print(lines[-1], flush=True)
    oracle.set_num_threads(default_threads)

    # machine probes next to the datasheet peaks
    plib = ctypes.CDLL(os.path.join(ROOT, "paper_2101_07948_amd", "libsdnn_probes.so"))
    plib.sdnn_probe_out_floats.restype = ctypes.c_int64
    for f in (plib.sdnn_probe_fma, plib.sdnn_probe_lds_read):
        f.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
        f.restype = ctypes.c_int32
    pout = torch.empty(int(plib.sdnn_probe_out_floats()), device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    def probe(f, iters):
        assert f(iters, ctypes.c_void_p(pout.data_ptr()), stream) == 0
    probe(plib.sdnn_probe_fma, 100)
    torch.cuda.synchronize()
    fi = 20000
    _, fms = _launch_times(lambda i: probe(plib.sdnn_probe_fma, fi), 5)
    fma_tf = pout.numel() * fi * 16 * 2 / (fms * 1e-3) / 1e12
    li = 4000
    _, lms = _launch_times(lambda i: probe(plib.sdnn_probe_lds_read, li), 5)
    lds_bytes = 256 * 16 * li * 8 * 1024
    lds_cu = lds_bytes / 256 / (lms * 1e-3)
    x = torch.empty(1 << 28, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    _, cms = _launch_times(lambda i: y.copy_(x), 10)
    hbm = 2.0 * x.numel() * 4 / (cms * 1e-3) / 1e9
    del x, y
    lines += ["", "## Machine probes (measured next to the datasheet peaks)", "",
              "| probe | measured | datasheet | fraction |", "|---|---|---|---|",
              f"| HBM stream copy (1 GiB read + 1 GiB write) | {hbm:.0f} GB/s | "
              f"{HBM_PEAK_GBS:.0f} GB/s | {hbm/HBM_PEAK_GBS:.2f} |",
              f"| unpacked FP32 FMA loop (v_fmaak_f32, 8 chains per thread, 16 waves per CU) | "
              f"{fma_tf:.1f} TFLOP/s | {ALU_PEAK_TFLOPS:.1f} TFLOP/s | {fma_tf/ALU_PEAK_TFLOPS:.2f} |",
              f"| LDS ds_read_b128 of 1 KB rows (16 waves per CU) | {lds_cu/1e9:.0f} GB/s per CU "
              f"= {lds_cu/2.4e9:.0f} B/clk at 2.4 GHz | 512 B/clk: one 4-byte B value per "
              f"FMA at the FP32 peak | {lds_cu/2.4e9/512:.2f} |"]
    print("\n".join(lines[-5:]), flush=True)
    text = "\n".join(lines) + "\n"
    os.makedirs(os.path.dirname(os.path.abspath(out_path)), exist_ok=True)
    open(out_path, "w").write(text)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-ms", type=float, default=300.0,
                    help="untimed run of the step before the warm-up steps, in ms of wall time")
    ap.add_argument("--N", type=int, default=4096)
    ap.add_argument("--layer", default="w0",
                    help="workload layer to time: w0 (the measured layer; default), c2, c3_w1, "
                         "c3_w2, c4, c5_proj, c5_ffn1, c5_ffn2 (counter passes on other layers)")
    ap.add_argument("--grouping", default="auto", choices=["auto", "order", "balanced"],
                    help="panel grouping of the plan (counter passes comparing groupings)")
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
                         "profiles/traffic_spmm_<layer>.json")
    ap.add_argument("--suite", metavar="OUT_MD",
                    help="time every configuration, the dense comparison, the row-order "
                         "ablation, the chained C5 stack, the convolutions, the paper-shaped "
                         "kernel problems, the CPU oracle at 1/4/all threads and the machine "
                         "probes; write a markdown report to OUT_MD")
    args = ap.parse_args()
    if args.suite:
        run_suite(args.suite)
        return
    if args.summarize_pmc:
        Ks = {"w0": 3072, "c2": 768, "c3_w1": 768, "c3_w2": 3072, "c4": 512, "c5_proj": 768,
              "c5_ffn1": 768, "c5_ffn2": 3072}
        Ns = {"c2": 1024, "c3_w1": 4096, "c3_w2": 4096, "c4": 3136, "c5_proj": 16384,
              "c5_ffn1": 16384, "c5_ffn2": 16384}
        summarize_pmc(*args.summarize_pmc, K=Ks[args.layer], N=Ns.get(args.layer, args.N),
                      layer=args.layer)
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
    layer_of = {"w0": ("w0", 0, {}), "c2": ("c2", 0, {}), "c3_w1": ("c3", 0, {}),
                "c3_w2": ("c3", 1, {}), "c4": ("c4", 0, {}), "c5_proj": ("c5", 0, {"num_layers": 1}),
                "c5_ffn1": ("c5", 4, {"num_layers": 1}), "c5_ffn2": ("c5", 5, {"num_layers": 1})}
    if args.layer not in layer_of:
        sys.exit(f"unknown --layer {args.layer}")
    wname, li, kw = layer_of[args.layer]
    w = inputs.workload(wname, N=None if args.layer != "w0" else args.N, **kw)
    L = w.layers[li]
    if li > 0:  # a later layer of a chain: a synthetic input of its own shape
        w.B = inputs.dense_B(L.W.K, w.N, inputs.CFG_TEST, 4242)
    W, N, M, K = L.W, w.N, L.W.M, L.W.K
    plan = sd.Plan.from_csr(W, grouping=args.grouping)
    info = plan.info

    bytes_set = 4 * (K * N + M * N)
    nsets = 1 if args.warm else max(1, math.ceil((1 << 30) / bytes_set))
    Bs = [torch.from_numpy(w.B).to(dev)]
    for _ in range(nsets - 1):
        Bs.append(Bs[0].clone())
    Cs = [torch.empty((M, N), device=dev) for _ in range(nsets)]
    bias = None if L.bias is None else torch.from_numpy(L.bias).to(dev)
    torch.cuda.synchronize()

    epi = L.epi
    _settle(lambda i: plan.spmm(Bs[i % nsets], Cs[i % nsets], bias, epi), args.settle_ms)
    for i in range(args.warmup):
        plan.spmm(Bs[i % nsets], Cs[i % nsets], bias, epi)
    torch.cuda.synchronize()

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(args.steps):
        plan.spmm(Bs[i % nsets], Cs[i % nsets], bias, epi)
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
    traffic = measured_traffic(args.layer)
    roof["traffic"] = traffic
    roof["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 4)
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
            plan.spmm(Bs[0], Cs[0], bias, epi)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(50):
            plan.spmm(Bs[0], Cs[0], bias, epi)
        e1.record()
        torch.cuda.synchronize()
        warm_ms = e0.elapsed_time(e1) / 50

    dense = None
    if not args.no_dense:
        Wd = torch.from_numpy(W.to_dense()).to(dev)
        Cd = torch.empty((M, N), device=dev)
        reps = 20

        def timed(fn):  # 100 ms settle, then the mean of `reps` back-to-back calls
            _settle(lambda i: fn(), 100.0)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        dms = timed(lambda: sd.dense_gemm(Wd, Bs[0], Cd, bias))
        dense = {"ms": round(dms, 4), "tflops": round(2.0 * M * K * N / (dms * 1e-3) / 1e12, 2),
                 "frac_of_fp32_peak": round(2.0 * M * K * N / (dms * 1e-3) / 1e12 / ALU_PEAK_TFLOPS, 4),
                 "sparse_speedup": round(dms / ms, 2)}
        # the vendor BLAS on the same dense product (torch.mm in FP32, TF32 off): context
        # next to the library's own dense kernel, not the comparison the target names
        torch.backends.cuda.matmul.allow_tf32 = False
        bms = timed(lambda: torch.mm(Wd, Bs[0], out=Cd))
        dense["vendor_blas"] = {"ms": round(bms, 4),
                                "tflops": round(2.0 * M * K * N / (bms * 1e-3) / 1e12, 2),
                                "sparse_speedup": round(bms / ms, 2)}
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
        "settle_ms": args.settle_ms,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": ("w0: W 768x3072 fp32, 90% uniform-random sparsity, "
                                f"B 3072x{N} fp32, bias, no activation") if args.layer == "w0"
                   else f"{args.layer}: W {M}x{K} fp32 (nnz {W.nnz}), B {K}x{N} fp32, bias, {L.epi}",
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
