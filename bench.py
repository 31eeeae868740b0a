"""Benchmark: one sparse-conv layer (Map + GMaS) per step on one MI355X.

A step runs the whole hot path on one seeded LiDAR-like scene (about 120k voxels,
submanifold K = 3, C_in = C_out = 64, float16): coordinate bounds, key packing and
radix sort, the double-traversed binary search with pair compaction (Map), then
metadata tables, gather, grouped MFMA GEMMs and scatter (GMaS).  Inputs are
resident in HBM before timing starts.  Prints one JSON line.

Per-phase times come from HIP events the library records on the launch stream
during the timed steps; the dominant kernel's algorithmic bytes (or flops) per
launch divided by its mean duration give the roofline figure.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparse-conv layer ms (Map + GMaS split); Map GB/s, GEMM TFLOP/s vs peak"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", type=int, default=1, help="scene recipe (1 = LiDAR 120k, 3 = indoor 300k)")
    p.add_argument("--channels", type=int, default=None, help="channel width for recipe 3")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--grouping", type=int, default=None)
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2401_06145_amd import binding as B
    from paper_2401_06145_amd import scenes

    dev = torch.device("cuda:0")
    wl = scenes.workload(args.workload, args.channels)
    L = wl.layers[0]
    coords_np = wl.coords
    n = len(coords_np)
    x_np = scenes.features(n, L.c_in, L.dtype, 2000 + args.workload)
    w_np = scenes.weights(L.K, L.c_in, L.c_out, L.dtype, 3000 + args.workload)
    tdt = B.TORCH_DTYPES[L.dtype]
    coords = torch.from_numpy(coords_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    w = torch.from_numpy(w_np).to(dev)
    mode = B.MODES[L.mode]
    opt = B.Options.make(grouping=args.grouping) if args.grouping is not None else None
    map_ws = torch.empty(B.spconv_map_workspace_bytes(n, 0, L.K, mode, opt), dtype=torch.uint8, device=dev)
    h = B.spconv_build_map(coords, None, L.K, L.stride, 1, mode, opt, map_ws)
    counts = B.spconv_map_counts(h)
    pairs = int(sum(counts))
    n_out = int(B.lib().spconv_map_n_out(h))
    fwd_ws = torch.empty(B.spconv_forward_workspace_bytes(h, L.c_in, L.c_out, B.DTYPES[tdt], opt), dtype=torch.uint8,
                         device=dev)
    plan = B.spconv_forward_plan(h, L.c_in, L.c_out, B.DTYPES[tdt], opt)
    B.spconv_free_map(h)
    y = torch.empty((n_out, L.c_out), dtype=tdt, device=dev)

    def step():
        hm = B.spconv_build_map(coords, None, L.K, L.stride, 1, mode, opt, map_ws)
        B.spconv_forward(hm, x, w, y, L.c_in, L.c_out, B.DTYPES[tdt], opt, fwd_ws)
        B.spconv_free_map(hm)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    B.spconv_profile_read(reset=True)
    B.spconv_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    B.spconv_profile_enable(False)
    phases = B.spconv_profile_read(reset=True)
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    ph_ms = {k: v[0] / args.steps for k, v in phases.items()}
    map_phases = ("bounds", "sort", "outcoords", "backward", "balance", "forward", "readback")
    gmas_phases = ("metadata", "gather", "gemm", "scatter")
    map_ms = sum(ph_ms[p] for p in map_phases)
    gmas_ms = sum(ph_ms[p] for p in gmas_phases)

    e = 4 if L.dtype == "f32" else 2
    ep = 4  # float32 partial buffer
    k3 = L.K ** 3
    k3p = (k3 + 3) // 4 * 4
    # compulsory bytes (sort 28 B/voxel, search 8|Q| + 12|P| + 8M + counts)
    map_bytes = 28 * n + 8 * n_out + 12 * n + 8 * pairs + 4 * (k3 + 1)
    gather_bytes = (n + pairs) * L.c_in * e + 4 * n * k3p
    scatter_bytes = (pairs * ep + n_out * e) * L.c_out + 4 * n_out * k3p
    gemm_flops = 2.0 * pairs * L.c_in * L.c_out
    gemm_bytes = pairs * (L.c_in * e + L.c_out * ep) + k3 * L.c_in * L.c_out * e
    cand = {
        "gather": ("hbm", gather_bytes, ph_ms["gather"]),
        "scatter": ("hbm", scatter_bytes, ph_ms["scatter"]),
        "forward_search": ("hbm", 8 * n_out + 12 * n + 8 * pairs, ph_ms["forward"]),
        "gemm": ("mfma", gemm_flops, ph_ms["gemm"]),
    }
    dom = max(cand, key=lambda k: cand[k][2])
    bound, work, t_ms = cand[dom]
    if bound == "hbm":
        achieved = work / (t_ms * 1e-3) / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes": work,
                "mean_launch_ms": t_ms}
    else:
        achieved = work / (t_ms * 1e-3) / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": achieved, "peak": MFMA_F16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / MFMA_F16_PEAK_TFLOPS, "traffic": None,
                "algorithmic_flops": work, "mean_launch_ms": t_ms}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(coords_np, x_np, w_np, L)

    out = {
        "metric": METRIC,
        "value": round(ms_per_step, 5),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": L.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "voxels": n, "out_voxels": n_out, "pairs": pairs, "K": L.K,
                   "c_in": L.c_in, "c_out": L.c_out, "mode": L.mode},
        "map_ms": round(map_ms, 5),
        "gmas_ms": round(gmas_ms, 5),
        "phases_ms": {k: round(v, 5) for k, v in ph_ms.items()},
        "map_gbps_compulsory": round(map_bytes / (map_ms * 1e-3) / 1e9, 2),
        "gemm_tflops": round(gemm_flops / (ph_ms["gemm"] * 1e-3) / 1e12, 3),
        "gemm_frac_mfma_f16": round(gemm_flops / (ph_ms["gemm"] * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 5),
        "gemm_operand_bytes": gemm_bytes,
        "padding_overhead": (plan.rows_padded - plan.rows_real) / max(plan.rows_real, 1),
        "gemm_launches": plan.n_gemm_launches,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))
    _ = np


def cpu_baseline(coords, x, w, L):
    """The oracle (hash-map kernel map + float64 Eq. 2), as it stands, on the host cores."""
    import oracle
    from paper_2401_06145_amd import scenes

    threads = oracle.max_threads()
    xf, wf = scenes.to_f64(x, L.dtype), scenes.to_f64(w, L.dtype)
    reps = 0
    t_total = 0.0
    while reps < 1 or (t_total < 10.0 and reps < 20):
        t0 = time.perf_counter()
        km = oracle.kernel_map(coords, None, L.K, 1, L.mode)
        oracle.features(xf, wf, km, nthreads=threads)
        t_total += time.perf_counter() - t0
        reps += 1
    return {"value": round(t_total * 1e3 / reps, 3), "unit": "ms", "cores": threads, "kind": "oracle",
            "sample": f"the full layer (kernel map + all output rows), {reps} repetition(s), mean"}


if __name__ == "__main__":
    main()
