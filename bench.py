"""Benchmark: one sparse-conv layer (Map + GMaS) per step on one MI355X.

A step runs the whole hot path on one seeded LiDAR-like scene (about 120k voxels,
submanifold K = 3, C_in = C_out = 64, float16): coordinate bounds, key packing and
radix sort, the double-traversed binary search with pair compaction and the
metadata tables (Map), then gather, grouped MFMA GEMMs and scatter (GMaS).  By default
the gather is fused into the GEMMs' operand loads (each GEMM reads its pairs' input rows
directly); the breakdown also times the layer with Algorithm 1's separate gather kernel
and buffer.  Inputs are resident in HBM before timing starts.  Prints one JSON line.

Measurement:
  1. an untimed pass with HIP events around every phase and kernel launch gives
     the per-phase split (Map ms, GMaS ms) and picks the dominant kernel (most
     GPU time per step);
  2. the timed steps record HIP events only around that kernel's launches (in one of
     every five steps, so that the event records do not load every step), on the
     stream it runs on; its algorithmic bytes (or flops) per launch over the mean
     launch duration give the roofline figure.
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
MFMA_PEAK_TFLOPS = {"f16": 2500.0, "bf16": 2500.0, "f32": 157.3}
MAP_PHASES = ("bounds", "sort", "hash", "outcoords", "backward", "balance", "metadata", "forward", "readback")
GMAS_PHASES = ("gather", "gemm", "scatter")
EVENT_EVERY = 5  # timed steps per step with events around the dominant kernel


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", type=int, default=1,
                   help="scene recipe (1 = LiDAR 120k, 3 = indoor 300k, 4 = UNet-style network on two LiDAR scenes)")
    p.add_argument("--channels", type=int, default=None, help="channel width for recipe 3")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--grouping", type=int, default=None)
    p.add_argument("--gather", choices=("fused", "buffer"), default="fused",
                   help="GEMM operand rows: loaded directly by the GEMM (fused, the library default) or "
                        "gathered into a buffer first (Algorithm 1)")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of this many MiB (HBM counter calibration)")
    return p.parse_args()


def copy_calibration(mib: int) -> None:
    """A plain device-to-device copy of known size: reads and writes `mib` MiB once."""
    import torch

    n = mib * 1024 * 1024 // 4
    src = torch.arange(n, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_mib": mib, "bytes_read": n * 4, "bytes_written": n * 4,
                      "dispatches": 3}))


def kernel_models(n, n_out, pairs, L, k3, passes, fused=True):
    """Algorithmic (compulsory) bytes or flops per launch of each kernel.

    Returns name -> (bound, amount).  See the measurement section of the design
    notes for the derivation of each figure.
    """
    e = 4 if L.dtype == "f32" else 2
    ep = e  # GEMM partials are stored in the layer dtype
    P = max(passes, 1)
    # scans per step: the match-count scan (one entry per work item, K^3 x source blocks
    # of 1024), plus one digit-offset scan per radix pass when the sort has between 257
    # and 1023 tiles of 2048 keys
    nb = -(-n // 1024)
    ntiles = -(-n // 2048)
    scan_lens = ([256 * ntiles] * P if 256 < ntiles < 1024 else []) + [k3 * nb]
    m = {
        "k_scan": ("hbm", 8.0 * sum(scan_lens) / len(scan_lens)),
        # radix passes: the first reads int32 coordinates (16 B/row), later ones key + row (12 B)
        "k_radix_scatter": ("hbm", (16 * n + 12 * n + (P - 1) * 24 * n) / P),
        "k_radix_hist": ("hbm", (16 * n + (P - 1) * 8 * n) / P),
        # by-bucket small sorts: each bucket's keys and rows read and written once
        "k_radix_local": ("hbm", 24 * n),
        "k_minmax": ("hbm", 16 * n),
        # forward search, count pass: query keys and source keys once, one result word per
        # (offset, query)
        "k_forward_count": ("hbm", 8 * n_out + 8 * n + 4 * k3 * n_out),
        # write pass: reads the results and the rows of the matches; writes the pair lists,
        # the query-side table's matches (in place) and the whole source-side table
        # (odd-K submanifold maps leave the source-side table to the first table-driven gather)
        "k_forward_write": ("hbm", 4 * k3 * n_out + 4 * n_out + 4 * n + 12 * pairs
                            + (0 if (L.mode == "subm" and L.K % 2 == 1) else 4 * k3 * n)),
        "k_backward": ("hbm", 8 * n_out),
        # source-side table fill (maps other than odd-K submanifold ones)
        "k_fill": ("hbm", 4 * k3 * n),
        # gather / scatter: feature rows, partial rows, one table entry per (offset, point), row map
        "k_gather": ("hbm", (n + pairs) * L.c_in * e + 4 * n * (k3 + 1)),
        "k_scatter": ("hbm", pairs * L.c_out * ep + n_out * L.c_out * e + 4 * n_out * (k3 + 1)),
        # GEMM: A rows (the gathered buffer, or with the fused gather each input row once
        # plus one row index per pair), partial rows, weights
        "k_gemm_bytes": ("hbm", (pairs * L.c_in * e if not fused else n * L.c_in * e + 4 * pairs)
                         + pairs * L.c_out * ep + k3 * L.c_in * L.c_out * e),
        "k_gemm_flops": ("mfma", 2.0 * pairs * L.c_in * L.c_out),
    }
    return m


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter record of this
    workload (profiles/hbm_traffic_*.json), or None if there is none or the
    kernel's sources changed since the counters were taken."""
    import glob

    from paper_2401_06145_amd import profsum

    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.json"))):
        with open(path) as fh:
            rec = json.load(fh)
        k = rec.get("kernels", {}).get(kernel)
        if rec.get("workload") != workload or not k:
            continue
        if k.get("source_sha256") != profsum.source_hash(kernel):
            return None
        return k["fetch_bytes"] + k["write_bytes"]
    return None


def main():
    args = parse()
    if args.calibrate_copy:
        copy_calibration(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    if args.workload == 4:
        bench_network(args)
        return
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
    gather = B.GATHER_FUSED if args.gather == "fused" else B.GATHER_BUFFER
    opt = B.Options.make(grouping=args.grouping, gather=gather)
    # the other gather form, timed in the breakdown pass for comparison
    alt_gather = B.GATHER_BUFFER if gather == B.GATHER_FUSED else B.GATHER_FUSED
    alt_opt = B.Options.make(grouping=args.grouping, gather=alt_gather)
    map_ws = torch.empty(B.spconv_map_workspace_bytes(n, 0, L.K, mode, opt), dtype=torch.uint8, device=dev)
    h = B.spconv_build_map(coords, None, L.K, L.stride, 1, mode, opt, map_ws)
    counts = B.spconv_map_counts(h)
    pairs = int(sum(counts))
    n_out = int(B.lib().spconv_map_n_out(h))
    fwd_ws = torch.empty(B.spconv_forward_workspace_bytes(h, L.c_in, L.c_out, B.DTYPES[tdt], opt),
                         dtype=torch.uint8, device=dev)
    alt_ws = torch.empty(B.spconv_forward_workspace_bytes(h, L.c_in, L.c_out, B.DTYPES[tdt], alt_opt),
                         dtype=torch.uint8, device=dev)
    plan = B.spconv_forward_plan(h, L.c_in, L.c_out, B.DTYPES[tdt], opt)
    B.spconv_free_map(h)
    y = torch.empty((n_out, L.c_out), dtype=tdt, device=dev)

    def step(fopt=opt, ws=fwd_ws):
        hm = B.spconv_build_map(coords, None, L.K, L.stride, 1, mode, opt, map_ws)
        B.spconv_forward(hm, x, w, y, L.c_in, L.c_out, B.DTYPES[tdt], fopt, ws)
        B.spconv_free_map(hm)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # 1. breakdown (untimed): one pass with events around the phases, then one pass
    #    per kernel with events around that kernel's launches only
    R = 10
    ids = B.profile_ids()

    def timed_pass(mask, alt=False):
        B.spconv_profile_read(reset=True)
        B.spconv_profile_enable(mask)
        for _ in range(R):
            if alt:
                step(alt_opt, alt_ws)
            else:
                step()
        torch.cuda.synchronize()
        B.spconv_profile_enable(False)
        return B.spconv_profile_read(reset=True)

    prof = timed_pass(B.PHASES_ALL)
    ph_ms = {k: v[0] / R for k, v in prof.items() if not k.startswith("k_")}
    alt_prof = timed_pass(B.PHASES_ALL, alt=True)
    alt_gmas = {p: alt_prof[p][0] / R for p in GMAS_PHASES}
    kern = {}
    for name, kid in ids.items():
        if name.startswith("k_"):
            ms, cnt = timed_pass(1 << kid)[name]
            if cnt > 0:
                kern[name] = (ms / R, cnt / R)
    dominant = max(kern, key=lambda k: kern[k][0])

    # 2. timed steps; events only around the dominant kernel's launches, in every
    #    EVENT_EVERY-th step (each event record costs the host a few microseconds,
    #    which would otherwise be charged to every step)
    mask = 1 << ids[dominant]
    sampled = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        on = i % EVENT_EVERY == 0
        if on:
            B.spconv_profile_enable(mask)
            sampled += 1
        step()
        if on:
            B.spconv_profile_enable(False)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    live = B.spconv_profile_read(reset=True)[dominant]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    mean_launch_ms = live[0] / live[1]
    launches_per_step = live[1] / sampled

    k3 = L.K ** 3
    passes = int(round(kern.get("k_radix_scatter", (0, 0))[1]))
    models = kernel_models(n, n_out, pairs, L, k3, passes, fused=gather == B.GATHER_FUSED)
    if dominant == "k_gemm":
        # with materialised buffers the GEMM's intensity is below the MFMA ridge: price it on HBM
        flops = models["k_gemm_flops"][1]
        byts = models["k_gemm_bytes"][1]
        ridge = MFMA_PEAK_TFLOPS[L.dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
        bound, work = ("hbm", byts) if flops / byts < ridge else ("mfma", flops)
    else:
        bound, work = models[dominant]
    if bound == "hbm":
        achieved = work / (mean_launch_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None, "kernel": dominant,
                "algorithmic_bytes_per_launch": int(work)}
    else:
        peak = MFMA_PEAK_TFLOPS[L.dtype]
        achieved = work / (mean_launch_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 5), "traffic": None, "kernel": dominant,
                "algorithmic_flops_per_launch": work}
    roof.update({"mean_launch_ms": round(mean_launch_ms, 6), "launches_per_step": launches_per_step,
                 "timed_launches": int(live[1]), "event_steps": f"1 in {EVENT_EVERY} timed steps"})
    tb = measured_traffic(dominant, wl.name)
    roof["traffic"] = round(tb) if tb is not None else None

    map_ms = sum(ph_ms.get(p, 0.0) for p in MAP_PHASES)
    gmas_ms = sum(ph_ms.get(p, 0.0) for p in GMAS_PHASES)
    map_bytes = 28 * n + 8 * n_out + 12 * n + 8 * pairs + 4 * (k3 + 1)
    gemm_ms = kern.get("k_gemm", (float("nan"), 1))[0]
    gemm_tflops = models["k_gemm_flops"][1] / (gemm_ms * 1e-3) / 1e12

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
        "kernels_ms_per_step": {k: round(v[0], 5) for k, v in sorted(kern.items(), key=lambda t: -t[1][0])},
        "map_gbps_compulsory": round(map_bytes / (map_ms * 1e-3) / 1e9, 2),
        "gemm_tflops": round(gemm_tflops, 3),
        "gemm_frac_mfma": round(gemm_tflops / MFMA_PEAK_TFLOPS[L.dtype], 5),
        "padding_overhead": (plan.rows_padded - plan.rows_real) / max(plan.rows_real, 1),
        "gemm_launches": plan.n_gemm_launches,
        "gather": args.gather,
        # the same layer with the other gather form (breakdown pass, phase events)
        "gmas_ms_other_gather": {"gather": "buffer" if args.gather == "fused" else "fused",
                                 **{p: round(v, 5) for p, v in alt_gmas.items()},
                                 "total": round(sum(alt_gmas.values()), 5)},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def bench_network(args):
    """One step = one forward of the UNet-style network on the two-scene batch (241,686
    voxels at level 0, float16, 46 convolutions): every kernel map is built inside the
    step (cached per coordinate set within the step, as the network reuses them), then
    every layer runs.  Reports ms per forward and the time split by phase and kernel."""
    import torch

    from paper_2401_06145_amd import binding as B
    from paper_2401_06145_amd import net, scenes

    dev = torch.device("cuda:0")
    wl = scenes.workload(4)
    coords = torch.from_numpy(wl.coords).to(dev)
    x0 = torch.from_numpy(scenes.features(len(wl.coords), net.STEM_C, "f16", 2004)).to(dev)
    ops = net.unet_ops()
    weights = net.UNet(coords).w  # device weights, built once (model parameters)

    def step():
        model = net.UNet(coords, ops=ops, weights=weights)
        return model.forward(x0)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    B.spconv_profile_read(reset=True)
    B.spconv_profile_enable(B.PHASES_ALL)
    R = 3
    for _ in range(R):
        step()
    torch.cuda.synchronize()
    B.spconv_profile_enable(False)
    prof = B.spconv_profile_read(reset=True)
    ph_ms = {k: v[0] / R for k, v in prof.items() if not k.startswith("k_") and v[1] > 0}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    n_conv = sum(1 for o in ops if o.kind == "conv")
    print(json.dumps({
        "metric": "UNet-style network forward ms (maps built inside the step)", "value": round(ms, 4), "unit": "ms",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": wl.name, "voxels": len(wl.coords), "convolutions": n_conv},
        "map_ms": round(sum(ph_ms.get(p, 0.0) for p in MAP_PHASES), 4),
        "gmas_ms": round(sum(ph_ms.get(p, 0.0) for p in GMAS_PHASES), 4),
        "phases_ms": {k: round(v, 4) for k, v in ph_ms.items()},
        "roofline": None, "cpu_baseline": None}))


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
