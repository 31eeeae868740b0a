"""Benchmark: one sparse-conv layer (Map + GMaS) per step on one MI355X.

Default workload (the largest single-GPU layer of the benchmark set): the seeded
indoor-like room scene, 300,231 voxels, submanifold K = 3, C_in = C_out = 256,
float16.  A step runs the whole hot path on it: coordinate bounds, key packing and
radix sort, the double-traversed binary search with pair compaction and the
metadata tables (Map, Section 5.1), then the grouped MFMA GEMMs with the gather
fused into their operand loads, and the scatter (GMaS, Section 5.2).  Inputs are
resident in HBM before timing starts.  Prints one JSON line.

Measurement:
  1. an untimed pass with HIP events around every phase and kernel launch gives
     the per-phase split (Map ms, GMaS ms) and picks the dominant kernel (most
     GPU time per step);
  2. the timed steps record HIP events only around that kernel's launches (in one of
     every five steps, so that the event records do not load every step), on the
     stream it runs on; its algorithmic work per launch over the mean launch
     duration gives the roofline figure.  The GEMMs are priced on MFMA with real-pair
     flops, 2 |M| C_in C_out (padding never credited); the HBM bytes the GEMM's
     dataflow needs and the counter-measured traffic are reported beside them.
  3. the oracle (kernel map in full, Eq. 2 on a seeded sample of output rows, scaled to
     all rows) on the host cores, with all threads and with one.

Extra keys: the same layer with float32 GEMM partials, the other gather form, the
LiDAR-like 120k layer (C = 64) and one UNet-style network forward, plus the MFMA
utilisation and L2 hit ratios from the committed counter profiles.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
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
MAP_KERNELS = ("k_minmax", "k_radix_hist", "k_radix_scatter", "k_radix_local", "k_backward", "k_forward_count",
               "k_scan", "k_forward_write", "k_pack", "k_down_keys", "k_unique", "k_fill")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", type=int, default=3,
                   help="scene recipe (1 = LiDAR 120k, 3 = indoor 300k, 4 = UNet-style network on two LiDAR scenes)")
    p.add_argument("--channels", type=int, default=None, help="channel width for recipe 3 (default 256)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="time the headline layer only (for counter and trace runs)")
    p.add_argument("--grouping", type=int, default=None)
    p.add_argument("--gather", choices=("fused", "buffer"), default="fused",
                   help="GEMM operand rows: loaded directly by the GEMM (fused, the library default) or "
                        "gathered into a buffer first (Algorithm 1)")
    p.add_argument("--partials", choices=("layer", "f32"), default="layer",
                   help="GEMM partial precision: the layer dtype (default) or float32")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of this many MiB (HBM counter calibration)")
    a = p.parse_args()
    if a.workload == 3 and a.channels is None:
        a.channels = 256
    return a


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


def kernel_models(n, n_out, pairs, L, k3, passes, fused=True, pelem=None, centre=False):
    """Algorithmic (compulsory) bytes or flops per launch of each kernel.

    Returns name -> (bound, amount).  See the measurement section of the design
    notes for the derivation of each figure.
    """
    e = 4 if L.dtype == "f32" else 2
    ep = e if pelem is None else pelem  # GEMM partial element size
    # with the submanifold centre offset multiplied inside the scatter, the GEMMs skip
    # its n_out pairs
    cr = n_out if centre else 0
    pg = pairs - cr  # the GEMMs' pairs
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
        "k_gemm_bytes": ("hbm", (pg * L.c_in * e if not fused else n * L.c_in * e + 4 * pg)
                         + pg * L.c_out * ep + (k3 - (1 if centre else 0)) * L.c_in * L.c_out * e),
        "k_gemm_flops": ("mfma", 2.0 * pg * L.c_in * L.c_out),
        # scatter with the centre offset: each output's own input row, the other offsets'
        # partial rows, one table entry per (offset, output), the row map, W_c, the output
        "k_scatter_centre": ("hbm", n_out * L.c_in * e + pg * L.c_out * ep + n_out * L.c_out * e
                             + 4 * n_out * (k3 + 1) + L.c_in * L.c_out * e),
        "k_scatter_centre_flops": ("mfma", 2.0 * cr * L.c_in * L.c_out),
    }
    return m


def _profile_records(prefix: str):
    import glob

    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", prefix + "*.json"))):
        with open(path) as fh:
            yield json.load(fh)


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter record of this
    workload (profiles/hbm_traffic_*.json), or None if there is none or the
    kernel's sources changed since the counters were taken."""
    from paper_2401_06145_amd import profsum

    for rec in _profile_records("hbm_traffic_"):
        k = rec.get("kernels", {}).get(kernel)
        if rec.get("workload") != workload or not k:
            continue
        if k.get("source_sha256") != profsum.source_hash(kernel):
            return None
        return k["fetch_bytes"] + k["write_bytes"]
    return None


def measured_counters(workload: str):
    """Per-kernel MFMA utilisation and L2 hit ratio of this workload from the
    committed counter records (profiles/counters_*.json); kernels whose sources
    changed since the counters were taken are left out."""
    from paper_2401_06145_amd import profsum

    out = {}
    for rec in _profile_records("counters_"):
        if rec.get("workload") != workload:
            continue
        for kid, k in rec.get("kernels", {}).items():
            if k.get("source_sha256") != profsum.source_hash(kid):
                continue
            d = out.setdefault(kid, {})
            for key in ("mfma_util_pct", "mfma_flops_executed", "l2_hit_pct"):
                if key in k:
                    d[key] = k[key]
    return out


class LayerBench:
    """One layer of a scene recipe on the GPU: inputs resident in HBM, map and forward
    workspaces allocated once, `step()` = a cold Map build plus the forward."""

    def __init__(self, workload, channels, gather="fused", grouping=None, partials="layer"):
        import torch

        from paper_2401_06145_amd import binding as B
        from paper_2401_06145_amd import scenes

        self.B = B
        dev = torch.device("cuda:0")
        self.wl = scenes.workload(workload, channels)
        L = self.L = self.wl.layers[0]
        self.coords_np = self.wl.coords
        n = self.n = len(self.coords_np)
        self.x_np = scenes.features(n, L.c_in, L.dtype, 2000 + workload)
        self.w_np = scenes.weights(L.K, L.c_in, L.c_out, L.dtype, 3000 + workload)
        self.tdt = B.TORCH_DTYPES[L.dtype]
        self.dt = B.DTYPES[self.tdt]
        self.coords = torch.from_numpy(self.coords_np).to(dev)
        self.x = torch.from_numpy(self.x_np).to(dev)
        self.w = torch.from_numpy(self.w_np).to(dev)
        self.mode = B.MODES[L.mode]
        self.fused = gather == "fused"
        g = B.GATHER_FUSED if self.fused else B.GATHER_BUFFER
        self.partial_dtype = 1 if partials == "f32" else 2
        self.grouping = grouping
        self.opt = B.Options.make(grouping=grouping, gather=g, partial_dtype=self.partial_dtype)
        self.map_ws = torch.empty(B.spconv_map_workspace_bytes(n, 0, L.K, self.mode, self.opt), dtype=torch.uint8,
                                  device=dev)
        h = B.spconv_build_map(self.coords, None, L.K, L.stride, 1, self.mode, self.opt, self.map_ws)
        self.counts = B.spconv_map_counts(h)
        self.pairs = int(sum(self.counts))
        self.n_out = int(B.lib().spconv_map_n_out(h))
        self.plan = B.spconv_forward_plan(h, L.c_in, L.c_out, self.dt, self.opt)
        self._h = h
        self._ws = {}
        self.y = torch.empty((self.n_out, L.c_out), dtype=self.tdt, device=dev)
        self.pelem = 4 if (self.partial_dtype == 1 or L.dtype == "f32") else 2

    def variant(self, **kw):
        """Options for a variant of the forward (same map), with its workspace."""
        import torch

        B = self.B
        base = {"gather": B.GATHER_FUSED if self.fused else B.GATHER_BUFFER, "partial_dtype": self.partial_dtype,
                "grouping": self.grouping}
        base.update(kw)
        opt = B.Options.make(**base)
        key = tuple(sorted(base.items()))
        if key not in self._ws:
            nb = B.spconv_forward_workspace_bytes(self._h, self.L.c_in, self.L.c_out, self.dt, opt)
            self._ws[key] = torch.empty(nb, dtype=torch.uint8, device=self.coords.device)
        return opt, self._ws[key]

    def step(self, fopt=None, ws=None):
        B, L = self.B, self.L
        if fopt is None:
            fopt, ws = self.variant()
        hm = B.spconv_build_map(self.coords, None, L.K, L.stride, 1, self.mode, self.opt, self.map_ws)
        B.spconv_forward(hm, self.x, self.w, self.y, L.c_in, L.c_out, self.dt, fopt, ws)
        B.spconv_free_map(hm)

    def close(self):
        if self._h is not None:
            self.B.spconv_free_map(self._h)
            self._h = None

    def timed_pass(self, mask, R=10, **variant):
        """R steps with HIP events around the phases / kernels in `mask`; returns the
        library's per-id record (summed ms, intervals)."""
        import torch

        B = self.B
        fopt, ws = self.variant(**variant)
        B.spconv_profile_read(reset=True)
        B.spconv_profile_enable(mask)
        for _ in range(R):
            self.step(fopt, ws)
        torch.cuda.synchronize()
        B.spconv_profile_enable(False)
        return B.spconv_profile_read(reset=True)

    def layer_ms(self, R=20, **variant):
        """Whole steps (Map build + forward) of a variant, no events: ms per step."""
        import torch

        fopt, ws = self.variant(**variant)
        for _ in range(3):
            self.step(fopt, ws)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(R):
            self.step(fopt, ws)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / R

    def phases(self, R=10, **variant):
        prof = self.timed_pass(self.B.PHASES_ALL, R, **variant)
        return {k: v[0] / R for k, v in prof.items() if not k.startswith("k_") and v[1] > 0}

    def kernels(self, R=10):
        """kernel id -> (ms per step, launches per step), one pass per kernel with
        events around that kernel's launches only."""
        out = {}
        for name, kid in self.B.profile_ids().items():
            if name.startswith("k_"):
                ms, cnt = self.timed_pass(1 << kid, R)[name]
                if cnt > 0:
                    out[name] = (ms / R, cnt / R)
        return out

    def timed(self, steps, kernel):
        """`steps` timed steps with events around `kernel`'s launches in one of every
        EVENT_EVERY steps.  Returns (ms per step, mean launch ms, launches per step,
        timed launches)."""
        import torch

        B = self.B
        fopt, ws = self.variant()
        mask = 1 << B.profile_ids()[kernel]
        sampled = 0
        B.spconv_profile_read(reset=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            on = i % EVENT_EVERY == 0
            if on:
                B.spconv_profile_enable(mask)
                sampled += 1
            self.step(fopt, ws)
            if on:
                B.spconv_profile_enable(False)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        live = B.spconv_profile_read(reset=True)[kernel]
        return (t1 - t0) * 1e3 / steps, live[0] / live[1], live[1] / sampled, int(live[1])


def roofline_for(kernel, models, mean_launch_ms, L, workload):
    """The dominant kernel's roofline: the GEMM on MFMA (real-pair flops), every other
    kernel on HBM (algorithmic bytes)."""
    if kernel == "k_gemm":
        flops = models["k_gemm_flops"][1]
        byts = models["k_gemm_bytes"][1]
        peak = MFMA_PEAK_TFLOPS[L.dtype]
        achieved = flops / (mean_launch_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 5), "traffic": None, "kernel": kernel,
                "algorithmic_flops_per_launch": flops,
                # the HBM side of the same launch: bytes the fused-gather dataflow must move
                # (input rows once, pair rows of partials, weights) and their rate
                "hbm_algorithmic_bytes_per_launch": int(byts),
                "hbm_gbs": round(byts / (mean_launch_ms * 1e-3) / 1e9, 2),
                "hbm_frac": round(byts / (mean_launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 5)}
    else:
        bound, work = models[kernel]
        achieved = work / (mean_launch_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None, "kernel": kernel,
                "algorithmic_bytes_per_launch": int(work)}
        if kernel + "_flops" in models:
            # the centre offset's MFMA work inside the same launch, against the MFMA peak
            fl = models[kernel + "_flops"][1]
            roof["mfma_flops_per_launch"] = fl
            roof["mfma_frac"] = round(fl / (mean_launch_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS[L.dtype], 5)
    tb = measured_traffic(kernel, workload)
    roof["traffic"] = round(tb) if tb is not None else None
    return roof


def main():
    args = parse()
    if args.calibrate_copy:
        copy_calibration(args.calibrate_copy)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): libspconv has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    if args.workload == 4:
        print(json.dumps(bench_network(args.steps, args.warmup)))
        return
    import torch

    lb = LayerBench(args.workload, args.channels, args.gather, args.grouping, args.partials)
    L = lb.L
    for _ in range(args.warmup):
        lb.step()
    torch.cuda.synchronize()

    # 1. breakdown (untimed)
    ph_ms = lb.phases()
    kern = lb.kernels()
    dominant = max(kern, key=lambda k: kern[k][0])

    # 2. timed steps
    ms_per_step, mean_launch_ms, launches_per_step, timed_launches = lb.timed(args.steps, dominant)

    k3 = L.K ** 3
    passes = int(round(kern.get("k_radix_scatter", (0, 0))[1]))
    models = kernel_models(lb.n, lb.n_out, lb.pairs, L, k3, passes, fused=lb.fused, pelem=lb.pelem,
                           centre=bool(lb.plan.centre))
    roof = roofline_for(dominant, models, mean_launch_ms, L, lb.wl.name)
    roof.update({"mean_launch_ms": round(mean_launch_ms, 6), "launches_per_step": launches_per_step,
                 "timed_launches": timed_launches, "event_steps": f"1 in {EVENT_EVERY} timed steps"})
    # the kernel with the next most time per step (at C = 256 the GEMM and the centre
    # scatter take about the same), priced the same way from the breakdown pass
    ranked = sorted((k for k in kern if k in models or k == "k_gemm"), key=lambda k: -kern[k][0])
    roof_next = None
    if len(ranked) > 1:
        second = ranked[1] if ranked[0] == dominant else ranked[0]
        ms2, cnt2 = kern[second]
        roof_next = roofline_for(second, models, ms2 / cnt2, L, lb.wl.name)
        roof_next.update({"mean_launch_ms": round(ms2 / cnt2, 6), "launches_per_step": cnt2,
                          "event_steps": "breakdown pass, events around this kernel only"})

    map_ms = sum(ph_ms.get(p, 0.0) for p in MAP_PHASES)
    gmas_ms = sum(ph_ms.get(p, 0.0) for p in GMAS_PHASES)
    n, n_out, pairs = lb.n, lb.n_out, lb.pairs
    map_bytes = 28 * n + 8 * n_out + 12 * n + 8 * pairs + 4 * (k3 + 1)
    gemm_ms = kern.get("k_gemm", (float("nan"), 1))[0]
    gemm_tflops = models["k_gemm_flops"][1] / (gemm_ms * 1e-3) / 1e12
    pname = "f32" if lb.pelem == 4 else L.dtype

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
        "config": {"workload": lb.wl.name, "voxels": n, "out_voxels": n_out, "pairs": pairs, "K": L.K,
                   "c_in": L.c_in, "c_out": L.c_out, "mode": L.mode, "gemm_partials": pname,
                   "centre_in_scatter": bool(lb.plan.centre)},
        "map_ms": round(map_ms, 5),
        "gmas_ms": round(gmas_ms, 5),
        "phases_ms": {k: round(v, 5) for k, v in ph_ms.items()},
        "kernels_ms_per_step": {k: round(v[0], 5) for k, v in sorted(kern.items(), key=lambda t: -t[1][0])},
        "map_gbps_compulsory": round(map_bytes / (map_ms * 1e-3) / 1e9, 2),
        "gemm_tflops": round(gemm_tflops, 3),
        "gemm_frac_mfma": round(gemm_tflops / MFMA_PEAK_TFLOPS[L.dtype], 5),
        "padding_overhead": (lb.plan.rows_padded - lb.plan.rows_real) / max(lb.plan.rows_real, 1),
        "gemm_launches": lb.plan.n_gemm_launches,
        "gather": args.gather,
        "roofline": roof,
        "roofline_next": roof_next,
    }
    counters = measured_counters(lb.wl.name)
    if counters:
        out["counters"] = counters

    if not args.no_extras:
        # the same layer with the other GMaS variants: phase events (a breakdown pass), and
        # whole steps without events beside the default's, timed back to back (phase sums
        # of two variants can rank them differently from their whole steps)
        def gmas_of(ph, **variant):
            return {**{p: round(ph.get(p, 0.0), 5) for p in GMAS_PHASES},
                    "total": round(sum(ph.get(p, 0.0) for p in GMAS_PHASES), 5),
                    "layer_ms": round(lb.layer_ms(**variant), 5), "default_layer_ms": round(lb.layer_ms(), 5)}

        B = lb.B
        other_p = 1 if lb.partial_dtype == 2 else 2
        out["gmas_ms_other_partials"] = {"gemm_partials": "f32" if other_p == 1 else L.dtype,
                                         **gmas_of(lb.phases(partial_dtype=other_p), partial_dtype=other_p)}
        other_g = B.GATHER_BUFFER if lb.fused else B.GATHER_FUSED
        out["gmas_ms_other_gather"] = {"gather": "buffer" if lb.fused else "fused",
                                       **gmas_of(lb.phases(gather=other_g), gather=other_g)}
        if lb.plan.centre:
            # the centre offset through the GEMM and its partial buffer, like the other offsets
            out["gmas_ms_centre_through_gemm"] = gmas_of(lb.phases(centre=1), centre=1)
    lb_cpu = (lb.coords_np, lb.x_np, lb.w_np, L)
    lb.close()
    del lb
    torch.cuda.empty_cache()
    if not args.no_extras:
        others = {}
        if args.workload != 1:
            others["lidar-120k-subm-k3-c64-f16"] = quick_layer(1, None)
        others["unet-2x-lidar-240k-f16"] = {k: v for k, v in bench_network(5, 2).items()
                                           if k in ("value", "unit", "map_ms", "gmas_ms")}
        out["other_workloads"] = others

    out["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(*lb_cpu)
    print(json.dumps(out))


def quick_layer(workload, channels, steps=20):
    """ms per layer (cold Map + forward) and the phase split of another layer recipe."""
    import torch

    lb = LayerBench(workload, channels)
    for _ in range(3):
        lb.step()
    ph = lb.phases()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        lb.step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    flops = 2.0 * lb.plan.rows_real * lb.L.c_in * lb.L.c_out  # the GEMMs' real pairs
    res = {"ms_per_layer": round(ms, 5), "map_ms": round(sum(ph.get(p, 0.0) for p in MAP_PHASES), 5),
           "gmas_ms": round(sum(ph.get(p, 0.0) for p in GMAS_PHASES), 5),
           "gemm_ms": round(ph.get("gemm", 0.0), 5),
           "gemm_frac_mfma": round(flops / (ph.get("gemm", float("nan")) * 1e-3) / 1e12
                                   / MFMA_PEAK_TFLOPS[lb.L.dtype], 5),
           "voxels": lb.n, "pairs": lb.pairs}
    lb.close()
    return res


def bench_network(steps, warmup):
    """One step = one forward of the UNet-style network on the two-scene batch (241,686
    voxels at level 0, float16, 46 convolutions): every kernel map is built inside the
    step (cached per coordinate set within the step, as the network reuses them), then
    every layer runs.  Returns ms per forward and the time split by phase."""
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

    for _ in range(warmup):
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
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    n_conv = sum(1 for o in ops if o.kind == "conv")
    return {
        "metric": "UNet-style network forward ms (maps built inside the step)", "value": round(ms, 4), "unit": "ms",
        "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": wl.name, "voxels": len(wl.coords), "convolutions": n_conv},
        "map_ms": round(sum(ph_ms.get(p, 0.0) for p in MAP_PHASES), 4),
        "gmas_ms": round(sum(ph_ms.get(p, 0.0) for p in GMAS_PHASES), 4),
        "phases_ms": {k: round(v, 4) for k, v in ph_ms.items()},
        "roofline": None, "cpu_baseline": None}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(coords, x, w, L, rows_all=96000, rows_one=24000):
    """The oracle (hash-map kernel map + float64 Eq. 2), as it stands, on the host cores.

    The kernel map is built in full (the oracle builds it on one thread); Eq. 2 runs on
    a seeded sample of output rows, once on every OpenMP thread and once on one thread,
    and its time is scaled to all rows (each output row costs the same work in
    expectation: the sample is uniform over rows)."""
    import numpy as np

    import oracle
    from paper_2401_06145_amd import scenes

    threads = oracle.max_threads()
    xf, wf = scenes.to_f64(x, L.dtype), scenes.to_f64(w, L.dtype)
    t0 = time.perf_counter()
    km = oracle.kernel_map(coords, None, L.K, 1, L.mode)
    map_ms = (time.perf_counter() - t0) * 1e3
    n_out = km.n_out
    rng = np.random.default_rng(4242)

    def feat_ms(nrows, nthreads):
        nrows = min(nrows, n_out)
        rows = np.sort(rng.choice(n_out, nrows, replace=False))
        t = time.perf_counter()
        oracle.features(xf, wf, km, rows=rows, nthreads=nthreads)
        return (time.perf_counter() - t) * 1e3 * n_out / nrows

    f_all = feat_ms(rows_all, threads)
    f_one = feat_ms(rows_one, 1)
    return {"value": round(map_ms + f_all, 3), "unit": "ms", "cores": threads, "kind": "oracle",
            "sample": (f"kernel map of all {len(coords)} voxels (one thread, as the oracle builds it); "
                       f"Eq. 2 on {min(rows_all, n_out)} seeded output rows on {threads} threads and on "
                       f"{min(rows_one, n_out)} rows on 1 thread, scaled to all {n_out} rows"),
            "cpu_model": cpu_model(), "map_ms": round(map_ms, 3), "features_ms": round(f_all, 3),
            "single_thread": {"value": round(map_ms + f_one, 3), "map_ms": round(map_ms, 3),
                              "features_ms": round(f_one, 3)}}


if __name__ == "__main__":
    main()
