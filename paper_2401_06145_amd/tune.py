"""Offline tuning of the layer's parameters on MI355X.

* ``tiles``: Algorithm 2 of the paper (Section 5.2.1), autotuning the Gather and
  Scatter tile size.  For each layer it builds the metadata of a few sampled
  point clouds, profiles Gather (and Scatter) for R rounds with every admissible
  tile T (a divisor of the channel count that covers whole 16-byte vectors), and
  keeps the fastest.  The sampled clouds are seeded synthetic scenes of the same
  recipe (the paper samples its dataset).  Gather tiles are timed on Algorithm 1's
  gather kernel (the buffer form).  For Scatter, the tile of one 16-byte partial
  vector per thread is the row-group kernel (a lane group per output row); the
  wider tiles are the one-thread-per-output-tile kernel.
* ``map``: the source-block size B, query-block limit C and thread-block size of the
  double-traversed binary search (Section 5.1.4), swept over powers of two.
* ``unet``: Algorithm 2 per layer over the UNet-style network's convolutions (the
  two-scene batch): the Scatter tile, the GEMM's rows per workgroup tile and, for
  Algorithm 1's gather kernel (the buffer form), the Gather tile; then the whole
  forward with the per-layer winners against the constant defaults.

Timings are HIP-event means recorded by the library on the launch stream.
Prints one JSON object per measured point and, at the end, the selection.

    python -m paper_2401_06145_amd.tune tiles --workload 1 --rounds 20
    python -m paper_2401_06145_amd.tune map --workload 1 3
    python -m paper_2401_06145_amd.tune unet --rounds 10
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import torch

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2401_06145_amd import binding as B  # noqa: E402
from paper_2401_06145_amd import scenes  # noqa: E402


def _timed(fn, kernel: str, rounds: int) -> float:
    """Mean ms of one kernel over `rounds` calls of fn (events around that kernel only)."""
    ids = B.profile_ids()
    fn()
    torch.cuda.synchronize()
    B.spconv_profile_read(reset=True)
    B.spconv_profile_enable(1 << ids[kernel])
    for _ in range(rounds):
        fn()
    torch.cuda.synchronize()
    B.spconv_profile_enable(False)
    ms, cnt = B.spconv_profile_read(reset=True)[kernel]
    return ms / max(cnt, 1)


def tile_candidates(c: int, elem: int, max_vectors: int = 16):
    """Divisors T of c with T * elem a multiple of 16 bytes and at most max_vectors vectors."""
    out = []
    for t in range(1, c + 1):
        if c % t == 0 and (t * elem) % 16 == 0 and (t * elem) // 16 <= max_vectors:
            out.append(t)
    return out


def tune_tiles(workloads, rounds: int, samples: int, channels):
    dev = torch.device("cuda:0")
    best_all = []
    for wi in workloads:
        for c in channels if wi == 3 else [None]:
            wl = scenes.workload(wi, c)
            L = wl.layers[0]
            tdt = B.TORCH_DTYPES[L.dtype]
            e = 4 if L.dtype == "f32" else 2
            # sampled clouds: the recipe's scene plus shuffled-row copies (new metadata each)
            clouds = [wl.coords]
            rng = torch.Generator().manual_seed(wi)
            for _ in range(samples - 1):
                perm = torch.randperm(len(wl.coords), generator=rng).numpy()
                clouds.append(wl.coords[perm])
            res = {"gather": {}, "scatter": {}}
            for coords_np in clouds:
                coords = torch.from_numpy(coords_np).to(dev)
                km = B.KernelMap.build(coords, L.K, L.stride, 1, L.mode)
                x = torch.from_numpy(scenes.features(len(coords_np), L.c_in, L.dtype, 7)).to(dev)
                w = torch.from_numpy(scenes.weights(L.K, L.c_in, L.c_out, L.dtype, 8)).to(dev)
                for t in tile_candidates(L.c_in, e):
                    # Algorithm 1's gather kernel (the default fuses the gather into the GEMM)
                    f = B.Forward(km, L.c_in, L.c_out, tdt, B.Options.make(t_gather=t, gather=B.GATHER_BUFFER))
                    ms = _timed(lambda: f(x, w), "k_gather", rounds)
                    res["gather"].setdefault(t, []).append(ms)
                for t in [t for t in tile_candidates(L.c_out, e) if t <= 64 and (t & (t - 1)) == 0 and t >= 4]:
                    # the scatter of every offset's partials (the default multiplies a
                    # submanifold layer's centre offset inside its own scatter kernel, which has no tile)
                    f = B.Forward(km, L.c_in, L.c_out, tdt, B.Options.make(t_scatter=t, centre=1))
                    ms = _timed(lambda: f(x, w), "k_scatter", rounds)
                    res["scatter"].setdefault(t, []).append(ms)
            sel = {}
            for op in ("gather", "scatter"):
                for t, v in sorted(res[op].items()):
                    print(json.dumps({"workload": wl.name, "op": op, "T": t, "mean_us": round(1e3 * sum(v) / len(v), 2)}),
                          flush=True)
                sel[op] = min(res[op], key=lambda t: sum(res[op][t]))
            best = {"workload": wl.name, "c_in": L.c_in, "c_out": L.c_out, "dtype": L.dtype,
                    "t_gather": sel["gather"], "t_scatter": sel["scatter"]}
            print(json.dumps({"selected": best}), flush=True)
            best_all.append(best)
    return best_all


def tune_map(workloads, rounds: int, Bs, Cqs, wgs=(256,)):
    dev = torch.device("cuda:0")
    best = []
    for wi in workloads:
        wl = scenes.workload(wi)
        L = wl.layers[0]  # (recipe 2: its downsampling layer)
        coords = torch.from_numpy(wl.coords).to(dev)
        n = len(wl.coords)
        mode = B.MODES[L.mode]
        results = {}
        for Bsz, Cq, wg in [(b_, c_, w_) for b_ in Bs for c_ in Cqs for w_ in wgs
                            if c_ % w_ == 0 and c_ // w_ in (1, 2, 4, 8)]:
            opt = B.Options.make(B=Bsz, Cq=Cq, wg=wg)
            ws = torch.empty(B.spconv_map_workspace_bytes(n, 0, L.K, mode, opt), dtype=torch.uint8, device=dev)

            def build():
                h = B.spconv_build_map(coords, None, L.K, L.stride, 1, mode, opt, ws)
                B.spconv_free_map(h)

            for _ in range(3):
                build()
            torch.cuda.synchronize()
            B.spconv_profile_read(reset=True)
            B.spconv_profile_enable(B.PHASES_ALL)
            for _ in range(rounds):
                build()
            torch.cuda.synchronize()
            B.spconv_profile_enable(False)
            ph = B.spconv_profile_read(reset=True)
            row = {k: round(ph[k][0] / rounds * 1e3, 1) for k in ("backward", "balance", "forward")}
            row["total_us"] = round(sum(row.values()), 1)
            results[(Bsz, Cq, wg)] = row["total_us"]
            print(json.dumps({"workload": wl.name, "voxels": n, "B": Bsz, "Cq": Cq, "wg": wg, **row}), flush=True)
        b = min(results, key=results.get)
        sel = {"workload": wl.name, "B": b[0], "Cq": b[1], "wg": b[2], "total_us": results[b],
               "default_us": results.get((1024, 1024, 256))}
        print(json.dumps({"selected": sel}), flush=True)
        best.append(sel)
    return best


def tune_unet(rounds: int, rows_cands=(64, 128, 256, 512, 1024, 2048, 4096), forward_steps: int = 20):
    """Algorithm 2 per layer of the UNet-style network, then the forward with the
    winners against the defaults.  Returns the per-layer table."""
    import time

    from paper_2401_06145_amd import net

    dev = torch.device("cuda:0")
    wl = scenes.workload(4)
    coords = torch.from_numpy(wl.coords).to(dev)
    ops = net.unet_ops()
    model = net.UNet(coords, ops=ops)
    model.build_maps()
    weights = model.w
    table = {}
    for op in ops:
        if op.kind != "conv":
            continue
        km = model._map(op.level, op.K, op.mode)
        x = torch.randn(km.n_in, op.c_in, device=dev).to(torch.float16)
        res = torch.randn(km.n_out, op.c_out, device=dev).to(torch.float16) if op.residual else None
        w = weights[op.out]

        def run(opt, kernel):
            f = B.Forward(km, op.c_in, op.c_out, torch.float16, opt)
            return _timed(lambda: f(x, w, residual=res, relu=op.relu), kernel, rounds)

        sc = {t: run(B.Options.make(t_scatter=t, centre=1), "k_scatter")
              for t in tile_candidates(op.c_out, 2) if 8 <= t <= 64 and (t & (t - 1)) == 0}
        gm = {r: run(B.Options.make(gemm_tile_rows=r), "k_gemm") for r in (0, *rows_cands)}
        # Algorithm 1's kernel takes tiles of 1, 2, 4, 8 or 16 16-byte vectors
        ga = {t: run(B.Options.make(t_gather=t, gather=B.GATHER_BUFFER), "k_gather")
              for t in tile_candidates(op.c_in, 2) if (t // 8) & (t // 8 - 1) == 0}
        row = {"layer": op.out, "mode": op.mode, "K": op.K, "level": op.level, "n_out": km.n_out,
               "pairs": sum(km.counts()), "c_in": op.c_in, "c_out": op.c_out,
               "scatter_us": {t: round(v * 1e3, 2) for t, v in sc.items()},
               "gemm_us": {r: round(v * 1e3, 2) for r, v in gm.items()},
               "gather_us": {t: round(v * 1e3, 2) for t, v in ga.items()},
               "t_scatter": min(sc, key=sc.get), "gemm_tile_rows": min(gm, key=gm.get),
               "t_gather": min(ga, key=ga.get)}
        print(json.dumps(row), flush=True)
        table[op.out] = row

    def forward_ms(layer_opts):
        m = net.UNet(coords, ops=ops, weights=weights, layer_opts=layer_opts)
        x0 = torch.randn(len(wl.coords), net.STEM_C, device=dev).to(torch.float16)
        for _ in range(3):
            net.UNet(coords, ops=ops, weights=weights, layer_opts=layer_opts).forward(x0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(forward_steps):
            net.UNet(coords, ops=ops, weights=weights, layer_opts=layer_opts).forward(x0)
        torch.cuda.synchronize()
        _ = m
        return (time.perf_counter() - t0) * 1e3 / forward_steps

    tuned = {k: B.Options.make(t_scatter=v["t_scatter"], gemm_tile_rows=v["gemm_tile_rows"]) for k, v in table.items()}
    res = []
    for _ in range(3):  # alternate, so drift hits both
        res.append((forward_ms(None), forward_ms(tuned)))
    d = sorted(r[0] for r in res)[1]
    t = sorted(r[1] for r in res)[1]
    print(json.dumps({"forward_ms_defaults": round(d, 4), "forward_ms_per_layer_table": round(t, 4),
                      "runs": [[round(a, 4), round(b, 4)] for a, b in res]}), flush=True)
    return table


def main(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = p.add_subparsers(dest="what", required=True)
    t = sub.add_parser("tiles")
    t.add_argument("--workload", type=int, nargs="+", default=[1])
    t.add_argument("--channels", type=int, nargs="+", default=[32, 64, 128, 256])
    t.add_argument("--rounds", type=int, default=20)
    t.add_argument("--samples", type=int, default=2)
    m = sub.add_parser("map")
    m.add_argument("--workload", type=int, nargs="+", default=[1, 3])
    m.add_argument("--rounds", type=int, default=20)
    m.add_argument("--B", type=int, nargs="+", default=[128, 256, 512, 1024, 2048, 4096])
    m.add_argument("--Cq", type=int, nargs="+", default=[256, 512, 1024, 2048])
    m.add_argument("--wg", type=int, nargs="+", default=[128, 256, 512])
    u = sub.add_parser("unet")
    u.add_argument("--rounds", type=int, default=10)
    a = p.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("tuning needs a GPU")
    if a.what == "tiles":
        tune_tiles(a.workload, a.rounds, a.samples, a.channels)
    elif a.what == "unet":
        tune_unet(a.rounds)
    else:
        tune_map(a.workload, a.rounds, a.B, a.Cq, a.wg)


if __name__ == "__main__":
    main()
