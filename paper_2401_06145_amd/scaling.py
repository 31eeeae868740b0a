"""Point-count scaling of the Map step on one MI355X.

Extends the paper's density study (Section 6.2: random clouds in a 400^3 volume
with 10^4 .. 10^6 points) to 16M voxels, to show where the Map kernels leave the
latency-bound regime.  For each size it builds the submanifold K = 3 map
(bounds, sort, backward search, balance, forward search, compaction) and reports
phase times from HIP events, the compulsory Map bytes per second, and each main
kernel's algorithmic bytes over its own event time.  Two scenes: uniform random
cells (the paper's Random set), and batches of LiDAR-like frames (~120k voxels
each, the outdoor recipe) up to the same sizes.

    python -m paper_2401_06145_amd.scaling --scene uniform --sizes 10000 100000 1000000 4000000 16000000
    python -m paper_2401_06145_amd.scaling --scene lidar --search sorted --sizes 1000000 4000000 16000000

``summarize`` turns the JSON rows (and rocprofv3 counter records of single-size
runs, made by profsum's ``counters`` and ``traffic`` summaries) into a Markdown
table.
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

HBM_PEAK_GBS = 8000.0


def cloud(scene: str, n: int, side: int):
    if scene == "lidar":
        return scenes.lidar_batch(n, 7000)
    return scenes.uniform_cells_large(n, side, 5000 + n % 997) if n > 1_000_000 else scenes.uniform_cells(n, side, 5000)


def measure(n: int, side: int, rounds: int, K: int = 3, hash_search: bool = False, scene: str = "uniform",
            search_opts: dict | None = None):
    dev = torch.device("cuda:0")
    c = cloud(scene, n, side)
    n = len(c)
    coords = torch.from_numpy(c).to(dev)
    opt = B.Options.make(search=1 if hash_search else 0, **(search_opts or {}))
    ws = torch.empty(B.spconv_map_workspace_bytes(n, 0, K, B.SPCONV_SUBM, opt), dtype=torch.uint8, device=dev)

    def build():
        h = B.spconv_build_map(coords, None, K, 1, 1, B.SPCONV_SUBM, opt, ws)
        B.spconv_free_map(h)
        return h

    h = B.spconv_build_map(coords, None, K, 1, 1, B.SPCONV_SUBM, opt, ws)
    pairs = sum(B.spconv_map_counts(h))
    B.spconv_free_map(h)
    for _ in range(2):
        build()
    torch.cuda.synchronize()
    ids = B.profile_ids()

    def timed(mask):
        B.spconv_profile_read(reset=True)
        B.spconv_profile_enable(mask)
        for _ in range(rounds):
            build()
        torch.cuda.synchronize()
        B.spconv_profile_enable(False)
        return B.spconv_profile_read(reset=True)

    ph = timed(B.PHASES_ALL)
    phases = {k: v[0] / rounds for k, v in ph.items() if not k.startswith("k_") and v[1] > 0}
    kern = {}
    for name in ("k_radix_scatter", "k_radix_hist", "k_backward", "k_forward_count", "k_forward_write",
                 "k_hash_insert", "k_hash_probe"):
        ms, cnt = timed(1 << ids[name])[name]
        if cnt:
            kern[name] = (ms / cnt, cnt / rounds)
    k3 = K ** 3
    map_ms = sum(phases.values())
    sort_ms = phases.get("sort", 0.0)
    # compulsory bytes: sort 28 B/voxel; search 8|Q| + 12|P| + 8M + counts
    map_bytes = 28 * n + 8 * n + 12 * n + 8 * pairs + 4 * (k3 + 1)
    passes = kern.get("k_radix_scatter", (0, 0))[1]
    per_launch = {
        "k_radix_scatter": (16 * n + 12 * n + (passes - 1) * 24 * n) / max(passes, 1),
        "k_forward_count": 8 * n + 8 * n + 4 * k3 * n,
        # reads the results and the rows of the matches; writes the pair lists and the
        # query-side table's matches (an odd-K submanifold map leaves the source-side
        # table to the first table-driven gather)
        "k_forward_write": 4 * k3 * n + 4 * n + 4 * n + 12 * pairs,
    }
    row = {"scene": scene, "voxels": n, "grid": side if scene == "uniform" else None,
           "search": "hash" if hash_search else "sorted", "pairs": pairs, "search_opts": search_opts or {},
           "map_ms": round(map_ms, 4),
           "phases_ms": {k: round(v, 4) for k, v in phases.items()},
           "map_gbps_compulsory": round(map_bytes / (map_ms * 1e-3) / 1e9, 1),
           "sort_gbps": round(28 * n / (sort_ms * 1e-3) / 1e9, 1) if sort_ms else None,
           "kernels": {}}
    for name, (ms, per_step) in kern.items():
        ent = {"mean_launch_ms": round(ms, 4), "launches_per_build": per_step}
        if name in per_launch:
            gbs = per_launch[name] / (ms * 1e-3) / 1e9
            ent.update({"gbps": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4)})
        row["kernels"][name] = ent
    return row


def main(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--sizes", type=int, nargs="+",
                   default=[10_000, 100_000, 1_000_000, 2_000_000, 4_000_000, 8_000_000, 16_000_000])
    p.add_argument("--rounds", type=int, default=10)
    p.add_argument("--search", choices=["sorted", "hash", "both"], default="both",
                   help="sorted-array search (the method), hash-table search (ablation), or both")
    p.add_argument("--scene", choices=["uniform", "lidar"], default="uniform")
    p.add_argument("--B", type=int, default=0, help="source block size (0: the library default)")
    p.add_argument("--Cq", type=int, default=0, help="query block limit (0: the library default)")
    p.add_argument("--wg", type=int, default=0, help="search workgroup size (0: the library default)")
    a = p.parse_args(argv)
    so = {k: v for k, v in (("B", a.B), ("Cq", a.Cq), ("wg", a.wg)) if v}
    if not torch.cuda.is_available():
        raise SystemExit("the sweep needs a GPU")
    for n in a.sizes:
        side = 400 if n <= 1_000_000 else 800
        for hs in ((False, True) if a.search == "both" else ((a.search == "hash"),)):
            print(json.dumps(measure(n, side, a.rounds, hash_search=hs, scene=a.scene, search_opts=so)), flush=True)


def summarize(rows_jsonl, counters, title, command, out=sys.stdout):
    """Markdown table of sorted-search rows (JSON lines) with, per size, the L2 hit
    ratio and measured HBM bytes of the Map kernels from counter records.

    counters: list of (voxels, counters_json_path, traffic_json_path)."""
    allrows = [json.loads(x) for x in open(rows_jsonl) if x.strip().startswith("{")]
    rows = [r for r in allrows if r["search"] == "sorted"]
    hashed = {r["voxels"]: r for r in allrows if r["search"] == "hash"}
    ctr = {}
    for v, cp, tp in counters:
        c = json.load(open(cp))["kernels"] if cp else {}
        t = json.load(open(tp))["kernels"] if tp else {}
        ctr[int(v)] = (c, t)
    kern = ("k_radix_scatter", "k_forward_count", "k_forward_write", "k_backward")
    lines = [f"# {title}", "", f"Command: `{command}`", "",
             "Map = bounds, sort, backward search, forward count, match scan and write pass (cold, with sort).",
             "GB/s columns: algorithmic bytes per launch over the kernel's mean event time; Map GB/s counts the",
             "compulsory bytes (28 B/voxel sort, 8|Q| + 12|P| + 8M search).  L2 hit % and measured MB/launch come",
             "from single-size rocprofv3 runs (TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum); FETCH_SIZE + WRITE_SIZE",
             "scaled by a 256 MiB copy), where taken.", "",
             "The hash-table search (the ablation: `spconv_options.search = 1`) builds the same map on the same",
             "cloud; its Map time and its ratio to the sorted search are the last two columns.", "",
             "| voxels | pairs | map ms | sort ms | forward ms | Map GB/s | radix pass GB/s | count GB/s | write GB/s |"
             " L2 hit % (radix / count / write / backward) | measured MB/launch (radix / count / write) |"
             " hash: map ms | hash / sorted |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        ph = r["phases_ms"]
        k = r["kernels"]
        c, t = ctr.get(r["voxels"], ({}, {}))
        hit = " / ".join(f"{c[x]['l2_hit_pct']:.1f}" if x in c and "l2_hit_pct" in c[x] else "-" for x in kern)
        mb = " / ".join(f"{(t[x]['fetch_bytes'] + t[x]['write_bytes']) / 1e6:.1f}" if x in t else "-"
                        for x in kern[:3])

        def g(name):
            return f"{k[name]['gbps']:.0f}" if name in k and "gbps" in k[name] else "-"
        lines.append(f"| {r['voxels']:,} | {r['pairs']:,} | {r['map_ms']:.4f} | {ph.get('sort', 0):.4f} | "
                     f"{ph.get('forward', 0):.4f} | {r['map_gbps_compulsory']:.1f} | {g('k_radix_scatter')} | "
                     f"{g('k_forward_count')} | {g('k_forward_write')} | {hit if c else '-'} | {mb if t else '-'} | "
                     + (f"{hashed[r['voxels']]['map_ms']:.4f} | {hashed[r['voxels']]['map_ms'] / r['map_ms']:.2f}x |"
                        if r["voxels"] in hashed else "- | - |"))
    print("\n".join(lines), file=out)


if __name__ == "__main__":
    main()
