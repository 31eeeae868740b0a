"""Summaries of rocprofv3 output for the committed profiles.

  stats    kernel-trace statistics (``--kernel-trace --stats``, CSV output) as a
           Markdown table, one row per kernel, with the command that produced it.
  traffic  HBM bytes per dispatch from two counter runs (FETCH_SIZE, then
           WRITE_SIZE, in KiB per dispatch), each scaled by what the same counter
           reads for a plain device copy of known size.  Writes a Markdown table
           and a JSON record that bench.py reads for the roofline's ``traffic``
           field; the record keeps a hash of each kernel's sources, so a kernel
           changed since the counters were taken reports no traffic.
  counters MFMA utilisation (the derived ``MfmaUtil`` counter: MFMA-busy cycles
           over GPU-active cycles times SIMDs, in percent), MFMA flops executed
           (``SQ_INSTS_VALU_MFMA_MOPS_F16`` x 512, padding rows included) and the
           L2 hit ratio (``TCC_HIT_sum`` / (``TCC_HIT_sum`` + ``TCC_MISS_sum``)) per
           kernel, from counter runs of one workload.  Writes a Markdown table and
           a JSON record (with the kernels' source hashes) that bench.py reports.

Kernel names are folded to the ids of the library's timing API (e.g. both radix
scatter variants are ``k_radix_scatter``), so per-dispatch figures line up with
bench.py's per-launch timings.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re
import sys

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")

# timing-API id -> source file holding the kernel
SOURCES = {
    "k_minmax": "map_kernels.hip", "k_radix_hist": "map_kernels.hip", "k_radix_scatter": "map_kernels.hip",
    "k_radix_local": "map_kernels.hip",
    "k_pack": "map_kernels.hip", "k_down_keys": "map_kernels.hip", "k_unique": "map_kernels.hip",
    "k_backward": "map_kernels.hip", "k_forward_count": "map_kernels.hip", "k_forward_write": "map_kernels.hip",
    "k_fill": "map_kernels.hip", "k_scan": "scan.hip", "k_gather": "gmas_kernels.hip",
    "k_scatter": "gmas_kernels.hip", "k_concat": "gmas_kernels.hip", "k_gemm": "gemm_mfma.hip",
    "k_transpose_w": "gemm_mfma.hip", "k_ts_from_pairs": "map_kernels.hip", "k_inverse_perm": "map_kernels.hip",
    "k_hash_insert": "map_kernels.hip", "k_hash_count": "map_kernels.hip", "k_hash_items": "map_kernels.hip",
    "k_scatter_centre": "gemm_mfma.hip",
}

FOLD = [
    (r"k_radix_(tile_scatter|pass)\b", "k_radix_scatter"),
    (r"k_radix_(tile_hist|upsweep)\b", "k_radix_hist"),
    (r"k_bucket_sort\b", "k_radix_local"),
    (r"k_forward_count\b", "k_forward_count"),
    (r"k_forward_write\b", "k_forward_write"),
    (r"k_gemm(_wide)?\b", "k_gemm"),
    (r"k_tile_(scan|reduce)\b", "k_scan"),
    (r"k_minmax_(partial|final)\b|k_layout\b", "k_minmax"),
    (r"k_scatter(_rows)?\b", "k_scatter"),
    (r"k_unique_(flags|write|tile_count|tile_write)\b", "k_unique"),
    (r"k_fill_u32\b", "k_fill"),
    (r"k_transpose_w(64)?\b", "k_transpose_w"),
]


def fold(name: str) -> str:
    for pat, rep in FOLD:
        if re.search(pat, name):
            return rep
    m = re.search(r"::(k_\w+)", name)
    if m:
        return m.group(1)
    return name.split("(")[0][:60]


def source_hash(kid: str) -> str | None:
    src = SOURCES.get(kid)
    if not src:
        return None
    h = hashlib.sha256()
    for f in ("common.h", src):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def cmd_stats(a) -> None:
    rows = list(csv.DictReader(open(a.csv)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    out = [f"# {a.title}", "", f"Command: `{a.command}`", "",
           "rocprofv3 kernel-trace statistics (all dispatches of the run, including the bench's",
           "warm-up and breakdown passes).", "",
           "| kernel | timing id | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"]
        short = re.sub(r"\(.*", "", name.replace("spc::(anonymous namespace)::", "")).replace("void ", "")
        out.append(f"| `{short[:70]}` | {fold(name)} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                   f"{float(r['TotalDurationNs']) / total * 100:.1f}% |")
    # per timing id: the mean over all dispatches of the kernels folded into it
    agg = collections.defaultdict(lambda: [0, 0.0])
    for r in rows:
        d = agg[fold(r["Name"])]
        d[0] += int(r["Calls"])
        d[1] += float(r["TotalDurationNs"])
    out += ["", "Per timing id (what bench.py's per-launch means compare with):", "",
            "| timing id | dispatches | mean us |", "|---|---|---|"]
    for kid, (n, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {kid} | {n} | {t / n / 1e3:.2f} |")
    print("\n".join(out))


def robust_mean(vals: list[float]) -> float:
    """Mean over dispatches, leaving out readings above 4x the median: the first
    dispatch of a kernel in a counter run has read tens to millions of times its
    steady value (a cold first build, or a wrapped-around counter), while the
    dispatches of one kernel in a run otherwise differ by well under 2x."""
    s = sorted(vals)
    med = s[len(s) // 2]
    keep = [v for v in vals if med <= 0 or v <= 4 * med]
    return sum(keep) / len(keep)


def _counter(path: str, counter: str) -> dict[str, list[float]]:
    per = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") == counter:
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return per


def _copy_scale(path: str, counter: str, true_bytes: float) -> float:
    per = _counter(path, counter)
    # the copy's dispatches are the ones with the most traffic
    name = max(per, key=lambda k: robust_mean(per[k]))
    kib = robust_mean(per[name])
    return true_bytes / (kib * 1024.0)


def cmd_traffic(a) -> None:
    nbytes = a.copy_mib * 1024 * 1024
    fs = _copy_scale(a.copy_fetch, "FETCH_SIZE", nbytes)
    ws = _copy_scale(a.copy_write, "WRITE_SIZE", nbytes)
    fetch = _counter(a.fetch, "FETCH_SIZE")
    write = _counter(a.write, "WRITE_SIZE")
    agg = {}
    for src, key in ((fetch, "fetch"), (write, "write")):
        for name, vals in src.items():
            kid = fold(name)
            d = agg.setdefault(kid, {"fetch": [], "write": []})
            d[key].extend(vals)
    rec = {"command_fetch": a.command_fetch, "command_write": a.command_write, "workload": a.workload,
           "fetch_scale": fs, "write_scale": ws, "copy_mib": a.copy_mib, "kernels": {}}
    lines = [f"# {a.title}", "", f"Counter runs: `{a.command_fetch}` and `{a.command_write}`;",
             f"calibration: the same two counters over a plain {a.copy_mib} MiB device copy "
             f"(`{a.command_copy}`), giving scale factors FETCH x{fs:.3f}, WRITE x{ws:.3f}.", "",
             "Bytes per dispatch (mean over the run's dispatches, readings above 4x the median left out),",
             "after scaling.", "",
             "| timing id | dispatches | HBM read MB | HBM write MB | total MB |", "|---|---|---|---|---|"]
    for kid, d in sorted(agg.items(), key=lambda t: -(sum(t[1]["fetch"]) + sum(t[1]["write"]))):
        if not d["fetch"] or not d["write"]:
            continue
        fb = robust_mean(d["fetch"]) * 1024 * fs
        wb = robust_mean(d["write"]) * 1024 * ws
        rec["kernels"][kid] = {"dispatches": len(d["fetch"]), "fetch_bytes": fb, "write_bytes": wb,
                               "source_sha256": source_hash(kid)}
        lines.append(f"| {kid} | {len(d['fetch'])} | {fb / 1e6:.3f} | {wb / 1e6:.3f} | {(fb + wb) / 1e6:.3f} |")
    with open(a.json, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    print("\n".join(lines))


def cmd_counters(a) -> None:
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for path in a.csv:
        for r in csv.DictReader(open(path)):
            vals[fold(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    rec = {"workload": a.workload, "commands": a.command, "kernels": {}}
    lines = [f"# {a.title}", "", "Counter runs (one rocprofv3 pass per counter group):", ""]
    lines += [f"* `{c}`" for c in a.command]
    lines += ["", "Per dispatch, mean over the runs' dispatches (readings above 4x the median left out).",
              "MFMA utilisation is rocprofv3's derived",
              "`MfmaUtil`; executed MFMA flops count every row the MFMAs process (padding and masked",
              "rows included); L2 hit ratio = TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum).", "",
              "| timing id | dispatches | MFMA util % | MFMA flops executed / dispatch | L2 hit % | L2 requests / dispatch |",
              "|---|---|---|---|---|---|"]
    for kid, d in sorted(vals.items()):
        k = {"source_sha256": source_hash(kid)}
        n = max(len(v) for v in d.values())
        # MFMA figures only for kernels that run MFMAs
        if d.get("SQ_INSTS_VALU_MFMA_MOPS_F16") and sum(d["SQ_INSTS_VALU_MFMA_MOPS_F16"]) > 0:
            k["mfma_flops_executed"] = 512.0 * robust_mean(d["SQ_INSTS_VALU_MFMA_MOPS_F16"])
            if d.get("MfmaUtil"):
                k["mfma_util_pct"] = robust_mean(d["MfmaUtil"])
        if d.get("TCC_HIT_sum") and d.get("TCC_MISS_sum"):
            hit, miss = robust_mean(d["TCC_HIT_sum"]), robust_mean(d["TCC_MISS_sum"])
            if hit + miss > 0:
                k["l2_hit_pct"] = 100.0 * hit / (hit + miss)
                k["l2_requests_per_dispatch"] = hit + miss
        if len(k) == 1:
            continue
        rec["kernels"][kid] = k

        def f(key, fmt):
            return fmt.format(k[key]) if key in k else "-"
        lines.append(f"| {kid} | {n} | {f('mfma_util_pct', '{:.1f}')} | {f('mfma_flops_executed', '{:.3e}')} | "
                     f"{f('l2_hit_pct', '{:.1f}')} | {f('l2_requests_per_dispatch', '{:.3e}')} |")
    with open(a.json, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    print("\n".join(lines))


def main(argv=None) -> None:
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = p.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--command", required=True)
    s.add_argument("--title", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-mib", type=int, required=True)
    t.add_argument("--command-fetch", required=True)
    t.add_argument("--command-write", required=True)
    t.add_argument("--command-copy", required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--title", required=True)
    t.add_argument("--json", required=True)
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--command", action="append", required=True)
    c.add_argument("--workload", required=True)
    c.add_argument("--title", required=True)
    c.add_argument("--json", required=True)
    a = p.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic, "counters": cmd_counters}[a.cmd](a)


if __name__ == "__main__":
    main(sys.argv[1:])
