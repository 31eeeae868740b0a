"""Helpers for the GPU parity tests: run the library through the C-ABI binding and
compare with the oracle (maps as per-offset pair sets, features normwise)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2401_06145_amd import binding as B
from paper_2401_06145_amd import scenes

DEV = torch.device("cuda:0")
TOL = {"f32": 1e-4, "f16": 1e-2, "bf16": 1e-2}


def say(msg: str) -> None:
    """Names the case before its GPU work starts (flushed, so a fault still shows it)."""
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype: str | None = None) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def gpu_pairs(km: B.KernelMap):
    pin, pout, cnt = km.all_pairs()
    torch.cuda.synchronize()
    return pin.cpu().numpy(), pout.cpu().numpy(), cnt


def assert_map_equal(km: B.KernelMap, okm: oracle.KernelMap) -> None:
    """Bit-exact per-offset pair sets.  Within one offset an output row meets at most
    one input, so sorting by output row gives a unique order to compare."""
    pin, pout, cnt = gpu_pairs(km)
    assert len(cnt) == okm.K3
    assert list(cnt) == okm.counts.tolist(), f"counts differ: {cnt} vs {okm.counts.tolist()}"
    s = 0
    for k in range(okm.K3):
        n = cnt[k]
        gi, go = pin[s:s + n], pout[s:s + n]
        o = np.argsort(go, kind="stable")
        oi, oo = okm.pairs(k)
        assert np.array_equal(go[o], oo), f"offset {k}: output rows differ"
        assert np.array_equal(gi[o], oi), f"offset {k}: input rows differ"
        s += n


def rel_err(y: np.ndarray, ref: np.ndarray) -> float:
    den = np.max(np.abs(ref)) if ref.size else 0.0
    if den == 0.0:
        return float(np.max(np.abs(y))) if y.size else 0.0
    return float(np.max(np.abs(y - ref)) / den)


def elem_err(y: np.ndarray, ref: np.ndarray) -> float:
    """Element-wise statistic reported next to the gated normwise error (not gated):
    max |y - ref| / (|ref| + rms(ref))."""
    if not ref.size:
        return 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(y - ref) / (np.abs(ref) + rms))) if rms > 0 else float(np.max(np.abs(y)))


def features_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return scenes.to_f64(a, dtype)
