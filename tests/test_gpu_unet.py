"""GPU parity of the UNet-style network on two LiDAR-like scenes (~240k voxels, f16).

The oracle runs the same op list on its own: hash-map kernel maps per level
(upsampling maps built directly in transposed mode, not by transposing), Eq. 1
for each level's coordinates, float64 features, and float64 ReLU / residual /
concatenation.  Checked: every level's coordinates and every kernel map
bit-exactly; every layer's output within the normwise f16 tolerance (the GPU
chain stores each layer in float16, the oracle chain keeps float64).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2401_06145_amd import net, scenes
from tests.gpu_helpers import DEV, TOL, assert_map_equal, rel_err, say, to_f64

pytestmark = pytest.mark.gpu


def _oracle_unet(coords0, x0, ops):
    coords = {0: coords0}
    maps = {}

    def omap(level, K, mode):
        key = (level, K, mode)
        if key in maps:
            return maps[key]
        t = 1 << level
        if mode == "subm":
            km = oracle.kernel_map(coords[level], None, K, t, "subm")
        elif mode == "down":
            q = oracle.out_coords(coords[level], 2, t)
            coords[level + 1] = q
            km = oracle.kernel_map(coords[level], q, K, t, "down")
        else:
            omap(level - 1, K, "down")
            km = oracle.kernel_map(coords[level], coords[level - 1], K, 1 << (level - 1), "up")
        maps[key] = km
        return km

    th = oracle.max_threads()
    vals = {"x0": x0}
    for op in ops:
        if op.kind == "alias":
            vals[op.out] = vals[op.inp]
        elif op.kind == "concat":
            vals[op.out] = np.concatenate([vals[op.inp], vals[op.other]], axis=1)
        else:
            km = omap(op.level, op.K, op.mode)
            y = oracle.features(vals[op.inp], scenes.to_f64(net.weights_for(op), "f16"), km, nthreads=th)
            if op.residual:
                y = y + vals[op.residual]
            if op.relu:
                y = np.maximum(y, 0.0)
            vals[op.out] = y
    return coords, maps, vals


def test_unet_two_lidar_scenes():
    wl = scenes.workload(4)
    c0 = wl.coords
    say(f"UNet on {len(c0)} voxels (two scenes)")
    x0 = scenes.features(len(c0), net.STEM_C, "f16", 2004)
    ops = net.unet_ops()
    model = net.UNet(torch.from_numpy(c0).to(DEV))
    got = model.forward(torch.from_numpy(x0).to(DEV), keep=True)
    torch.cuda.synchronize()
    ocoords, omaps, ovals = _oracle_unet(c0, scenes.to_f64(x0, "f16"), ops)
    for lvl in range(1, 5):
        assert np.array_equal(model.coords[lvl].cpu().numpy(), ocoords[lvl]), f"level {lvl} coordinates"
    for key, okm in omaps.items():
        assert_map_equal(model.maps[key], okm)
    worst = 0.0
    for op in ops:
        if op.kind != "conv":
            continue
        e = rel_err(to_f64(got[op.out]), ovals[op.out])
        worst = max(worst, e)
        print(f"{op.out:10s} level {op.level} K={op.K} {op.mode:4s} {op.c_in:3d}->{op.c_out:3d} error {e:.2e}",
              flush=True)
        assert e <= TOL["f16"], f"{op.out}: normwise error {e}"
    print(f"worst layer error {worst:.2e}; {len([o for o in ops if o.kind == 'conv'])} convs, "
          f"level sizes {[len(ocoords[l]) for l in range(5)]}", flush=True)
