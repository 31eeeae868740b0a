"""GPU parity of the SparseResNet21-style encoder (odd-K strided downsampling) in
bfloat16 on the 120k LiDAR scene.

Every level's coordinates and every kernel map (including the K=3 stride-2
downsampling maps) are checked bit-exactly against the oracle's.  Each of the 21
layers is checked on its own: the oracle gets the GPU's own layer input (and
residual) widened exactly to float64, so the per-layer normwise bf16 tolerance
bounds that layer's error, not the chain's.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2401_06145_amd import net, scenes
from tests.gpu_helpers import DEV, TOL, assert_map_equal, rel_err, say, to_f64

pytestmark = pytest.mark.gpu


def test_resnet_bf16_per_layer():
    wl = scenes.workload(1)
    c0 = wl.coords
    say(f"ResNet21-style encoder, bf16, {len(c0)} voxels")
    ops = net.resnet_ops()
    x0 = scenes.features(len(c0), net.STEM_C, "bf16", 4001)
    x0_t = torch.from_numpy(x0.view(np.int16)).view(torch.bfloat16).to(DEV)
    model = net.Network(torch.from_numpy(c0).to(DEV), dtype=torch.bfloat16, ops=ops)
    got = model.forward(x0_t, keep=True)
    torch.cuda.synchronize()

    coords = {0: c0}
    for lvl in range(1, 5):
        coords[lvl] = oracle.out_coords(coords[lvl - 1], 2, 1 << (lvl - 1))
        assert np.array_equal(model.coords[lvl].cpu().numpy(), coords[lvl]), f"level {lvl} coordinates"
    th = oracle.max_threads()
    worst = 0.0
    for op in ops:
        t = 1 << op.level
        if op.mode == "subm":
            okm = oracle.kernel_map(coords[op.level], None, op.K, t, "subm")
        else:
            okm = oracle.kernel_map(coords[op.level], coords[op.level + 1], op.K, t, "down")
        assert_map_equal(model.maps[(op.level, op.K, op.mode)], okm)
        xin = to_f64(got[op.inp])
        y = oracle.features(xin, scenes.to_f64(net.weights_for(op, "bf16"), "bf16"), okm, nthreads=th)
        if op.residual:
            y = y + to_f64(got[op.residual])
        if op.relu:
            y = np.maximum(y, 0.0)
        e = rel_err(to_f64(got[op.out]), y)
        worst = max(worst, e)
        print(f"{op.out:8s} level {op.level} K={op.K} {op.mode:4s} {op.c_in:3d}->{op.c_out:3d} error {e:.2e}",
              flush=True)
        assert e <= TOL["bf16"], f"{op.out}: normwise error {e}"
    print(f"worst layer error {worst:.2e}; level sizes {[len(coords[l]) for l in range(5)]}", flush=True)
