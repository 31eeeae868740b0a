"""The allocation-free forward (spconv_forward_noalloc) against spconv_forward_ex.

Both run the same kernels; the allocation-free call takes its workspace from the
library's own device array, so its output must be bit-identical to the call with a
caller workspace.  Two calls in a row, the second on a smaller input, check that the
array's leftovers from the first call do not leak into the second; a layer beyond
the array's size is refused before any device work."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2401_06145_amd import binding as B
from paper_2401_06145_amd import scenes
from tests.gpu_helpers import TOL, rel_err, say, to_dev, to_f64

pytestmark = pytest.mark.gpu


def _layer(n, c, dtype, seed):
    coords = np.ascontiguousarray(scenes.workload(1).coords[:n])
    x = scenes.features(n, c, dtype, seed)
    w = scenes.weights(3, c, c, dtype, seed + 1)
    res = scenes.features(n, c, dtype, seed + 2)
    return coords, x, w, res


@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_noalloc_matches_forward_twice(dtype):
    tdt = B.TORCH_DTYPES[dtype]
    for n, c, relu in ((40000, 64, True), (9000, 32, False)):
        say(f"no-alloc forward {dtype}: {n} voxels, C={c}, relu={relu}")
        coords, x, w, res = _layer(n, c, dtype, 500 + n % 97)
        km = B.KernelMap.build(to_dev(coords), 3)
        xd, wd, rd = to_dev(x, dtype), to_dev(w, dtype), to_dev(res, dtype)
        need = B.spconv_forward_workspace_bytes(km.handle, c, c, B.DTYPES[tdt])
        assert 0 < need <= (64 << 20)
        ref = B.Forward(km, c, c, tdt)(xd, wd, residual=rd, relu=relu)
        y = torch.full((n, c), float("nan"), dtype=tdt, device=xd.device)
        B.spconv_forward_noalloc(km.handle, xd, wd, y, c, c, B.DTYPES[tdt], residual=rd, relu=relu)
        torch.cuda.synchronize()
        assert torch.equal(y, ref), "allocation-free forward differs from the forward with a workspace"
        # and both against the oracle
        okm = oracle.kernel_map(coords, None, 3, 1, "subm")
        yo = oracle.features(scenes.to_f64(x, dtype), scenes.to_f64(w, dtype), okm) + scenes.to_f64(res, dtype)
        if relu:
            yo = np.maximum(yo, 0.0)
        assert rel_err(to_f64(y), yo) <= TOL[dtype]


def test_noalloc_refuses_a_layer_beyond_its_array():
    say("no-alloc forward: layer beyond the scratch array")
    coords = np.ascontiguousarray(scenes.workload(1).coords[:60000])
    km = B.KernelMap.build(to_dev(coords), 3)
    c = 512  # partials alone: ~160k pairs x 512 x 2 bytes, beyond 64 MiB
    need = B.spconv_forward_workspace_bytes(km.handle, c, c, B.SPCONV_F16)
    assert need > (64 << 20)
    x = torch.zeros((60000, c), dtype=torch.float16, device="cuda:0")
    w = torch.zeros((27, c, c), dtype=torch.float16, device="cuda:0")
    y = torch.zeros((60000, c), dtype=torch.float16, device="cuda:0")
    with pytest.raises(B.SpconvError) as ei:
        B.spconv_forward_noalloc(km.handle, x, w, y, c, c, B.SPCONV_F16)
    assert ei.value.status == B.SPCONV_ENOSPC
