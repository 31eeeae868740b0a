"""Dense float64 convolutions on tiny zero-filled voxel grids (torch CPU).

A sparse convolution over active sites equals a dense 3D cross-correlation over
a zero-filled grid, read back at the active output sites (Section 2.1, Eq. 2
restricted to a grid).  This is an implementation independent of the oracle:
it has no hash table and no kernel map; the library routine does the sums.

Weight layout: W[k][c_in][c_out] with k = ix K^2 + iy K + iz maps to torch's
conv3d weight w[c_out, c_in, ix, iy, iz] (conv_transpose3d: w[c_in, c_out, ...]).
Coordinates must be non-negative multiples of the spacing t.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def _torch_weight(w: np.ndarray, K: int, transposed: bool) -> torch.Tensor:
    k3, cin, cout = w.shape
    wt = torch.from_numpy(np.ascontiguousarray(w, dtype=np.float64)).reshape(K, K, K, cin, cout)
    if transposed:
        return wt.permute(3, 4, 0, 1, 2).contiguous()  # [cin, cout, K, K, K]
    return wt.permute(4, 3, 0, 1, 2).contiguous()  # [cout, cin, K, K, K]


def _low_pad(K: int) -> int:
    return (K - 1) // 2 if K % 2 == 1 else 0


def _scatter_dense(coords: np.ndarray, x: np.ndarray, t: int, dims, lo: int) -> torch.Tensor:
    g = coords[:, 1:] // t
    nb = int(coords[:, 0].max()) + 1
    dense = torch.zeros((nb, x.shape[1]) + tuple(int(d) for d in dims), dtype=torch.float64)
    b = torch.from_numpy(coords[:, 0].astype(np.int64))
    gi = [torch.from_numpy((g[:, a] + lo).astype(np.int64)) for a in range(3)]
    dense[b, :, gi[0], gi[1], gi[2]] = torch.from_numpy(np.asarray(x, dtype=np.float64))
    return dense


def _gather_dense(out: torch.Tensor, coords: np.ndarray, grid_div: int) -> np.ndarray:
    g = coords[:, 1:] // grid_div
    b = torch.from_numpy(coords[:, 0].astype(np.int64))
    gi = [torch.from_numpy(g[:, a].astype(np.int64)) for a in range(3)]
    return out[b, :, gi[0], gi[1], gi[2]].numpy().copy()


def subm(coords, x, w, K, t=1):
    """Submanifold conv: outputs at the input sites."""
    lo = _low_pad(K)
    hi = K - 1 - lo
    dims = coords[:, 1:].max(0) // t + 1 + lo + hi
    dense = _scatter_dense(coords, x, t, dims, lo)
    out = F.conv3d(dense, _torch_weight(w, K, False))
    return _gather_dense(out, coords, t)


def down(coords, x, w, K, s, t, out_coords):
    """Strided conv: outputs at out_coords (multiples of t*s)."""
    lo = _low_pad(K)
    hi = K - 1 - lo
    dims = coords[:, 1:].max(0) // t + 1 + lo + hi + s
    dense = _scatter_dense(coords, x, t, dims, lo)
    out = F.conv3d(dense, _torch_weight(w, K, False), stride=s)
    return _gather_dense(out, out_coords, t * s)


def up(coarse, x, w, K, s, t, fine):
    """Transposed conv from coarse sites (multiples of t*s) to fine sites (multiples of t)."""
    lo = _low_pad(K)
    dims = np.maximum(coarse[:, 1:].max(0) // (t * s), fine[:, 1:].max(0) // (t * s)) + 2
    dense = _scatter_dense(coarse, x, t * s, dims, 0)
    out = F.conv_transpose3d(dense, _torch_weight(w, K, True), stride=s, padding=lo)
    return _gather_dense(out, fine, t)
