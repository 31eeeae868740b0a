"""Sparse networks built from the library's layers (the paper's networks,
Section 6.1, are of these kinds): a UNet-style network (the recipe used as a
parity workload: two LiDAR-like scenes in one batch, float16) and a
SparseResNet21-style encoder with odd-K strided downsampling.

UNet wiring (channels C_in -> C_out; every conv is followed by ReLU, except the
last conv of a residual block, where ReLU follows the add):
  stem      two submanifold K=3 convs at level 0, 32 -> 32 -> 32
  encoder   4 stages (levels 1..4): K=2 s=2 downsample C_prev -> C, then two
            residual blocks of two K=3 convs; C = 32, 64, 128, 256
  decoder   4 stages (levels 3..0): K=2 s=2 transposed upsample, concatenation
            with the encoder output of that level, a residual block whose skip
            is a K=1 projection (C_up + C_skip -> C), and an identity residual
            block; C = 256, 128, 96, 96
Level l holds coordinates that are multiples of t = 2^l.

Kernel maps are built once per coordinate set and reused: submanifold maps per
level (K=3 and K=1), downsampling maps per level, and the upsampling maps as
transposes of the downsampling ones.  Level l+1's coordinates are the sorted
outputs of the level-l downsampling map, so maps on them skip the sort
(Section 5.1.1).  The GPU runner below and the CPU oracle in the tests both
interpret the same op list.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import binding as B
from . import scenes

STEM_C = 32
ENC_C = (32, 64, 128, 256)
DEC_C = (256, 128, 96, 96)


@dataclass
class Op:
    """One step of the network on named tensors."""
    kind: str            # "conv" | "concat" | "alias"
    out: str
    inp: str
    level: int = 0       # level of the input tensor
    K: int = 3
    mode: str = "subm"   # "subm" | "down" | "up"
    c_in: int = 0
    c_out: int = 0
    relu: bool = True
    residual: str | None = None
    other: str | None = None   # concat: second operand
    seed: int = 0


def unet_ops(weight_seed: int = 30_000) -> list[Op]:
    ops: list[Op] = []

    def conv(out, inp, level, K, mode, c_in, c_out, relu=True, residual=None):
        ops.append(Op("conv", out, inp, level, K, mode, c_in, c_out, relu, residual, seed=weight_seed + len(ops)))

    conv("stem1", "x0", 0, 3, "subm", STEM_C, STEM_C)
    conv("enc0", "stem1", 0, 3, "subm", STEM_C, STEM_C)
    prev, c_prev = "enc0", STEM_C
    for i, c in enumerate(ENC_C, start=1):
        conv(f"e{i}_d", prev, i - 1, 2, "down", c_prev, c)
        cur = f"e{i}_d"
        for r in range(2):
            conv(f"e{i}_r{r}_h", cur, i, 3, "subm", c, c)
            conv(f"e{i}_r{r}", f"e{i}_r{r}_h", i, 3, "subm", c, c, relu=True, residual=cur)
            cur = f"e{i}_r{r}"
        ops.append(Op("alias", f"enc{i}", cur))  # a second name for the stage output (no copy)
        prev, c_prev = f"enc{i}", c
    skips = {0: ("enc0", STEM_C), 1: ("enc1", ENC_C[0]), 2: ("enc2", ENC_C[1]), 3: ("enc3", ENC_C[2])}
    for j, c in enumerate(DEC_C, start=1):
        lvl = 4 - j  # output level of this stage
        conv(f"d{j}_u", prev, lvl + 1, 2, "up", c_prev, c)
        sk, c_sk = skips[lvl]
        ops.append(Op("concat", f"d{j}_cat", f"d{j}_u", lvl, other=sk, c_in=c + c_sk, c_out=c + c_sk))
        conv(f"d{j}_b0_h", f"d{j}_cat", lvl, 3, "subm", c + c_sk, c)
        conv(f"d{j}_b0_p", f"d{j}_cat", lvl, 1, "subm", c + c_sk, c, relu=False)
        conv(f"d{j}_b0", f"d{j}_b0_h", lvl, 3, "subm", c, c, relu=True, residual=f"d{j}_b0_p")
        conv(f"d{j}_b1_h", f"d{j}_b0", lvl, 3, "subm", c, c)
        conv(f"d{j}_b1", f"d{j}_b1_h", lvl, 3, "subm", c, c, relu=True, residual=f"d{j}_b0")
        prev, c_prev = f"d{j}_b1", c
    return ops


RES_C = (32, 64, 128, 256)


def resnet_ops(weight_seed: int = 40_000) -> list[Op]:
    """A SparseResNet21-style encoder (the paper's other network family, Section 6.1):
    a submanifold K=3 stem (32 -> 32), then 4 stages of a K=3 stride-2 convolution
    (odd-K strided downsampling; C_prev -> C) and two basic residual blocks of two K=3
    convolutions each, C = 32, 64, 128, 256: 21 convolutions."""
    ops: list[Op] = []

    def conv(out, inp, level, K, mode, c_in, c_out, relu=True, residual=None):
        ops.append(Op("conv", out, inp, level, K, mode, c_in, c_out, relu, residual, seed=weight_seed + len(ops)))

    conv("stem", "x0", 0, 3, "subm", STEM_C, RES_C[0])
    prev, c_prev = "stem", RES_C[0]
    for i, c in enumerate(RES_C, start=1):
        conv(f"s{i}_d", prev, i - 1, 3, "down", c_prev, c)
        cur = f"s{i}_d"
        for r in range(2):
            conv(f"s{i}_b{r}_h", cur, i, 3, "subm", c, c)
            conv(f"s{i}_b{r}", f"s{i}_b{r}_h", i, 3, "subm", c, c, relu=True, residual=cur)
            cur = f"s{i}_b{r}"
        prev, c_prev = cur, c
    return ops


def weights_for(op: Op, dtype: str = "f16") -> np.ndarray:
    return scenes.weights(op.K, op.c_in, op.c_out, dtype, op.seed)


class Network:
    """GPU runner of an op list: builds and caches the kernel maps, then runs the ops."""

    def __init__(self, coords: torch.Tensor, dtype: torch.dtype = torch.float16, ops: list[Op] | None = None,
                 weights: dict | None = None, layer_opts: dict | None = None):
        self.dev = coords.device
        self.dtype = dtype
        self.ops = ops or unet_ops()
        # per-layer forward options (a tuned table: op name -> binding.Options), else defaults
        self.layer_opts = layer_opts or {}
        self.coords = {0: coords}
        self.maps: dict = {}
        self.fwd: dict = {}
        dname = {torch.float16: "f16", torch.bfloat16: "bf16", torch.float32: "f32"}[dtype]
        self.w = weights if weights is not None else {}
        for op in self.ops if weights is None else []:
            if op.kind == "conv":
                w = weights_for(op, dname)
                t = torch.from_numpy(w.view(np.int16) if dname == "bf16" else w)
                self.w[op.out] = (t.view(torch.bfloat16) if dname == "bf16" else t).to(self.dev)

    def _map(self, level: int, K: int, mode: str) -> B.KernelMap:
        key = (level, K, mode)
        if key in self.maps:
            return self.maps[key]
        t = 1 << level
        presorted = B.Options.make(presorted=1) if level > 0 else None
        if mode == "subm":
            km = B.KernelMap.build(self._coords(level), K, 1, t, "subm", opt=presorted)
        elif mode == "down":
            km = B.KernelMap.build(self._coords(level), K, 2, t, "down", opt=presorted)
            self.coords[level + 1] = km.out_coords()
        else:  # up from `level` to level - 1: transpose of the level - 1 downsampling map
            km = self._map(level - 1, K, "down").transpose()
        self.maps[key] = km
        return km

    def _coords(self, level: int) -> torch.Tensor:
        if level not in self.coords:
            self._map(level - 1, 2, "down")
        return self.coords[level]

    def build_maps(self) -> None:
        for op in self.ops:
            if op.kind == "conv":
                self._map(op.level, op.K, op.mode)

    def forward(self, x0: torch.Tensor, keep: bool = False) -> dict:
        """Runs the network; returns the final output, or every named tensor if keep."""
        self.build_maps()
        t = {"x0": x0}
        for op in self.ops:
            if op.kind == "alias":
                t[op.out] = t[op.inp]
            elif op.kind == "concat":
                t[op.out] = B.spconv_concat_rows(t[op.inp], t[op.other])
            else:
                km = self._map(op.level, op.K, op.mode)
                lo = self.layer_opts.get(op.out)
                key = (id(km), op.c_in, op.c_out, op.out if lo is not None else None)
                if key not in self.fwd:
                    self.fwd[key] = B.Forward(km, op.c_in, op.c_out, self.dtype, lo)
                res = t[op.residual] if op.residual else None
                t[op.out] = self.fwd[key](t[op.inp], self.w[op.out], residual=res, relu=op.relu)
        return t if keep else {"out": t[self.ops[-1].out]}


UNet = Network  # the default op list is the UNet above
