"""GPU parity: the HIP library (through the C-ABI) against the CPU oracle.

Kernel maps must match bit-exactly as per-offset pair sets; features must be
within the normwise tolerance max|y - y_ref| / max|y_ref| <= 1e-4 (f32) or
1e-2 (f16, bf16).  Inputs are seeded; expected values come from the oracle only.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2401_06145_amd import binding as B
from paper_2401_06145_amd import scenes
from tests.gpu_helpers import DEV, TOL, assert_map_equal, elem_err, gpu_pairs, rel_err, say, to_dev, to_f64

pytestmark = pytest.mark.gpu


def _cloud(seed, n, lo, hi, nb=2, t=1):
    rng = np.random.default_rng(seed)
    side = hi - lo
    cells = rng.choice(nb * side ** 3, n, replace=False)
    b = cells // side ** 3
    r = cells % side ** 3
    x, y, z = r // side ** 2 + lo, (r // side) % side + lo, r % side + lo
    c = np.stack([b, x * t, y * t, z * t], axis=1).astype(np.int32)
    return np.ascontiguousarray(c)


def _conv_gpu(coords, x, w, K, stride=1, t=1, mode="subm", out_coords=None, opt=None, dtype="f32"):
    dc = to_dev(coords)
    doc = to_dev(out_coords) if out_coords is not None else None
    km = B.KernelMap.build(dc, K, stride, t, mode, doc, opt)
    f = B.Forward(km, x.shape[1], w.shape[2], B.TORCH_DTYPES[dtype], opt)
    y = f(to_dev(x, dtype), to_dev(w, dtype))
    torch.cuda.synchronize()
    return km, y


# ----------------------------------------------------------------------------
# Small clouds: many source blocks, pivot edges, split query blocks
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("K", [1, 2, 3, 5])
@pytest.mark.parametrize("Bsz,Cq", [(64, 256), (256, 512), (1024, 2048)])
def test_subm_small(K, Bsz, Cq):
    say(f"subm small K={K} B={Bsz} Cq={Cq}")
    c = _cloud(10 + K, 3000, -9, 9)
    x = scenes.features(len(c), 16, "f32", 1)
    w = scenes.weights(K, 16, 16, "f32", 2)
    opt = B.Options.make(B=Bsz, Cq=Cq)
    km, y = _conv_gpu(c, x, w, K, opt=opt)
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    assert_map_equal(km, okm)
    ref = oracle.features(x, w, okm)
    assert rel_err(to_f64(y), ref) <= TOL["f32"]


@pytest.mark.parametrize("wg,Cq", [(128, 256), (128, 1024), (512, 512), (512, 2048)])
def test_search_workgroup_sizes(wg, Cq):
    """The forward search's workgroup size (Section 5.1.4's thread-block size) changes
    only the launch shape: maps equal the oracle's, SUBM and DOWN."""
    say(f"search workgroup size {wg}, Cq {Cq}")
    c = _cloud(60, 6000, -12, 12)
    opt = B.Options.make(B=256, Cq=Cq, wg=wg)
    km = B.KernelMap.build(to_dev(c), 3, opt=opt)
    assert_map_equal(km, oracle.kernel_map(c, None, 3, 1, "subm"))
    kd = B.KernelMap.build(to_dev(c), 2, 2, 1, "down", opt=opt)
    q = oracle.out_coords(c, 2, 1)
    assert np.array_equal(kd.out_coords().cpu().numpy(), q)
    assert_map_equal(kd, oracle.kernel_map(c, q, 2, 1, "down"))


@pytest.mark.parametrize("G", [2, 3, 9, 27, 64])
def test_count_pass_offset_groups(G):
    """Offsets per count-pass workgroup change only the launch shape.  Groups of
    several offsets search runs of nearby query blocks together (runs split where
    the x offset changes, blocks empty for some offsets): the maps equal the
    oracle's, SUBM with K = 3 and 5 (K^3 = 125: groups capped at 64), DOWN and UP."""
    say(f"count-pass offset groups G={G}")
    c = _cloud(61, 5000, -11, 11)
    opt = B.Options.make(B=64, Cq=256, count_group=G)
    for K in (3, 5):
        km = B.KernelMap.build(to_dev(c), K, opt=opt)
        assert_map_equal(km, oracle.kernel_map(c, None, K, 1, "subm"))
    # a sparse cloud: many source blocks see no queries at some offsets
    sp = _cloud(62, 1500, -40, 40)
    assert_map_equal(B.KernelMap.build(to_dev(sp), 3, opt=opt), oracle.kernel_map(sp, None, 3, 1, "subm"))
    kd = B.KernelMap.build(to_dev(c), 2, 2, 1, "down", opt=opt)
    q = oracle.out_coords(c, 2, 1)
    assert_map_equal(kd, oracle.kernel_map(c, q, 2, 1, "down"))
    ku = B.KernelMap.build(to_dev(q), 3, 2, 1, "up", to_dev(c), opt)
    assert_map_equal(ku, oracle.kernel_map(q, c, 3, 1, "up"))


@pytest.mark.parametrize("c", [64, 256])
def test_gemm_tile_rows_result_neutral(c):
    """Rows per GEMM workgroup tile change the launch shape only: bit-identical output."""
    say(f"GEMM tile rows, C={c}")
    cl = scenes.workload(1).coords[:30000].copy()
    x = scenes.features(len(cl), c, "f16", 21)
    w = scenes.weights(3, c, c, "f16", 22)
    km = B.KernelMap.build(to_dev(cl), 3)
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    base = B.Forward(km, c, c, torch.float16)(xd, wd)
    for rows in (16, 100, 512, 5000, 1 << 20):
        y = B.Forward(km, c, c, torch.float16, B.Options.make(gemm_tile_rows=rows))(xd, wd)
        assert torch.equal(y, base), f"gemm_tile_rows={rows} changed the result"


@pytest.mark.parametrize("K,s,t", [(2, 2, 1), (3, 2, 1), (2, 2, 2), (2, 3, 1), (3, 3, 2)])
@pytest.mark.parametrize("Bsz", [64, 256])
def test_down_up_small(K, s, t, Bsz):
    say(f"down/up small K={K} s={s} t={t} B={Bsz}")
    c = _cloud(20 + K + s, 2500, -10, 10, t=t)
    x = scenes.features(len(c), 8, "f32", 3)
    w = scenes.weights(K, 8, 16, "f32", 4)
    opt = B.Options.make(B=Bsz, Cq=256)
    km, y = _conv_gpu(c, x, w, K, s, t, "down", opt=opt)
    q = oracle.out_coords(c, s, t)
    qg = km.out_coords().cpu().numpy()
    assert np.array_equal(qg, q), "DOWN output coordinates differ from Eq. 1"
    okm = oracle.kernel_map(c, q, K, t, "down")
    assert_map_equal(km, okm)
    assert rel_err(to_f64(y), oracle.features(x, w, okm)) <= TOL["f32"]
    # transposed conv back to the fine sites: built directly, and by transposing
    xc = scenes.features(len(q), 16, "f32", 5)
    wu = scenes.weights(K, 16, 16, "f32", 6)
    oup = oracle.kernel_map(q, c, K, t, "up")
    yref = oracle.features(xc, wu, oup)
    kup, yu = _conv_gpu(q, xc, wu, K, s, t, "up", out_coords=c, opt=opt)
    assert_map_equal(kup, oup)
    assert rel_err(to_f64(yu), yref) <= TOL["f32"]
    kt = km.transpose()
    yt = B.Forward(kt, 16, 16, torch.float32)(to_dev(xc), to_dev(wu))
    torch.cuda.synchronize()
    assert_map_equal(kt, oup)
    assert rel_err(to_f64(yt), yref) <= TOL["f32"]


def test_negative_and_wide_coordinates():
    say("negative / wide coordinates")
    rng = np.random.default_rng(5)
    base = _cloud(30, 2000, -6, 6)
    base[:, 1] = base[:, 1] * 1000 - 7          # wide, negative x
    base[:, 3] = base[:, 3] - 100000            # far negative z
    assert len(np.unique(base, axis=0)) == len(base)
    x = scenes.features(len(base), 4, "f32", 7)
    w = scenes.weights(3, 4, 16, "f32", 8)
    km, y = _conv_gpu(base, x, w, 3)
    okm = oracle.kernel_map(base, None, 3, 1, "subm")
    assert_map_equal(km, okm)
    assert rel_err(to_f64(y), oracle.features(x, w, okm)) <= TOL["f32"]
    _ = rng


def test_sort_pass_planning_wide_then_narrow():
    """The host plans the sort's passes before the device has laid out the keys:
    a key wider than planned is detected and the build redone with enough passes;
    a narrower one runs the extra passes as copies.  Wide (41-bit), narrow and
    wide-again clouds in turn, each checked against the oracle's map; DOWN maps
    sort their output keys with the same plan."""
    say("sort pass planning")
    narrow = _cloud(40, 3000, -8, 8)                       # ~14 key bits
    wide = _cloud(41, 3000, -8, 8)
    wide[:, 1] *= 400                                      # x, y, z over ~2^12 each
    wide[:, 2] *= 300
    wide[:, 3] *= 500
    wide[:, 0] += 2                                        # b up to 3
    assert len(np.unique(wide, axis=0)) == len(wide)
    for c, mode, K, s_ in ((wide, "subm", 3, 1), (narrow, "subm", 3, 1), (wide, "down", 2, 2),
                           (narrow, "down", 3, 2), (wide, "subm", 3, 1)):
        dc = to_dev(c)
        km = B.KernelMap.build(dc, K, s_, 1, mode)
        q = oracle.out_coords(c, s_, 1) if mode == "down" else None
        okm = oracle.kernel_map(c, q, K, 1, mode)
        assert_map_equal(km, okm)
        if mode == "down":
            assert np.array_equal(km.out_coords().cpu().numpy(), q)


# ----------------------------------------------------------------------------
# Hand example and the paper's segment example
# ----------------------------------------------------------------------------

def test_hand_two_voxel_example():
    say("hand two-voxel example")
    p = np.array([[0, 0, 0, 0], [0, 1, 0, 0]], np.int32)
    x = np.zeros((2, 4), np.float32)
    x[:, 0] = [1, 2]
    w = np.zeros((27, 4, 16), np.float32)
    w[:, 0, 0] = np.arange(27) + 1
    km, y = _conv_gpu(p, x, w, 3)
    assert y[:, 0].cpu().tolist() == [60.0, 33.0]
    assert float(y[:, 1:].abs().max()) == 0.0
    w2 = np.zeros((8, 4, 16), np.float32)
    w2[:, 0, 0] = np.arange(8) + 1
    kd, yd = _conv_gpu(p, x, w2, 2, 2, 1, "down")
    assert yd[:, 0].cpu().tolist() == [11.0]
    xc = np.zeros((1, 16), np.float32)
    xc[0, 0] = 3
    w3 = np.zeros((8, 16, 16), np.float32)
    w3[:, 0, 0] = np.arange(8) + 1
    yu = B.Forward(kd.transpose(), 16, 16, torch.float32)(to_dev(xc), to_dev(w3))
    assert yu[:, 0].cpu().tolist() == [3.0, 15.0]


# ----------------------------------------------------------------------------
# Workloads at full size
# ----------------------------------------------------------------------------

def _workload_layer(i, c=None, rows=None):
    wl = scenes.workload(i, c)
    L = wl.layers[0]
    coords = wl.coords
    say(f"workload {i} ({wl.name}): {len(coords)} voxels")
    x = scenes.features(len(coords), L.c_in, L.dtype, 2000 + i)
    w = scenes.weights(L.K, L.c_in, L.c_out, L.dtype, 3000 + i)
    km, y = _conv_gpu(coords, x, w, L.K, L.stride, 1, L.mode, dtype=L.dtype)
    okm = oracle.kernel_map(coords, None, L.K, 1, "subm")
    assert_map_equal(km, okm)
    xf, wf = scenes.to_f64(x, L.dtype), scenes.to_f64(w, L.dtype)
    if rows is None:
        ref = oracle.features(xf, wf, okm)
        got = to_f64(y)
    else:
        sel = np.sort(np.random.default_rng(99).choice(len(coords), rows, replace=False))
        ref = oracle.features(xf, wf, okm, rows=sel)
        got = to_f64(y)[sel]
    err = rel_err(got, ref)
    print(f"workload {i} c={L.c_in}: pairs={sum(km.counts())} normwise error {err:.3e} "
          f"(element-wise max |y-ref|/(|ref|+rms(ref)) {elem_err(got, ref):.3e}, rows "
          f"{'all' if rows is None else rows})", flush=True)
    assert err <= TOL[L.dtype]
    return km, okm


def test_workload0_uniform_f32():
    _workload_layer(0)


def test_workload1_lidar_f16():
    _workload_layer(1)


@pytest.mark.parametrize("c", [32, 64, 128, 256])
def test_workload3_indoor_f16(c):
    # every output row up to C = 64; 4000 sampled rows at C = 128 and 256, where the
    # oracle's float64 sums over all 300k rows would take minutes
    _workload_layer(3, c, rows=None if c <= 64 else 4000)


def test_streamed_outputs_of_the_plain_scatter():
    """The 300k indoor scene at C = 256 with the centre offset through the GEMM: the
    plain scatter writes 154 MB of outputs and the GEMM 525 MB of partials, both
    past the sizes from which they go out with non-temporal stores.  The row-group
    and the tiled scatter give the same bits (also with float32 partials), within
    tolerance of the oracle on sampled rows."""
    wl = scenes.workload(3, 256)
    L = wl.layers[0]
    coords = wl.coords
    say(f"streamed plain scatter, {len(coords)} voxels, C=256")
    x = scenes.features(len(coords), 256, "f16", 2203)
    w = scenes.weights(3, 256, 256, "f16", 3203)
    km = B.KernelMap.build(to_dev(coords), 3)
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    y_row = B.Forward(km, 256, 256, torch.float16, B.Options.make(centre=1))(xd, wd)
    y_tiled = B.Forward(km, 256, 256, torch.float16, B.Options.make(centre=1, t_scatter=16))(xd, wd)
    assert torch.equal(y_row, y_tiled)
    y32 = B.Forward(km, 256, 256, torch.float16, B.Options.make(centre=1, partial_dtype=1))(xd, wd)
    y32t = B.Forward(km, 256, 256, torch.float16, B.Options.make(centre=1, partial_dtype=1, t_scatter=16))(xd, wd)
    assert torch.equal(y32, y32t)
    okm = oracle.kernel_map(coords, None, 3, 1, "subm")
    sel = np.sort(np.random.default_rng(98).choice(len(coords), 3000, replace=False))
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm, rows=sel)
    assert rel_err(to_f64(y_row)[sel], ref) <= TOL["f16"]
    assert rel_err(to_f64(y32)[sel], ref) <= TOL["f16"]


def test_workload2_down_up_f16():
    wl = scenes.workload(2)
    coords = wl.coords
    say(f"workload 2: {len(coords)} voxels")
    Ld, Lu = wl.layers
    x = scenes.features(len(coords), Ld.c_in, "f16", 2002)
    w = scenes.weights(2, Ld.c_in, Ld.c_out, "f16", 3002)
    km, y = _conv_gpu(coords, x, w, 2, 2, 1, "down", dtype="f16")
    q = oracle.out_coords(coords, 2, 1)
    assert np.array_equal(km.out_coords().cpu().numpy(), q)
    okm = oracle.kernel_map(coords, q, 2, 1, "down")
    assert_map_equal(km, okm)
    assert okm.counts.sum() == len(coords)
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm)
    assert rel_err(to_f64(y), ref) <= TOL["f16"]
    # upsample back with the transposed map; the oracle uses its own inputs
    xc = scenes.features(len(q), Lu.c_in, "f16", 2102)
    wu = scenes.weights(2, Lu.c_in, Lu.c_out, "f16", 3102)
    kt = km.transpose()
    yu = B.Forward(kt, Lu.c_in, Lu.c_out, torch.float16)(to_dev(xc), to_dev(wu))
    torch.cuda.synchronize()
    oup = oracle.kernel_map(q, coords, 2, 1, "up")
    assert_map_equal(kt, oup)
    refu = oracle.features(scenes.to_f64(xc, "f16"), scenes.to_f64(wu, "f16"), oup)
    assert rel_err(to_f64(yu), refu) <= TOL["f16"]


# ----------------------------------------------------------------------------
# Parity-neutral parameters, determinism, dtypes
# ----------------------------------------------------------------------------

def test_grouping_tiles_partials_are_result_neutral():
    say("grouping / tiles / partial precision")
    c = scenes.workload(1).coords[:40000].copy()
    x = scenes.features(len(c), 64, "f16", 11)
    w = scenes.weights(3, 64, 64, "f16", 12)
    dc = to_dev(c)
    km = B.KernelMap.build(dc, 3)
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    # the centre offset through the GEMM, like the other offsets (the tiles apply)
    base = B.Forward(km, 64, 64, torch.float16, B.Options.make(centre=1))(xd, wd)
    # the default computes the centre inside the scatter
    base_c = B.Forward(km, 64, 64, torch.float16)(xd, wd)
    infos = []
    for g in (B.GROUP_RAGGED, B.GROUP_SORTED, B.GROUP_MAPORDER):
        for tg, ts in ((8, 8), (16, 16), (64, 32), (32, 64)):
            opt = B.Options.make(grouping=g, t_gather=tg, t_scatter=ts, gather=B.GATHER_BUFFER)
            y = B.Forward(km, 64, 64, torch.float16, opt)(xd, wd)
            assert torch.equal(y, base), f"grouping {g} tiles {tg}/{ts} changed the result"
        y = B.Forward(km, 64, 64, torch.float16, B.Options.make(grouping=g))(xd, wd)
        assert torch.equal(y, base_c), f"grouping {g} changed the result with the centre in the scatter"
        infos.append(km.plan(64, 64, torch.float16, B.Options.make(grouping=g)))
    # sorted grouping never pads more than map-order grouping with the same cost model
    assert infos[0].rows_padded == infos[0].rows_real
    assert infos[1].rows_padded <= infos[2].rows_padded
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm)
    # float32 partials; the default float16 partials keep a 3x margin under the f16 tolerance
    y32 = B.Forward(km, 64, 64, torch.float16, B.Options.make(partial_dtype=1, t_scatter=4))(xd, wd)
    e32, e16 = rel_err(to_f64(y32), ref), rel_err(to_f64(base), ref)
    ec = rel_err(to_f64(base_c), ref)
    print(f"normwise error: float32 partials {e32:.2e}, float16 partials {e16:.2e}, "
          f"float16 partials with the centre in the scatter {ec:.2e}", flush=True)
    assert e32 <= TOL["f16"] and e16 <= TOL["f16"] / 3 and ec <= TOL["f16"] / 3


@pytest.mark.parametrize("K,c_out,pd", [
    (3, 16, 0),     # two lanes per output row, 32 groups per wave
    (3, 96, 0),     # 12 lanes per row: five groups per wave, four idle lanes
    (5, 64, 0),     # 125 offsets: several table batches per lane
    (3, 512, 0),    # one wave per row
    (3, 1024, 0),   # two vectors per lane
    (3, 256, 1),    # float32 partials: four channels per lane
    (5, 16, 1),
])
def test_row_scatter_matches_tiled_and_oracle(K, c_out, pd):
    """The row-group scatter (default tile) and the tiled scatter sum the same
    partials in the same offset order: identical outputs, also with the fused
    residual + ReLU epilogue; both within tolerance of the oracle."""
    say(f"row scatter K={K} c_out={c_out} partials={'f32' if pd else 'f16'}")
    c = _cloud(70 + K, 3000, -6, 6)
    x = scenes.features(len(c), 32, "f16", 71)
    w = scenes.weights(K, 32, c_out, "f16", 72)
    km = B.KernelMap.build(to_dev(c), K)
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    res = to_dev(scenes.features(len(c), c_out, "f16", 73), "f16")
    row = B.Options.make(partial_dtype=pd, centre=1)
    tiled = B.Options.make(partial_dtype=pd, t_scatter=16, centre=1)
    assert km.plan(32, c_out, torch.float16, row).t_scatter == (4 if pd else 8)
    y_row = B.Forward(km, 32, c_out, torch.float16, row)(xd, wd)
    y_tiled = B.Forward(km, 32, c_out, torch.float16, tiled)(xd, wd)
    assert torch.equal(y_row, y_tiled)
    e_row = B.Forward(km, 32, c_out, torch.float16, row)(xd, wd, residual=res, relu=True)
    e_tiled = B.Forward(km, 32, c_out, torch.float16, tiled)(xd, wd, residual=res, relu=True)
    assert torch.equal(e_row, e_tiled)
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm)
    assert rel_err(to_f64(y_row), ref) <= TOL["f16"]
    ref_e = np.maximum(ref + to_f64(res), 0.0)
    assert rel_err(to_f64(e_row), ref_e) <= TOL["f16"]


@pytest.mark.parametrize("dtype,c_in,c_out,pd", [
    ("f32", 16, 32, 0),     # fallback kernel
    ("f16", 16, 16, 0),     # half of one 32-deep k-step is padding
    ("f16", 48, 64, 0),     # padding inside the second k-step
    ("f16", 64, 64, 1),     # float32 partials
    ("bf16", 64, 32, 1),    # fallback kernel, bf16
    ("bf16", 96, 32, 0),
    ("f16", 256, 128, 0),   # W^T staged from the transposed copy
    ("f16", 384, 256, 0),   # two column slices per tile, their workgroups 8 ids apart
    ("f16", 512, 256, 1),   # the same with float32 partials
])
def test_gather_forms_bit_identical(dtype, c_in, c_out, pd):
    """GEMMs that load each pair's input row directly (the fused gather) see the
    same operands in the same order as GEMMs reading Algorithm 1's gathered
    buffer, so the two forms agree bit for bit, with and without group padding."""
    say(f"gather forms {dtype} {c_in}->{c_out} partials {pd}")
    c = _cloud(77, 6000, -12, 12)
    x = scenes.features(len(c), c_in, dtype, 21)
    w = scenes.weights(3, c_in, c_out, dtype, 22)
    km = B.KernelMap.build(to_dev(c), 3)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    td = B.TORCH_DTYPES[dtype]
    ys = {}
    for g in (B.GATHER_BUFFER, B.GATHER_FUSED):
        for grp in (B.GROUP_RAGGED, B.GROUP_SORTED):
            opt = B.Options.make(gather=g, grouping=grp, partial_dtype=pd, centre=1)
            assert km.plan(c_in, c_out, td, opt).gather == g
            ys[g, grp] = B.Forward(km, c_in, c_out, td, opt)(xd, wd)
    assert km.plan(c_in, c_out, td).gather == B.GATHER_FUSED  # the default
    base = ys[B.GATHER_BUFFER, B.GROUP_RAGGED]
    for key, y in ys.items():
        assert torch.equal(y, base), f"gather form / grouping {key} changed the result"
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, dtype), scenes.to_f64(w, dtype), okm)
    assert rel_err(to_f64(base), ref) <= TOL[dtype]


@pytest.mark.parametrize("search,K", [(0, 3), (0, 5), (1, 3), (1, 5)])
def test_source_table_filled_on_first_table_gather(search, K):
    """An odd-K submanifold map leaves its source-side metadata table to the first
    forward call that gathers through it (the table is filled from the pair
    lists then).  Sorted-search maps index the table by sorted position,
    hash-table maps by caller row.  Two table-driven calls must equal the fused
    gather's output bit for bit, and the oracle within tolerance."""
    say(f"source-side table on first use, search={search} K={K}")
    c = _cloud(300 + 10 * search + K, 5000, -11, 11)
    x = scenes.features(len(c), 32, "f16", 301)
    w = scenes.weights(K, 32, 32, "f16", 302)
    km = B.KernelMap.build(to_dev(c), K, opt=B.Options.make(search=search))
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    td = B.TORCH_DTYPES["f16"]
    y_fused = B.Forward(km, 32, 32, td, B.Options.make(gather=B.GATHER_FUSED, centre=1))(xd, wd)
    fwd = B.Forward(km, 32, 32, td, B.Options.make(gather=B.GATHER_BUFFER))
    for _ in range(2):
        assert torch.equal(fwd(xd, wd), y_fused)
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm)
    assert rel_err(to_f64(y_fused), ref) <= TOL["f16"]


@pytest.mark.parametrize("K,dtype,c_in,c_out,pd,epi", [
    (3, "f16", 32, 32, 0, False),
    (3, "f16", 48, 64, 0, True),     # padding inside the second k-step; residual + ReLU
    (5, "f16", 64, 64, 0, False),    # 125 offsets: several table batches per row
    (1, "f16", 64, 32, 0, True),     # K = 1: the whole layer is the centre
    (3, "bf16", 64, 96, 0, True),
    (3, "bf16", 128, 128, 1, False), # float32 partials
    (3, "f16", 256, 256, 1, True),   # W^T staged from the transposed copy, float32 partials
    (3, "f16", 96, 192, 0, False),   # six column-tile pairs, c_in rounded up to four k-steps
])
def test_centre_offset_in_scatter(K, dtype, c_in, c_out, pd, epi):
    """The submanifold centre offset multiplied inside the scatter (the GEMM skips it):
    within tolerance of the oracle, with and without the residual + ReLU epilogue, and
    close to the path that sends the centre through the GEMM (the sums differ only in
    rounding: the centre's product is never rounded to the partial type)."""
    say(f"centre in scatter K={K} {dtype} {c_in}->{c_out} partials {pd} epilogue {epi}")
    c = _cloud(500 + K, 5000, -10, 10)
    x = scenes.features(len(c), c_in, dtype, 501)
    w = scenes.weights(K, c_in, c_out, dtype, 502)
    km = B.KernelMap.build(to_dev(c), K)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    td = B.TORCH_DTYPES[dtype]
    on = B.Options.make(partial_dtype=pd, centre=2)
    off = B.Options.make(partial_dtype=pd, centre=1)
    pi_on, pi_off = km.plan(c_in, c_out, td, on), km.plan(c_in, c_out, td, off)
    assert pi_on.centre == 1 and pi_off.centre == 0
    assert pi_off.rows_real - pi_on.rows_real == len(c)  # the GEMM skips the centre's rows
    assert km.plan(c_in, c_out, td).centre == 1          # the default
    res = to_dev(scenes.features(len(c), c_out, dtype, 503), dtype) if epi else None
    y_on = B.Forward(km, c_in, c_out, td, on)(xd, wd, residual=res, relu=epi)
    y_off = B.Forward(km, c_in, c_out, td, off)(xd, wd, residual=res, relu=epi)
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, dtype), scenes.to_f64(w, dtype), okm)
    if epi:
        ref = np.maximum(ref + to_f64(res), 0.0)
    e_on, e_off = rel_err(to_f64(y_on), ref), rel_err(to_f64(y_off), ref)
    print(f"normwise error: centre in scatter {e_on:.2e}, through the GEMM {e_off:.2e} "
          f"(element-wise {elem_err(to_f64(y_on), ref):.2e})", flush=True)
    assert e_on <= TOL[dtype] and e_off <= TOL[dtype]
    assert rel_err(to_f64(y_on), to_f64(y_off)) <= TOL[dtype]
    # deterministic: the same call twice gives the same bits
    assert torch.equal(B.Forward(km, c_in, c_out, td, on)(xd, wd, residual=res, relu=epi), y_on)


def test_centre_in_scatter_unsupported_cases():
    """centre = 2 demands the fused centre and fails cleanly where it does not apply;
    centre = 0 falls back to the GEMM path there."""
    say("centre in scatter: unsupported cases")
    c = _cloud(520, 2000, -8, 8)
    km = B.KernelMap.build(to_dev(c), 3)
    kd = B.KernelMap.build(to_dev(c), 2, 2, 1, "down")
    k2 = B.KernelMap.build(to_dev(c), 2)  # even K: no centre offset
    f16 = torch.float16
    req = B.Options.make(centre=2)
    for m, ci, co, td, opt in ((kd, 32, 32, f16, req), (k2, 32, 32, f16, req),
                              (km, 32, 32, torch.float32, req),
                              (km, 32, 16, f16, req), (km, 512, 32, f16, req), (km, 32, 512, f16, req),
                              (km, 32, 32, f16, B.Options.make(centre=2, gather=B.GATHER_BUFFER))):
        with pytest.raises(B.SpconvError) as ei:
            m.plan(ci, co, td, opt)
        assert ei.value.status == B.SPCONV_EUNSUPPORTED
        dflt = B.Options.make(gather=opt.gather)
        assert m.plan(ci, co, td, dflt).centre == 0
    with pytest.raises(B.SpconvError) as ei:
        km.plan(32, 32, f16, B.Options.make(centre=3))
    assert ei.value.status == B.SPCONV_EINVAL


@pytest.mark.parametrize("c_in", [16, 48])
def test_padding_lanes_feed_exact_zeros(c_in):
    """When c_in does not fill the 32-deep MFMA k-steps, the padding lanes read a
    dummy row (input row 0) and must still feed zeros: with an infinity in row 0,
    only the outputs that row 0 really reaches may be non-finite."""
    say(f"k padding with a non-finite dummy row, c_in={c_in}")
    c = _cloud(78, 3000, -9, 9)
    x = scenes.features(len(c), c_in, "f16", 23)
    x[0, :] = np.inf
    w = scenes.weights(3, c_in, 32, "f16", 24)
    km = B.KernelMap.build(to_dev(c), 3)
    xd, wd = to_dev(x, "f16"), to_dev(w, "f16")
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    reached = np.zeros(len(c), dtype=bool)
    reached[okm.pout[okm.pin == 0]] = True
    assert 0 < reached.sum() < len(c)
    keep = ~reached
    xf = scenes.to_f64(x, "f16")
    xf[0, :] = 0.0  # row 0 does not reach the kept rows
    ref = oracle.features(xf, scenes.to_f64(w, "f16"), okm)[keep]
    for g in (B.GATHER_BUFFER, B.GATHER_FUSED):
        y = B.Forward(km, c_in, 32, torch.float16, B.Options.make(gather=g))(xd, wd)
        got = to_f64(y)[keep]
        assert np.isfinite(got).all(), f"gather form {g}: padding lanes leaked the dummy row"
        assert rel_err(got, ref) <= TOL["f16"]


def test_large_cloud_scanned_sort_many_tiles():
    """2.4M voxels: 1172 radix tiles of 2048 keys, below the one-kernel passes (from
    4.2M keys), so each pass scans the digit-major histograms on the device; also
    the DOWN map's output sort.  K = 2 keeps the oracle's map fast."""
    say("large uniform cloud, 2.4M voxels")
    c = scenes.uniform_cells(2_400_000, 400, 4242)
    km = B.KernelMap.build(to_dev(c), 2)
    okm = oracle.kernel_map(c, None, 2, 1, "subm")
    assert_map_equal(km, okm)
    qd = B.KernelMap.build(to_dev(c), 2, 2, 1, "down")
    q = oracle.out_coords(c, 2, 1)
    assert np.array_equal(qd.out_coords().cpu().numpy(), q)


def test_large_query_table_streamed():
    """2.6M voxels at K = 3: the per-(offset, query) table holds 281 MB, past the
    size from which the count pass writes it with non-temporal stores."""
    say("large uniform cloud, 2.6M voxels, K=3")
    c = scenes.uniform_cells(2_600_000, 400, 4250)
    km = B.KernelMap.build(to_dev(c), 3)
    assert_map_equal(km, oracle.kernel_map(c, None, 3, 1, "subm"))


def test_larger_cloud_one_kernel_sort_passes_with_larger_tiles():
    """4.5M voxels: past 1024 tiles of 4096 keys, so the sort runs one kernel per
    pass (tile ranks + look-back) with 16 keys per thread; K = 2 keeps the oracle's
    map fast."""
    say("large uniform cloud, 4.5M voxels")
    c = scenes.uniform_cells_large(4_500_000, 480, 4343)
    km = B.KernelMap.build(to_dev(c), 2)
    okm = oracle.kernel_map(c, None, 2, 1, "subm")
    assert_map_equal(km, okm)


def test_mid_cloud_summed_sort_offsets():
    """0.7M voxels: 342 radix tiles of 2048 keys, whose offsets every scatter
    workgroup sums from the tile histograms itself (more than the 256 tiles of the
    1024-key sorts)."""
    say("mid-size uniform cloud, 0.7M voxels")
    c = scenes.uniform_cells(700_000, 400, 4341)
    km = B.KernelMap.build(to_dev(c), 3)
    assert_map_equal(km, oracle.kernel_map(c, None, 3, 1, "subm"))


def test_mid_cloud_scanned_sort_offsets():
    """1.3M voxels: 635 radix tiles, between the per-workgroup offset sums and the
    one-kernel passes, so each pass scans the digit-major histograms on the device.
    Also about 65k forward-search work items; features checked on sampled rows."""
    say("mid-size uniform cloud, 1.3M voxels")
    c = scenes.uniform_cells(1_300_000, 400, 4343)
    x = scenes.features(len(c), 16, "f16", 4344)
    w = scenes.weights(3, 16, 16, "f16", 4345)
    km, y = _conv_gpu(c, x, w, 3, dtype="f16")
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    assert_map_equal(km, okm)
    rows = np.sort(np.random.default_rng(4346).choice(len(c), 4000, replace=False))
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm, rows=rows)
    assert rel_err(to_f64(y)[rows], ref) <= TOL["f16"]


@pytest.mark.parametrize("side", [123, 194])
def test_sort_with_one_shared_low_digit(side):
    """Every key shares its lowest radix digit: z takes multiples of 256, so the
    first pass puts each whole tile in one bin (the largest 16-bit tile and group
    counts the fused small sorts can meet), and the next pass splits on z's high
    bits.  side 123: ~121k voxels, 1024-key tiles; side 194: ~301k voxels,
    2048-key tiles."""
    say(f"shared low digit, {side}x{side}x8 lattice")
    g = np.stack(np.meshgrid(np.arange(side), np.arange(side), np.arange(8) * 256, indexing="ij"), -1).reshape(-1, 3)
    c = np.concatenate([np.zeros((len(g), 1), np.int64), g], 1).astype(np.int32)
    c = c[np.random.default_rng(side).permutation(len(c))]
    x = scenes.features(len(c), 16, "f16", side + 1)
    w = scenes.weights(3, 16, 16, "f16", side + 2)
    km, y = _conv_gpu(c, x, w, 3, dtype="f16")
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    assert_map_equal(km, okm)
    rows = np.sort(np.random.default_rng(side + 3).choice(len(c), 2000, replace=False))
    ref = oracle.features(scenes.to_f64(x, "f16"), scenes.to_f64(w, "f16"), okm, rows=rows)
    assert rel_err(to_f64(y)[rows], ref) <= TOL["f16"]


def test_sort_bucket_over_capacity_redone_digit_by_digit():
    """A dense 128 x 128 plane at x = 0 plus one point at x = 1000: x takes the key's
    top bits, so all 16384 plane points share the top digit and fall in one bucket,
    twice what one workgroup sorts.  The first build raises the bucket flag and is
    redone digit by digit; the second uses the plan kept for this input.  Both maps
    must equal the oracle's."""
    say("bucket over capacity, 16385 voxels")
    g = np.stack(np.meshgrid(np.arange(128), np.arange(128), indexing="ij"), -1).reshape(-1, 2)
    plane = np.concatenate([np.zeros((len(g), 2), np.int64), g], 1)
    c = np.concatenate([plane, [[0, 1000, 0, 0]]]).astype(np.int32)
    c = c[np.random.default_rng(77).permutation(len(c))]
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    dc = to_dev(c)
    for _ in range(2):
        assert_map_equal(B.KernelMap.build(dc, 3), okm)


@pytest.mark.parametrize("m", [1000, 1024, 1025, 2049, 8191, 8192])
def test_sort_one_bucket_of_m_keys(m):
    """The first m points of a 128 x 128 plane at x = 0 plus one point at x = 1000:
    the plane fills one bucket of exactly m keys, the far point a bucket of one.
    The sizes sit at the bucket sort's boundaries: one item per lane up to 1024
    keys, two from 1025, three from 2049, and 8192, the most one workgroup sorts
    without a redo.  The map must equal the oracle's."""
    say(f"one bucket of {m} keys")
    g = np.stack(np.meshgrid(np.arange(128), np.arange(128), indexing="ij"), -1).reshape(-1, 2)[:m]
    plane = np.concatenate([np.zeros((m, 2), np.int64), g], 1)
    c = np.concatenate([plane, [[0, 1000, 0, 0]]]).astype(np.int32)
    c = c[np.random.default_rng(m).permutation(len(c))]
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    assert_map_equal(B.KernelMap.build(to_dev(c), 3), okm)


@pytest.mark.parametrize("seed", range(12))
def test_random_clouds_maps_match_oracle(seed):
    """Seeded sweep of random clouds: 1 to 60k voxels in 1 to 4 batches, cubes of
    side 4 to 119 placed anywhere in [-600, 720), K in {2, 3, 5}.  The sizes keep the
    by-bucket sort, so bucket sizes, empty and lone-key buckets and digit
    collisions in the ranking vary from case to case.  Maps must equal the
    oracle's."""
    rng = np.random.default_rng(9000 + seed)
    K = int(rng.choice([2, 3, 5]))
    nb = int(rng.integers(1, 5))
    side = int(rng.integers(4, 120))
    lo = int(rng.integers(-600, 600))
    n = int(min(rng.integers(1, 60000), nb * side ** 3))
    say(f"random cloud seed={seed}: n={n} batches={nb} side={side} lo={lo} K={K}")
    c = _cloud(9100 + seed, n, lo, lo + side, nb=nb)
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    assert_map_equal(B.KernelMap.build(to_dev(c), K), okm)


def test_deterministic_pairs():
    say("deterministic pair order")
    c = scenes.workload(1).coords
    dc = to_dev(c)
    a = gpu_pairs(B.KernelMap.build(dc, 3))
    b = gpu_pairs(B.KernelMap.build(dc, 3))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]


def test_bf16_layer():
    say("bf16 layer")
    c = _cloud(40, 5000, -12, 12)
    x = scenes.features(len(c), 32, "bf16", 13)
    w = scenes.weights(3, 32, 48, "bf16", 14)
    km, y = _conv_gpu(c, x, w, 3, dtype="bf16")
    okm = oracle.kernel_map(c, None, 3, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, "bf16"), scenes.to_f64(w, "bf16"), okm)
    assert rel_err(to_f64(y), ref) <= TOL["bf16"]


@pytest.mark.parametrize("K,c", [(5, 64), (3, 256)])
def test_bf16_partial_precision(K, c):
    """bf16 layers sum per-offset GEMM partials in float32, the partials themselves
    stored in bf16 (the default) or float32.  With float32 partials the only error
    left is the output's rounding to bf16, at most 2^-8 of max|y| normwise (8
    significant bits); the default adds one bf16 rounding per offset and must meet
    the tolerance.  Both errors are printed."""
    say(f"bf16 partial precision K={K} C={c}")
    cl = _cloud(41 + K, 6000, -12, 12)
    x = scenes.features(len(cl), c, "bf16", 15)
    w = scenes.weights(K, c, c, "bf16", 16)
    okm = oracle.kernel_map(cl, None, K, 1, "subm")
    ref = oracle.features(scenes.to_f64(x, "bf16"), scenes.to_f64(w, "bf16"), okm)
    km = B.KernelMap.build(to_dev(cl), K)
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    y32 = B.Forward(km, c, c, torch.bfloat16, B.Options.make(partial_dtype=1))(xd, wd)
    y16 = B.Forward(km, c, c, torch.bfloat16)(xd, wd)
    torch.cuda.synchronize()
    assert_map_equal(km, okm)
    e32, e16 = rel_err(to_f64(y32), ref), rel_err(to_f64(y16), ref)
    print(f"bf16 K={K} C={c}: normwise error with float32 partials {e32:.2e}, with bf16 partials {e16:.2e}",
          flush=True)
    assert e32 <= 2.0 ** -8 * 1.01
    assert e16 <= TOL["bf16"]


def test_f32_widest_input():
    """f32 at the widest input the boundary takes (1024 channels): the general
    GEMM holds one 16-column tile of W_k^T (65.8 KB) in LDS."""
    say("f32 c_in = 1024")
    cl = _cloud(44, 1500, -7, 7)
    x = scenes.features(len(cl), 1024, "f32", 17)
    w = scenes.weights(3, 1024, 16, "f32", 18)
    km, y = _conv_gpu(cl, x, w, 3)
    okm = oracle.kernel_map(cl, None, 3, 1, "subm")
    assert rel_err(to_f64(y), oracle.features(x, w, okm)) <= TOL["f32"]


# ----------------------------------------------------------------------------
# Edge cases and error paths
# ----------------------------------------------------------------------------

def test_empty_and_single():
    say("empty and single-voxel inputs")
    e = torch.zeros((0, 4), dtype=torch.int32, device=DEV)
    km = B.KernelMap.build(e, 3)
    assert km.n_out == 0 and sum(km.counts()) == 0
    kd = B.KernelMap.build(e, 2, 2, 1, "down")
    assert kd.n_out == 0
    one = np.array([[3, -5, 7, 11]], np.int32)
    x = np.ones((1, 4), np.float32)
    w = scenes.weights(3, 4, 16, "f32", 1)
    km1, y = _conv_gpu(one, x, w, 3)
    cnt = km1.counts()
    assert sum(cnt) == 1 and cnt[13] == 1
    assert np.allclose(to_f64(y)[0], w[13].sum(0), rtol=1e-6)


def test_isolated_rows_get_zeros():
    say("rows without pairs")
    c = np.array([[0, 0, 0, 0], [0, 10, 10, 10]], np.int32)
    x = np.ones((2, 4), np.float32)
    w = scenes.weights(3, 4, 16, "f32", 1)
    w[13] = 0  # centre weight zero: both rows have only the centre pair
    km, y = _conv_gpu(c, x, w, 3)
    assert float(y.abs().max()) == 0.0


def test_error_duplicates_and_range():
    say("duplicate / out-of-range coordinates")
    dup = to_dev(np.array([[0, 1, 2, 3], [0, 5, 5, 5], [0, 1, 2, 3]], np.int32))
    with pytest.raises(B.SpconvError) as ei:
        B.KernelMap.build(dup, 3)
    assert ei.value.status == B.SPCONV_EDUP
    big = to_dev(np.array([[0, -2**31, 0, -2**31], [0, 2**31 - 1, 2**31 - 1, 2**31 - 1]], np.int32))
    with pytest.raises(B.SpconvError) as ei:
        B.KernelMap.build(big, 3)
    assert ei.value.status == B.SPCONV_ERANGE


# ----------------------------------------------------------------------------
# Hash-table search (the prior-art Map, an ablation of the sorted-array search)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("K", [1, 2, 3, 5])
def test_hash_search_subm_small(K):
    say(f"hash-table search K={K}")
    c = _cloud(70 + K, 4000, -10, 10)
    x = scenes.features(len(c), 16, "f32", 71)
    w = scenes.weights(K, 16, 16, "f32", 72)
    km, y = _conv_gpu(c, x, w, K, opt=B.Options.make(search=1, Cq=256))
    okm = oracle.kernel_map(c, None, K, 1, "subm")
    assert_map_equal(km, okm)
    assert rel_err(to_f64(y), oracle.features(x, w, okm)) <= TOL["f32"]


def test_hash_search_lidar_matches_sorted_search():
    say("hash-table search on the 120k LiDAR layer")
    wl = scenes.workload(1)
    L = wl.layers[0]
    x = scenes.features(len(wl.coords), L.c_in, L.dtype, 2001)
    w = scenes.weights(L.K, L.c_in, L.c_out, L.dtype, 3001)
    kh, yh = _conv_gpu(wl.coords, x, w, L.K, dtype=L.dtype, opt=B.Options.make(search=1))
    ks, ys = _conv_gpu(wl.coords, x, w, L.K, dtype=L.dtype)
    assert_map_equal(kh, oracle.kernel_map(wl.coords, None, L.K, 1, "subm"))
    assert list(kh.counts()) == list(ks.counts())
    # same pairs, summed in the same offset order: the outputs agree exactly
    assert torch.equal(yh, ys)


def test_hash_search_errors():
    say("hash-table search errors")
    dup = to_dev(np.array([[0, 1, 2, 3], [0, 5, 5, 5], [0, 1, 2, 3]], np.int32))
    with pytest.raises(B.SpconvError) as ei:
        B.KernelMap.build(dup, 3, opt=B.Options.make(search=1))
    assert ei.value.status == B.SPCONV_EDUP
    c = to_dev(_cloud(73, 200, -4, 4))
    with pytest.raises(B.SpconvError) as ei:
        B.KernelMap.build(c, 2, 2, 1, "down", opt=B.Options.make(search=1))
    assert ei.value.status == B.SPCONV_EUNSUPPORTED


def test_error_forward_args():
    say("forward argument errors")
    c = _cloud(50, 100, -3, 3)
    km = B.KernelMap.build(to_dev(c), 3)
    with pytest.raises(B.SpconvError) as ei:
        B.Forward(km, 16, 20, torch.float32)  # c_out not a multiple of 16
    assert ei.value.status == B.SPCONV_EUNSUPPORTED
    f = B.Forward(km, 16, 16, torch.float32)
    tiny = torch.empty(1, dtype=torch.uint8, device=DEV)
    with pytest.raises(B.SpconvError) as ei:
        B.spconv_forward(km.handle, torch.zeros(len(c), 16, device=DEV), torch.zeros(27, 16, 16, device=DEV),
                         torch.zeros(len(c), 16, device=DEV), 16, 16, B.SPCONV_F32, None, tiny)
    assert ei.value.status == B.SPCONV_ENOSPC
    _ = f
