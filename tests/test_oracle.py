"""Pins for the CPU oracle (runs without a GPU).

Each test checks the oracle against something other than itself: values the
paper prints (fixtures in tests/golden/), a hand-computed example, dense float64
convolutions by torch on tiny grids, brute-force all-pairs kernel maps, and
invariants the mathematics fixes.
"""
from __future__ import annotations

import itertools
import os

import numpy as np
import pytest

import oracle
from tests import dense_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows.setdefault(key, []).append([int(v) for v in vals])
    return rows


def _cloud(rng, n, lo, hi, nb=1, t=1):
    """n distinct random voxels with x,y,z in [lo, hi) (multiples of t), b in [0, nb)."""
    pts = set()
    while len(pts) < n:
        b = int(rng.integers(0, nb))
        p = tuple(int(v) * t for v in rng.integers(lo, hi, 3))
        pts.add((b,) + p)
    c = np.array(sorted(pts), dtype=np.int32)
    return np.ascontiguousarray(c[rng.permutation(len(c))])


# ----------------------------------------------------------------------------
# Offsets (Section 2.1)
# ----------------------------------------------------------------------------

def test_offsets_match_paper_delta_5_2():
    g = _golden("paper_offsets.txt")
    K, t = g["K"][0][0], g["t"][0][0]
    d = oracle.offsets(K, t)
    axis = g["axis_values"][0]
    assert set(map(tuple, d.tolist())) == set(itertools.product(axis, axis, axis))
    assert tuple(d[0]) == tuple(g["first"][0])


@pytest.mark.parametrize("K", [1, 3, 5, 7])
def test_offsets_odd_symmetry_and_centre(K):
    d = oracle.offsets(K, 1)
    k3 = K ** 3
    assert d.shape == (k3, 3)
    # centre offset sits in the middle of the enumeration; opposite offsets pair up
    assert tuple(d[(k3 - 1) // 2]) == (0, 0, 0)
    assert np.array_equal(d[::-1], -d)
    assert len(set(map(tuple, d.tolist()))) == k3


@pytest.mark.parametrize("K,t", [(2, 1), (2, 4), (4, 2)])
def test_offsets_even(K, t):
    d = oracle.offsets(K, t)
    assert set(map(tuple, d.tolist())) == set(itertools.product(range(0, K * t, t), repeat=3))
    assert tuple(d[0]) == (0, 0, 0)
    # x-major enumeration: k = ix K^2 + iy K + iz
    assert tuple(d[1]) == (0, 0, t) and tuple(d[K]) == (0, t, 0) and tuple(d[K * K]) == (t, 0, 0)


# ----------------------------------------------------------------------------
# Output coordinates (Eq. 1)
# ----------------------------------------------------------------------------

def test_out_coords_hand_cases():
    assert oracle.out_coords(np.array([[0, -1, 0, 0]]), 2).tolist() == [[0, -2, 0, 0]]
    assert oracle.out_coords(np.array([[0, 0, 0, 0], [0, 1, 0, 0]]), 2).tolist() == [[0, 0, 0, 0]]
    assert oracle.out_coords(np.array([[3, -3, 5, -8]]), 4).tolist() == [[3, -4, 4, -8]]
    # spacing t multiplies the cell: t = 2, s = 2 -> cells of 4
    assert oracle.out_coords(np.array([[0, 6, -2, 2]]), 2, 2).tolist() == [[0, 4, -4, 0]]


def test_out_coords_sorted_like_paper_examples():
    g = _golden("paper_search_order.txt")
    srt = np.array(g["sorted"], dtype=np.int32)
    coords = np.concatenate([np.zeros((len(srt), 1), np.int32), srt], axis=1)
    shuffled = coords[np.random.default_rng(0).permutation(len(coords))]
    out = oracle.out_coords(shuffled, 1)
    assert np.array_equal(out[:, 1:], srt)
    seg = _golden("paper_segment.txt")
    q = np.concatenate([np.zeros((4, 1), np.int32), np.array(seg["q"], np.int32)], axis=1)
    assert np.array_equal(oracle.out_coords(q[::-1].copy(), 1), q)


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("s,t", [(1, 1), (2, 1), (2, 2), (3, 1)])
def test_out_coords_cell_property(seed, s, t):
    rng = np.random.default_rng(seed)
    c = _cloud(rng, 60, -7, 7, nb=2, t=t)
    q = oracle.out_coords(c, s, t)
    g = s * t
    # outputs are distinct, sorted, and multiples of the cell size
    assert len({tuple(r) for r in q.tolist()}) == len(q)
    assert [tuple(r) for r in q.tolist()] == sorted(tuple(r) for r in q.tolist())
    assert np.all(q[:, 1:] % g == 0)
    qs = {tuple(r) for r in q.tolist()}
    # every input lies in exactly one output cell [q, q + g)^3 of its batch, and every cell is used
    used = set()
    for p in c.tolist():
        owners = [r for r in qs if r[0] == p[0] and all(r[a] <= p[a] < r[a] + g for a in (1, 2, 3))]
        assert len(owners) == 1
        used.add(owners[0])
    assert used == qs


# ----------------------------------------------------------------------------
# Kernel map (Eq. 3): brute force, invariants, paper examples
# ----------------------------------------------------------------------------

def _brute_map(in_c, out_c, K, t, mode):
    """All-pairs enumeration of p_j == q_i + delta_k (transposed: q_i == p_j + delta_k)."""
    c = (K - 1) // 2 if K % 2 == 1 else 0
    sets = []
    for ix in range(K):
        for iy in range(K):
            for iz in range(K):
                d = (t * (ix - c), t * (iy - c), t * (iz - c))
                s = set()
                for i, q in enumerate(out_c.tolist()):
                    for j, p in enumerate(in_c.tolist()):
                        if p[0] != q[0]:
                            continue
                        if mode == "up":
                            hit = all(q[a + 1] == p[a + 1] + d[a] for a in range(3))
                        else:
                            hit = all(p[a + 1] == q[a + 1] + d[a] for a in range(3))
                        if hit:
                            s.add((j, i))
                sets.append(s)
    return sets


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("K", [1, 2, 3, 5])
def test_kernel_map_subm_brute_force(seed, K):
    rng = np.random.default_rng(100 + seed)
    c = _cloud(rng, 40, -3, 4, nb=2)
    km = oracle.kernel_map(c, None, K, 1, "subm")
    assert km.as_sets() == _brute_map(c, c, K, 1, "subm")
    # each list is in ascending output row
    for k in range(km.K3):
        assert np.all(np.diff(km.pairs(k)[1]) > 0)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("K,s,t", [(2, 2, 1), (3, 2, 1), (2, 2, 2), (2, 3, 1)])
def test_kernel_map_down_up_brute_force(seed, K, s, t):
    rng = np.random.default_rng(200 + seed)
    c = _cloud(rng, 40, -4, 4, nb=2, t=t)
    q = oracle.out_coords(c, s, t)
    km = oracle.kernel_map(c, q, K, t, "down")
    assert km.as_sets() == _brute_map(c, q, K, t, "down")
    up = oracle.kernel_map(q, c, K, t, "up")
    assert up.as_sets() == _brute_map(q, c, K, t, "up")


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("K", [3, 5])
def test_kernel_map_subm_invariants(seed, K):
    rng = np.random.default_rng(300 + seed)
    c = _cloud(rng, 200, -5, 5, nb=2)
    km = oracle.kernel_map(c, None, K, 1, "subm")
    k3 = K ** 3
    centre = (k3 - 1) // 2
    pin, pout = km.pairs(centre)
    assert np.array_equal(pin, np.arange(len(c))) and np.array_equal(pout, np.arange(len(c)))
    sets = km.as_sets()
    for k in range(k3):
        assert sets[k3 - 1 - k] == {(i, j) for (j, i) in sets[k]}
    assert km.counts.sum() <= k3 * len(c)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("t", [1, 2, 8])
def test_kernel_map_down_partition_and_up_swap(seed, t):
    rng = np.random.default_rng(400 + seed)
    c = _cloud(rng, 300, -6, 6, nb=2, t=t)
    q = oracle.out_coords(c, 2, t)
    km = oracle.kernel_map(c, q, 2, t, "down")
    # K = s = 2: every input appears exactly once over all offsets
    assert km.counts.sum() == len(c)
    assert np.array_equal(np.sort(km.pin), np.arange(len(c)))
    up = oracle.kernel_map(q, c, 2, t, "up")
    assert np.array_equal(up.counts, km.counts)
    assert up.as_sets() == [{(i, j) for (j, i) in s} for s in km.as_sets()]
    assert np.array_equal(np.sort(up.pout), np.arange(len(c)))


def test_kernel_map_paper_segment_example():
    g = _golden("paper_segment.txt")
    q = np.concatenate([np.zeros((4, 1), np.int32), np.array(g["q"], np.int32)], axis=1)
    seg = np.concatenate([np.zeros((4, 1), np.int32), np.array(g["seg"], np.int32)], axis=1)
    # inputs are exactly the segment's queries -> every query of that offset hits, in order
    K = 3
    d = tuple(g["delta"][0])
    k = [tuple(r) for r in oracle.offsets(K, 1).tolist()].index(d)
    km = oracle.kernel_map(seg, q, K, 1, "down")
    pin, pout = km.pairs(k)
    assert pout.tolist() == [0, 1, 2, 3] and pin.tolist() == [0, 1, 2, 3]


def test_hand_two_voxel_example():
    g = _golden("hand_two_voxel.txt")
    p = np.array([[0, 0, 0, 0], [0, 1, 0, 0]], np.int32)
    x = np.array([[1.0], [2.0]])
    w3 = (np.arange(27, dtype=np.float64) + 1).reshape(27, 1, 1)
    oc, km, y = oracle.conv(p, x, w3, 3, 1, 1, "subm")
    assert y[:, 0].tolist() == g["subm_y"][0]
    want = [set() for _ in range(27)]
    for k, j, i in g["subm_pairs"]:
        want[k].add((j, i))
    assert km.as_sets() == want
    w2 = (np.arange(8, dtype=np.float64) + 1).reshape(8, 1, 1)
    q, kmd, yd = oracle.conv(p, x, w2, 2, 2, 1, "down")
    assert q.tolist() == g["down_q"]
    assert yd[:, 0].tolist() == g["down_y"][0]
    want = [set() for _ in range(8)]
    for k, j, i in g["down_pairs"]:
        want[k].add((j, i))
    assert kmd.as_sets() == want
    _, _, yu = oracle.conv(q, np.array([[3.0]]), w2, 2, 2, 1, "up", out_coords_=p)
    assert yu[:, 0].tolist() == g["up_y"][0]


def test_errors():
    dup = np.array([[0, 1, 2, 3], [0, 1, 2, 3]], np.int32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.kernel_map(dup, None, 3, 1, "subm")
    assert e.value.status == -3
    with pytest.raises(oracle.OracleError):
        oracle.offsets(0, 1)
    with pytest.raises(oracle.OracleError):
        oracle.out_coords(dup, 0)
    empty = np.zeros((0, 4), np.int32)
    km = oracle.kernel_map(empty, None, 3, 1, "subm")
    assert km.counts.sum() == 0


# ----------------------------------------------------------------------------
# Features (Eq. 2) against dense float64 convolutions
# ----------------------------------------------------------------------------

def _rel_err(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("K,t", [(1, 1), (2, 1), (3, 1), (3, 2), (5, 1)])
def test_features_subm_vs_dense(seed, K, t):
    rng = np.random.default_rng(500 + seed)
    c = _cloud(rng, 150, 0, 8, nb=2, t=t)
    cin, cout = 3, 5
    x = rng.standard_normal((len(c), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    _, _, y = oracle.conv(c, x, w, K, 1, t, "subm")
    ref = dense_ref.subm(c, x, w, K, t)
    assert _rel_err(y, ref) < 1e-12


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("K,s,t", [(2, 2, 1), (2, 2, 2), (3, 2, 1), (2, 3, 1)])
def test_features_down_up_vs_dense(seed, K, s, t):
    rng = np.random.default_rng(600 + seed)
    # negative coordinates: the oracle runs on the cloud, the dense reference on the
    # cloud shifted by a multiple of the cell size (floor then commutes with the shift)
    shift = 4 * s * t
    c = _cloud(rng, 150, -4, 4, nb=2, t=t)
    cs = c.copy()
    cs[:, 1:] += shift
    cin, cout = 3, 4
    x = rng.standard_normal((len(c), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    q, _, y = oracle.conv(c, x, w, K, s, t, "down")
    qs = q.copy()
    qs[:, 1:] += shift
    assert np.array_equal(qs, oracle.out_coords(cs, s, t))
    ref = dense_ref.down(cs, x, w, K, s, t, qs)
    assert _rel_err(y, ref) < 1e-12
    if K == s:  # transposed conv from the coarse sites back to the fine ones
        xc = rng.standard_normal((len(q), cout))
        wu = rng.standard_normal((K ** 3, cout, cin))
        _, _, yu = oracle.conv(q, xc, wu, K, s, t, "up", out_coords_=c)
        refu = dense_ref.up(qs, xc, wu, K, s, t, cs)
        assert _rel_err(yu, refu) < 1e-12


def test_features_rows_and_threads_deterministic():
    rng = np.random.default_rng(7)
    c = _cloud(rng, 400, -6, 6, nb=2)
    x = rng.standard_normal((len(c), 8))
    w = rng.standard_normal((27, 8, 6))
    km = oracle.kernel_map(c, None, 3, 1, "subm")
    y1 = oracle.features(x, w, km, nthreads=1)
    y8 = oracle.features(x, w, km, nthreads=8)
    assert np.array_equal(y1, y8)
    rows = rng.choice(len(c), 50, replace=False)
    assert np.array_equal(oracle.features(x, w, km, rows=rows), y1[rows])
