"""Pins of the oracle's alternative pre-encoder signals (Table 5's low-res
frame difference and dHash, in the readings stated in the oracle: luma box
means on a G x G grid, rounded half up, L1 over 255 G^2; dHash bits of an
8 x 9 grid of box means, Hamming over 64).  Checked against closed forms
(solid frames, exact half-way means, uneven cells, ramps and step edges), an
independent numpy formulation on random frames, the metric axioms, and the
keep rule on a static video."""
import numpy as np
import pytest

import oracle


def luma(frames):
    """BT.601 integer luma (C = 3) or the value (C = 1), as int64."""
    f = frames.astype(np.int64)
    if f.shape[-1] == 1:
        return f[..., 0]
    return (299 * f[..., 0] + 587 * f[..., 1] + 114 * f[..., 2] + 500) // 1000


def np_cell_means(frames, gh, gw):
    """Second formulation: per-pixel cell index arrays and np.add.at."""
    n, H, W = frames.shape[:3]
    y = luma(frames)
    cy = (np.arange(H) * gh) // H
    cx = (np.arange(W) * gw) // W
    cell = (cy[:, None] * gw + cx[None, :]).ravel()
    out = np.zeros((n, gh * gw), np.int64)
    area = np.bincount(cell, minlength=gh * gw).astype(np.int64)
    for t in range(n):
        s = np.zeros(gh * gw, np.int64)
        np.add.at(s, cell, y[t].ravel())
        out[t] = (s + area // 2) // area
    return out


def np_dhash(frames):
    m = np_cell_means(frames, 8, 9).reshape(-1, 8, 9)
    return (m[:, :, 1:] > m[:, :, :-1]).reshape(-1, 64).astype(np.uint32)


def dist(rows, i, j, two_m):
    return oracle.l1(rows[i], rows[j]) / two_m


def test_solid_frames_closed_form():
    """Grey solid frames v1, v2: every cell mean is v, D = G^2 |v1 - v2|,
    distance |v1 - v2| / 255 (exactly, in any grid)."""
    vals = [0, 17, 128, 255]
    f = np.stack([np.full((24, 40, 3), v, np.uint8) for v in vals])
    for G in (2, 4, 8):
        rows = oracle.signature(f, oracle.FRAMEDIFF, G)
        assert rows.shape == (4, G * G)
        for t, v in enumerate(vals):
            assert np.all(rows[t] == v)
        two_m = oracle.signal_two_m(oracle.FRAMEDIFF, G)
        assert two_m == 255 * G * G
        for i in range(4):
            for j in range(4):
                assert oracle.l1(rows[i], rows[j]) == G * G * abs(vals[i] - vals[j])
    # primaries through the BT.601 luma: (76, 150, 29) for R, G, B at 255
    prim = np.zeros((3, 8, 8, 3), np.uint8)
    for c in range(3):
        prim[c, ..., c] = 255
    rows = oracle.signature(prim, oracle.FRAMEDIFF, 2)
    assert rows[:, 0].tolist() == [76, 150, 29]


def test_cell_mean_rounds_half_up():
    """4 x 4 grey frames on a 2 x 2 grid: cell (0, 0) holds the 2 x 2 block;
    its mean 1/4, 1/2, 3/4, 5/4, 3/2 rounds to 0, 1, 1, 1, 2."""
    cases = [([0, 0, 0, 1], 0), ([0, 0, 1, 1], 1), ([0, 1, 1, 1], 1), ([1, 1, 1, 2], 1), ([1, 1, 2, 2], 2)]
    f = np.zeros((len(cases), 4, 4, 1), np.uint8)
    for t, (block, _) in enumerate(cases):
        f[t, 0:2, 0:2, 0] = np.array(block).reshape(2, 2)
    rows = oracle.signature(f, oracle.FRAMEDIFF, 2)
    assert rows[:, 0].tolist() == [want for _, want in cases]
    assert np.all(rows[:, 1:] == 0)


def test_uneven_cells():
    """H = 5, W = 3 on a 2 x 2 grid: rows 0-2 / 3-4 ((2y) div 5), columns
    0-1 / 2 ((2x) div 3); pixel (y, x) = 10 y + x."""
    f = np.array([[[10 * y + x] for x in range(3)] for y in range(5)], np.uint8)[None]
    rows = oracle.signature(f, oracle.FRAMEDIFF, 2)
    # cell (0,0): y 0-2, x 0-1: values 0,1,10,11,20,21 -> 63/6 = 10.5 -> 11
    # cell (0,1): y 0-2, x 2: 2,12,22 -> 12
    # cell (1,0): y 3-4, x 0-1: 30,31,40,41 -> 35.5 -> 36
    # cell (1,1): y 3-4, x 2: 32,42 -> 37
    assert rows[0].tolist() == [11, 12, 36, 37]


@pytest.mark.parametrize("shape,G", [((5, 33, 47, 3), 4), ((3, 64, 64, 1), 16), ((2, 90, 160, 3), 32),
                                     ((2, 37, 29, 3), 2), ((1, 48, 48, 3), 48)])
def test_framediff_matches_numpy(shape, G):
    rng = np.random.default_rng([2609, 3675, 61, G])
    f = rng.integers(0, 256, size=shape, dtype=np.uint8)
    assert np.array_equal(oracle.signature(f, oracle.FRAMEDIFF, G), np_cell_means(f, G, G))


@pytest.mark.parametrize("shape", [(4, 8, 9, 3), (3, 33, 47, 3), (2, 90, 160, 1), (2, 120, 120, 3)])
def test_dhash_matches_numpy(shape):
    rng = np.random.default_rng([2609, 3675, 62, shape[1]])
    f = rng.integers(0, 256, size=shape, dtype=np.uint8)
    assert np.array_equal(oracle.signature(f, oracle.DHASH), np_dhash(f))


def test_dhash_ramps_and_edges():
    """Brightness rising left to right sets all 64 bits, falling or constant
    sets none; a step at a cell boundary between cell columns 4 and 5 sets
    exactly the 8 bits of that pair; rising vs falling are at distance 1."""
    W, H = 90, 40
    x = np.arange(W)
    up = np.broadcast_to((x * 255 // (W - 1)).astype(np.uint8)[None, :, None], (H, W, 3))
    down = up[:, ::-1]
    flat = np.full((H, W, 3), 100, np.uint8)
    step = np.where(x[None, :, None] >= 50, 200, 20).astype(np.uint8) * np.ones((H, 1, 3), np.uint8)
    rows = oracle.signature(np.stack([up, down, flat, step]), oracle.DHASH)
    assert rows[0].sum() == 64 and rows[1].sum() == 0 and rows[2].sum() == 0
    bits = rows[3].reshape(8, 8)
    assert np.all(bits[:, 4] == 1) and bits.sum() == 8
    assert oracle.signal_two_m(oracle.DHASH) == 64
    assert oracle.l1(rows[0], rows[1]) == 64


@pytest.mark.parametrize("kind,G", [(oracle.FRAMEDIFF, 8), (oracle.DHASH, 0)])
def test_signal_distance_is_a_metric(kind, G):
    rng = np.random.default_rng([2609, 3675, 63, kind])
    f = rng.integers(0, 256, size=(6, 32, 36, 3), dtype=np.uint8)
    rows = oracle.signature(f, kind, G)
    two_m = oracle.signal_two_m(kind, G)
    for i in range(6):
        assert dist(rows, i, i, two_m) == 0
        for j in range(6):
            dij = dist(rows, i, j, two_m)
            assert 0 <= dij <= 1 and dij == dist(rows, j, i, two_m)
            for k in range(6):
                assert dij <= dist(rows, i, k, two_m) + dist(rows, k, j, two_m) + 1e-12


def test_signals_reject_grids_finer_than_the_image():
    f = np.zeros((1, 4, 8, 3), np.uint8)
    with pytest.raises(ValueError):
        oracle.signature(f, oracle.FRAMEDIFF, 8)   # 8 > H = 4
    with pytest.raises(ValueError):
        oracle.signature(f, oracle.DHASH)          # H < 8


@pytest.mark.parametrize("kind,G", [(oracle.FRAMEDIFF, 4), (oracle.DHASH, 0)])
def test_keep_rule_on_a_static_video(kind, G):
    """Identical frames: every distance is 0, so the rule keeps frame 0, the
    gap-rule frames L_max, 2 L_max, ... and the last frame (Eqs. 3-5 with the
    safeguards), for any threshold above 0."""
    T, L = 70, 30
    f = np.full((T, 16, 18, 3), 90, np.uint8)
    rows = oracle.signature(f, kind, G)
    two_m = oracle.signal_two_m(kind, G)
    scores, mask, kept = oracle.ngff_select(rows, two_m // 2, 0.1, L, 4)
    assert np.flatnonzero(mask).tolist() == [0, 30, 60, 69]
    assert np.all(scores[1:] == 0)
