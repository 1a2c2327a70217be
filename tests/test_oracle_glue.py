"""Pins of the oracle's coarse-to-fine glue (candidate compaction of the NGFF
mask, Sec. 3.1-3.2; removal of the frames outside S_e from a token sequence
with the kept frames in chronological order, Sec. 3.3), against hand-built
cases, numpy's own routines and a row-by-row brute force."""
import numpy as np
import pytest

import oracle


def test_mask_compact_worked_example():
    # frames 0..7 in two streams of 4 (and a partial third of 0): kept 1, 2, 4, 7
    mask = np.array([0, 1, 1, 0, 1, 0, 0, 1], np.uint8)
    idx, seg = oracle.mask_compact(mask, 4)
    assert idx.tolist() == [1, 2, 4, 7]
    assert seg.tolist() == [0, 2, 4]
    idx, seg = oracle.mask_compact(mask, 3)   # segments [0,3) [3,6) [6,8)
    assert seg.tolist() == [0, 2, 3, 4]
    idx, seg = oracle.mask_compact(mask, 0)   # one stream
    assert seg.tolist() == [0, 4]


@pytest.mark.parametrize("n,seg_len", [(0, 0), (0, 5), (1, 0), (1, 1), (7, 100), (1000, 1), (1000, 37),
                                       (4096, 512), (5000, 0)])
def test_mask_compact_matches_numpy(n, seg_len):
    rng = np.random.default_rng([2609, 3675, 77, n, seg_len])
    for p in (0.0, 0.3, 1.0):
        mask = (rng.random(n) < p).astype(np.uint8) * rng.integers(1, 256, n).astype(np.uint8)
        idx, seg = oracle.mask_compact(mask, seg_len)
        assert np.array_equal(idx, np.flatnonzero(mask))
        nseg = -(-n // seg_len) if seg_len > 0 else 1
        bounds = [min(s * seg_len, n) for s in range(nseg)] if seg_len > 0 else [0]
        expect = [int(np.count_nonzero(mask[:b])) for b in bounds] + [int(np.count_nonzero(mask))]
        assert seg.tolist() == expect


def brute_gather(src, offs, sel, capacity):
    n_rows = src.shape[0]
    rows, lens = [], []
    for f in sel:
        if 0 <= f < len(offs) - 1:
            lo = min(max(int(offs[f]), 0), n_rows)
            hi = max(lo, min(max(int(offs[f + 1]), 0), n_rows))
            rows += list(range(lo, hi))
            lens.append(hi - lo)
        else:
            lens.append(0)
    out_offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    rows = np.array(rows[:capacity], dtype=np.int64)
    return src[rows] if rows.size else src[:0], out_offs, rows


def test_gather_worked_example():
    # 5 frames of 3 tokens; S_e = {1, 3} keeps tokens 3..5 and 9..11 in order
    src = np.arange(15 * 4, dtype=np.int16).reshape(15, 4)
    offs = np.arange(0, 16, 3, dtype=np.int32)
    dst, out_offs, rows = oracle.gather_frames(src, offs, np.array([1, 3, -1, -1], np.int32))
    assert rows.tolist() == [3, 4, 5, 9, 10, 11]
    assert out_offs.tolist() == [0, 3, 6, 6, 6]
    assert np.array_equal(dst, src[[3, 4, 5, 9, 10, 11]])


@pytest.mark.parametrize("row_shape,dtype", [((7,), np.uint8), ((3, 5), np.uint16), ((28, 128), np.uint16),
                                             ((1,), np.float32)])
def test_gather_matches_brute_force(row_shape, dtype):
    rng = np.random.default_rng([2609, 3675, 78, len(row_shape)])
    n_frames = 40
    sizes = rng.integers(0, 9, n_frames)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    n_rows = int(offs[-1])
    src = rng.integers(0, 60000, (n_rows,) + row_shape).astype(dtype)
    sel = np.sort(rng.choice(n_frames, 12, replace=False)).astype(np.int32)
    sel = np.concatenate([sel, [-1, -1, n_frames, 1 << 30]]).astype(np.int32)
    for cap in (-1, 0, 5, n_rows):
        dst, out_offs, rows = oracle.gather_frames(src, offs, sel, cap)
        c = n_rows if cap < 0 else cap
        bdst, boffs, brows = brute_gather(src, offs, sel, c)
        assert np.array_equal(out_offs, boffs)
        assert np.array_equal(rows, brows)
        assert np.array_equal(dst, bdst)


def test_gather_malformed_offsets_are_clamped():
    src = np.arange(10, dtype=np.uint8).reshape(10, 1)
    offs = np.array([-5, 3, 2, 40, 7], np.int32)   # [0,3) [3,3) [2,10) [10,10)
    dst, out_offs, rows = oracle.gather_frames(src, offs, np.array([0, 1, 2, 3], np.int32))
    assert out_offs.tolist() == [0, 3, 3, 11, 11]
    assert rows.tolist() == [0, 1, 2] + list(range(2, 10))
