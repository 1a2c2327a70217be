"""Pins of the oracle's online reading of the keep rule (Sec. 3.2 applied as
frames of the growing video prefix arrive, Sec. 3.1): a hand-computed stream,
its equality with the one-shot rule once the end-of-stream safeguards are
applied, causality, and the degenerate thresholds."""
import numpy as np
import pytest

import oracle


def two_bin(frames):
    return np.array(frames, dtype=np.uint32)


def test_hand_computed_stream():
    # mass M = 10, 2M = 20: D([10,0],[0,10]) = 20 (s = 1), D([10,0],[5,5]) = 10 (s = 0.5)
    h = two_bin([[10, 0], [10, 0], [0, 10], [0, 10], [5, 5]])
    s, m, r = oracle.ngff_scan_open(h, 10, 0.6, 30)
    assert m.tolist() == [1, 0, 1, 0, 0] and r == 2
    assert s.tolist() == [1.0, 0.0, 1.0, 0.0, 0.5]
    final, added = oracle.ngff_finish(m, 4)
    # frame 4 is the last; 3 kept < 4, so floor(i*4/3) = 0, 1, 2, 4 are added where missing
    assert final.tolist() == [1, 1, 1, 0, 1] and added.tolist() == [1, 4, -1, -1, -1]
    s, m, r = oracle.ngff_scan_open(h, 10, 0.6, 2)   # the gap rule forces frame 4
    assert m.tolist() == [1, 0, 1, 0, 1] and r == 4


def random_stream(seed, T, nbins=12, mass=60, scenes=5):
    rng = np.random.default_rng([2609, 3675, 92, seed])
    cut = np.sort(rng.integers(0, T, scenes))
    base = rng.dirichlet(np.ones(nbins), scenes + 1)
    h = np.zeros((T, nbins), np.uint32)
    for t in range(T):
        p = base[np.searchsorted(cut, t, side="right")]
        h[t] = rng.multinomial(mass, p)
    return h


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("L_max,M_min", [(30, 4), (5, 4), (1, 2), (0, 4), (12, 0), (7, 9)])
def test_open_then_finish_equals_one_shot(seed, L_max, M_min):
    T = [1, 2, 17, 64, 150, 301][seed]
    h = random_stream(seed, T)
    for tau in (-1.0, 0.05, 0.2, 0.5, 2.0):
        s, m, _ = oracle.ngff_scan_open(h, 60, tau, L_max)
        final, added = oracle.ngff_finish(m, M_min)
        s1, m1, k1 = oracle.ngff_select(h, 60, tau, L_max, M_min)
        assert np.array_equal(s.view(np.uint32), s1.view(np.uint32))
        assert np.array_equal(final, m1) and int(final.sum()) == int(k1[0])
        assert sorted(a for a in added if a >= 0) == np.flatnonzero(final & ~m.astype(bool)).tolist()


@pytest.mark.parametrize("L_max", [30, 4, 0])
def test_causal(L_max):
    h = random_stream(11, 200)
    s, m, _ = oracle.ngff_scan_open(h, 60, 0.15, L_max)
    for t in (1, 2, 31, 99, 150, 199):
        sp, mp, rp = oracle.ngff_scan_open(h[:t], 60, 0.15, L_max)
        assert np.array_equal(sp.view(np.uint32), s[:t].view(np.uint32)) and np.array_equal(mp, m[:t])
        assert rp == int(np.flatnonzero(m[:t]).max())


def test_degenerate_thresholds():
    h = random_stream(3, 50)
    _, m, _ = oracle.ngff_scan_open(h, 60, -1.0, 30)   # every frame novel enough
    assert m.all()
    _, m, _ = oracle.ngff_scan_open(h, 60, 1.5, 7)     # only frame 0 and the gap rule
    assert np.flatnonzero(m).tolist() == list(range(0, 50, 7))
    _, m, _ = oracle.ngff_scan_open(h, 60, 1.5, 0)     # no gap rule: frame 0 only
    assert np.flatnonzero(m).tolist() == [0]
    final, added = oracle.ngff_finish(m, 4)
    assert np.flatnonzero(final).tolist() == [0, 16, 32, 49] and added.tolist() == [16, 32, 49, -1, -1]
