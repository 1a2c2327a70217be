"""Pins for the NGFF oracle (Sec. 3.2): closed-form frames, invariants,
brute force and an independent formulation of the keep rule.

Nothing here compares the oracle with itself: histograms are checked against
hand-built frames whose counts are known and against numpy.bincount over an
explicit bin-edge digitisation; distances against hand-computed values; the
keep rule against closed-form streams and against a second formulation that
works in the integer domain (next-candidate chains and a threshold-vectorised
scan).
"""
import numpy as np
import pytest

import oracle
from oracle import GRAY, JOINT3D, PER_CHANNEL
from paper_2609_03675_amd import synth


def edge_bin(v, B):
    """Bin of v/255 among B equal bins over [0, 1] (value 1.0 in the last bin),
    by comparison with explicit edges b/B."""
    x = np.asarray(v, dtype=np.float64) / 255.0
    return np.digitize(x, np.arange(1, B) / B)


def luma(r, g, b):
    """BT.601 luma rounded half up, in exact rationals (r,g,b integers)."""
    from fractions import Fraction
    y = Fraction(299 * int(r) + 587 * int(g) + 114 * int(b), 1000)
    return int(y + Fraction(1, 2))  # floor(y + 1/2), y >= 0


def solid(n, H, W, rgb):
    f = np.empty((n, H, W, 3), dtype=np.uint8)
    f[...] = np.asarray(rgb, dtype=np.uint8)
    return f


# ----------------------------------------------------------------- bin rule --

@pytest.mark.parametrize("B", [2, 4, 8, 16, 32, 64, 128, 256])
def test_bin_edges_equal_shift_for_power_of_two(B):
    """For power-of-two B the normalised-range bins equal v >> (8 - log2 B)."""
    v = np.arange(256)
    shift = 8 - int(np.log2(B))
    assert np.array_equal(edge_bin(v, B), v >> shift)


@pytest.mark.parametrize("B", [8, 16, 32])
def test_bin_rule_over_all_values(B):
    """One frame holding every byte value once per channel: each bin receives
    exactly the values the edge rule puts there."""
    v = np.arange(256, dtype=np.uint8)
    f = np.stack([v, v, v], axis=-1).reshape(1, 16, 16, 3)
    h = oracle.histogram(f, B, PER_CHANNEL)[0]
    expect = np.bincount(edge_bin(v, B), minlength=B)
    for c in range(3):
        assert np.array_equal(h[c * B:(c + 1) * B], expect)


# -------------------------------------------------------- closed-form frames --

@pytest.mark.parametrize("mode,B", [(PER_CHANNEL, 16), (PER_CHANNEL, 32), (JOINT3D, 8),
                                    (GRAY, 32), (JOINT3D, 4), (GRAY, 256)])
def test_solid_colour_single_bin(mode, B):
    rgb = (200, 17, 96)
    H, W = 9, 13
    N = H * W
    h = oracle.histogram(solid(1, H, W, rgb), B, mode)[0]
    br, bg, bb = (int(edge_bin(x, B)) for x in rgb)
    expect = np.zeros(oracle.nbins(mode, B), dtype=np.int64)
    if mode == PER_CHANNEL:
        expect[br] += N
        expect[B + bg] += N
        expect[2 * B + bb] += N
    elif mode == JOINT3D:
        expect[(br * B + bg) * B + bb] = N
    else:
        expect[int(edge_bin(luma(*rgb), B))] = N
    assert np.array_equal(h, expect)


def test_two_colour_split_counts():
    H, W = 20, 30
    N = H * W
    k = 137
    f = solid(1, H, W, (10, 100, 250)).reshape(N, 3)
    f[:k] = (250, 10, 100)
    f = f.reshape(1, H, W, 3)
    B = 32
    h = oracle.histogram(f, B, PER_CHANNEL)[0]
    # channel R: k pixels at 250, N-k at 10
    assert h[edge_bin(250, B)] == k and h[edge_bin(10, B)] == N - k
    assert h[B + edge_bin(10, B)] == k and h[B + edge_bin(100, B)] == N - k
    assert h[2 * B + edge_bin(100, B)] == k and h[2 * B + edge_bin(250, B)] == N - k
    assert h.sum() == 3 * N
    j = oracle.histogram(f, 8, JOINT3D)[0]
    assert sorted(j[j > 0].tolist()) == sorted([k, N - k])


@pytest.mark.parametrize("B", [8, 16, 32])
def test_ramp_uniform_bins(B):
    """v = x over W = 256 columns: every bin holds N/B pixels per channel."""
    H, W = 3, 256
    row = np.arange(256, dtype=np.uint8)
    f = np.broadcast_to(row[None, :, None], (H, W, 3)).copy()[None]
    h = oracle.histogram(f, B, PER_CHANNEL)[0]
    assert np.all(h == H * W // B)


def test_gray_of_equal_channels_is_identity():
    v = np.arange(256, dtype=np.uint8)
    f = np.stack([v, v, v], axis=-1).reshape(1, 16, 16, 3)
    g = oracle.histogram(f, 256, GRAY)[0]
    assert np.all(g == 1)  # Y = v for R = G = B = v: one pixel per intensity
    single = oracle.histogram(v.reshape(1, 16, 16), 256, GRAY)[0]
    assert np.array_equal(g, single)


@pytest.mark.parametrize("rgb,y", [((255, 0, 0), 76), ((0, 255, 0), 150), ((0, 0, 255), 29),
                                   ((255, 255, 255), 255), ((0, 0, 0), 0)])
def test_gray_primaries_textbook_luma(rgb, y):
    """BT.601 luma of the primaries: 0.299*255 = 76.2, 0.587*255 = 149.7, 0.114*255 = 29.1."""
    h = oracle.histogram(solid(1, 2, 2, rgb), 256, GRAY)[0]
    assert h[y] == 4 and h.sum() == 4


def test_gray_random_pixels_match_rational_luma():
    r = np.random.default_rng(5)
    px = r.integers(0, 256, size=(1, 8, 8, 3)).astype(np.uint8)
    h = oracle.histogram(px, 256, GRAY)[0]
    ys = [luma(*p) for p in px.reshape(-1, 3)]
    assert np.array_equal(h, np.bincount(ys, minlength=256))


# ---------------------------------------------------------------- invariants --

@pytest.mark.parametrize("mode,B", [(PER_CHANNEL, 32), (JOINT3D, 8), (GRAY, 32)])
def test_mass_and_permutation_invariance(mode, B):
    f = synth.random_frames(1, 3, 24, 40)
    h = oracle.histogram(f, B, mode)
    N = 24 * 40
    if mode == PER_CHANNEL:
        assert np.all(h.reshape(3, 3, B).sum(axis=2) == N)
    else:
        assert np.all(h.sum(axis=1) == N)
    assert oracle.mass(mode, 24, 40) == h[0].sum()
    perm = np.random.default_rng(2).permutation(N)
    g = f.reshape(3, N, 3)[:, perm].reshape(f.shape)
    assert np.array_equal(oracle.histogram(g, B, mode), h)


@pytest.mark.parametrize("mode,B", [(PER_CHANNEL, 16), (PER_CHANNEL, 32), (JOINT3D, 8),
                                    (GRAY, 32)])
def test_histogram_vs_bincount(mode, B):
    """Brute force with numpy: digitise by explicit edges, then bincount."""
    f = synth.frames(1, 0, 0, 8)
    h = oracle.histogram(f, B, mode)
    n = f.shape[0]
    px = f.reshape(n, -1, 3).astype(np.int64)
    for t in range(n):
        if mode == PER_CHANNEL:
            e = np.concatenate([np.bincount(edge_bin(px[t, :, c], B), minlength=B) for c in range(3)])
        elif mode == JOINT3D:
            b = edge_bin(px[t], B)
            e = np.bincount((b[:, 0] * B + b[:, 1]) * B + b[:, 2], minlength=B ** 3)
        else:
            y = (299 * px[t, :, 0] + 587 * px[t, :, 1] + 114 * px[t, :, 2] + 500) // 1000
            e = np.bincount(edge_bin(y, B), minlength=B)
        assert np.array_equal(h[t], e)


# ----------------------------------------------------------------- distances --

def test_tv_identical_zero_and_disjoint_one():
    B = 32
    a = solid(1, 10, 10, (0, 0, 0))
    b = solid(1, 10, 10, (255, 255, 255))
    frames = np.concatenate([a, a, b])
    for mode, bins in [(PER_CHANNEL, B), (JOINT3D, 8), (GRAY, B)]:
        h = oracle.histogram(frames, bins, mode)
        M = oracle.mass(mode, 10, 10)
        s, _, _ = oracle.ngff_select(h, M, tau=2.0, L_max=0, M_min=0)
        assert s[1] == 0.0              # identical consecutive frames: novelty 0
        assert s[2] == 1.0              # disjoint colours: maximal novelty (D = 2M)
        assert oracle.l1(h[0], h[2]) == 2 * M


def test_tv_metric_properties_and_rounding():
    f = synth.frames(2, 0, 0, 6)
    h = oracle.histogram(f, 32, PER_CHANNEL)
    M = oracle.mass(PER_CHANNEL, 448, 448)
    D = np.array([[oracle.l1(h[i], h[j]) for j in range(6)] for i in range(6)])
    assert np.array_equal(D, D.T) and np.all(np.diag(D) == 0)
    for i in range(6):
        for j in range(6):
            for k in range(6):
                assert D[i, k] <= D[i, j] + D[j, k]
    assert np.all((D >= 0) & (D <= 2 * M))
    # fl32 score is within half an fp32 ulp of the fp64 TV of normalised
    # histograms; with tau > 1 and no L_max nothing is kept, so r(t) = 0
    hn = h.astype(np.float64) / M
    s, _, _ = oracle.ngff_select(h, M, tau=2.0, L_max=0, M_min=0)
    for t in range(1, 6):
        tv = max(0.5 * np.abs(hn[t] - hn[t - 1]).sum(), 0.5 * np.abs(hn[t] - hn[0]).sum())
        assert abs(float(s[t]) - tv) <= 0.5 * np.spacing(np.float32(tv)) * (1 + 1e-9)


def test_per_channel_tv_is_mean_of_channel_tvs():
    f = synth.frames(2, 0, 10, 2)
    B = 32
    h = oracle.histogram(f, B, PER_CHANNEL).astype(np.int64)
    N = 448 * 448
    per = [0.5 * np.abs(h[1, c * B:(c + 1) * B] - h[0, c * B:(c + 1) * B]).sum() / N for c in range(3)]
    s, _, _ = oracle.ngff_select(h, 3 * N, tau=2.0, L_max=0, M_min=0)
    assert abs(float(s[1]) - np.mean(per)) < 1e-7


# ---------------------------------------------------------------- keep rule --

def test_static_video_closed_form():
    """Identical frames: only forced keeps survive: {0, T-1} and every L_max."""
    T, L = 100, 30
    h = oracle.histogram(solid(T, 4, 4, (1, 2, 3)), 16, PER_CHANNEL)
    s, m, kept = oracle.ngff_select(h, 48, tau=0.3, L_max=L, M_min=4)
    assert np.flatnonzero(m).tolist() == [0, 30, 60, 90, 99]
    assert kept.tolist() == [5]
    assert s[0] == 1.0 and np.all(s[1:] == 0)


def test_alternating_frames_all_kept():
    a, b = solid(1, 5, 5, (0, 0, 0)), solid(1, 5, 5, (255, 255, 255))
    f = np.concatenate([a, b] * 10)
    h = oracle.histogram(f, 32, PER_CHANNEL)
    for tau in (0.0, 0.5, 1.0):
        _, m, _ = oracle.ngff_select(h, 75, tau=tau, L_max=30, M_min=4)
        assert m.all()


def drift_stream(T=40, side=80, cap=20):
    """Frame t has min(t, cap) * N/20 pixels switched to a disjoint colour."""
    N = side * side
    f = np.empty((T, N, 3), dtype=np.uint8)
    for t in range(T):
        k = min(t, cap) * N // 20
        f[t] = (0, 0, 0)
        f[t, :k] = (255, 255, 255)
    return f.reshape(T, side, side, 3)


def test_drift_ramp_reference_term():
    """Gradual drift is caught only by the reference term s_ref = 0.05 (t - r):
    with tau = 0.3 every sixth frame is kept (Eq. 3-5), then the last."""
    f = drift_stream()
    h = oracle.histogram(f, 32, PER_CHANNEL)
    M = oracle.mass(PER_CHANNEL, 80, 80)
    s, m, _ = oracle.ngff_select(h, M, tau=np.float32(0.3), L_max=30, M_min=4)
    assert np.flatnonzero(m).tolist() == [0, 6, 12, 18, 39]
    assert s[1] == np.float32(0.05) and s[6] == np.float32(0.3)
    # adjacent term alone (reference = previous frame) would never reach 0.3
    assert np.all(s[1:20][[i for i in range(19) if (i + 1) % 6]] < np.float32(0.3))


def test_top_up_uniform_spacing():
    T = 10
    h = oracle.histogram(solid(T, 3, 3, (9, 9, 9)), 16, PER_CHANNEL)
    _, m, kept = oracle.ngff_select(h, 27, tau=0.5, L_max=30, M_min=4)
    assert np.flatnonzero(m).tolist() == [0, 3, 6, 9]  # floor(i*9/3)
    assert kept.tolist() == [4]
    _, m, _ = oracle.ngff_select(h[:3], 27, tau=0.5, L_max=30, M_min=8)
    assert m.all()  # M_min >= T keeps everything


@pytest.mark.parametrize("T", [1, 2])
def test_short_streams_keep_all(T):
    h = oracle.histogram(solid(T, 3, 3, (9, 9, 9)), 16, PER_CHANNEL)
    s, m, _ = oracle.ngff_select(h, 27, tau=0.9, L_max=30, M_min=0)
    assert m.all() and s[0] == 1.0


def chain_select(h, M, theta, L, T):
    """Second formulation in the integer domain: from each kept r, jump to
    next(r) = min{t > r : max(D(t,t-1), D(t,r)) >= theta or t - r >= L or t = T-1}."""
    D = lambda i, j: int(np.abs(h[i].astype(np.int64) - h[j].astype(np.int64)).sum())
    keep = [0]
    r = 0
    while r < T - 1:
        t = r + 1
        while not (t == T - 1 or max(D(t, t - 1), D(t, r)) >= theta or (L > 0 and t - r >= L)):
            t += 1
        keep.append(t)
        r = t
    return keep


@pytest.mark.parametrize("seed", range(6))
def test_keep_rule_matches_chain_formulation(seed):
    f = synth.random_frames(seed, 50, 6, 7, scenes=6)
    h = oracle.histogram(f, 16, PER_CHANNEL)
    M = oracle.mass(PER_CHANNEL, 6, 7)
    for theta in (0, 5, 40, 90, 200, 2 * M + 1):
        tau = np.float32(theta) / np.float32(2 * M)
        for L in (0, 1, 4, 30):
            _, m, _ = oracle.ngff_select(h, M, tau=tau, L_max=L, M_min=0)
            assert np.flatnonzero(m).tolist() == chain_select(h, M, theta, L, 50)


def test_segments_are_independent():
    f = synth.random_frames(3, 60, 5, 5, scenes=8)
    h = oracle.histogram(f, 16, PER_CHANNEL)
    M = oracle.mass(PER_CHANNEL, 5, 5)
    taus = np.array([0.1, 0.2, 0.35, 0.5], dtype=np.float32)
    s, m, kept = oracle.ngff_select(h, M, tau=taus, L_max=7, M_min=3, seg_len=16)
    for i, t0 in enumerate(range(0, 60, 16)):
        s1, m1, k1 = oracle.ngff_select(h[t0:t0 + 16], M, tau=taus[i], L_max=7, M_min=3)
        assert np.array_equal(s[t0:t0 + 16], s1) and np.array_equal(m[t0:t0 + 16], m1)
        assert kept[i] == k1[0]


# ---------------------------------------------------------- calibration rule --

def vectorised_counts(h, M, L, M_min, thetas):
    """Kept count (top-up included) for every integer threshold at once."""
    h = h.astype(np.int64)
    T = h.shape[0]
    th = np.asarray(thetas, dtype=np.int64)
    r = np.zeros(th.size, dtype=np.int64)
    keep = np.zeros((th.size, T), dtype=bool)
    keep[:, 0] = True
    for t in range(1, T):
        dadj = np.abs(h[t] - h[t - 1]).sum()
        dref = np.abs(h[t][None, :] - h[r]).sum(axis=1)
        k = (np.maximum(dadj, dref) >= th) | (t == T - 1)
        if L > 0:
            k |= (t - r) >= L
        keep[:, t] = k
        r = np.where(k, t, r)
    cnt = keep.sum(axis=1)
    if M_min >= 2:
        for i in np.flatnonzero(cnt < M_min):
            for j in range(M_min):
                keep[i, (j * (T - 1)) // (M_min - 1)] = True
        cnt = keep.sum(axis=1)
    return cnt


@pytest.mark.parametrize("case", ["tiny_workload", "random_a", "random_b"])
def test_calibration_brute_force_all_thresholds(case):
    if case == "tiny_workload":
        wl = synth.WORKLOADS[1]
        f = synth.frames(1)
        B, H, W, target = wl.bins, wl.H, wl.W, wl.target
    else:
        seed = 11 if case == "random_a" else 12
        f = synth.random_frames(seed, 40, 4, 6, scenes=9)
        B, H, W, target = 16, 4, 6, 13
    h = oracle.histogram(f, B, PER_CHANNEL)
    M = oracle.mass(PER_CHANNEL, H, W)
    L = 30 if case == "tiny_workload" else 5
    theta, tau = oracle.ngff_calibrate(h, M, target, L_max=L, M_min=4)
    allth = np.arange(0, 2 * M + 2)
    cnt = vectorised_counts(h, M, L, 4, allth)
    ok = np.flatnonzero(cnt <= target)
    theta_bf = int(allth[ok[0]]) if ok.size else 2 * M + 1
    # the oracle answers with the smallest candidate distance >= the brute-force
    # minimum; both keep the same frames
    T = h.shape[0]
    cands = {0, 2 * M + 1}
    for t in range(1, T):
        for k in range(1, min(L, t) + 1):
            cands.add(oracle.l1(h[t], h[t - k]))
    assert int(theta[0]) == min(c for c in cands if c >= theta_bf)
    assert cnt[int(theta[0])] == cnt[theta_bf] <= target
    assert tau[0] == np.float32(theta[0]) / np.float32(2 * M)
    _, m, kept = oracle.ngff_select(h, M, tau=tau[0], L_max=L, M_min=4)
    assert kept[0] == cnt[theta_bf]


def test_count_not_monotone_in_threshold_exists():
    """The kept count can rise with the threshold (r(t) depends on history),
    which is why calibration evaluates every candidate."""
    found = False
    for seed in range(200):
        f = synth.random_frames(1000 + seed, 12, 2, 3, scenes=12)
        h = oracle.histogram(f, 8, PER_CHANNEL)
        M = oracle.mass(PER_CHANNEL, 2, 3)
        c = vectorised_counts(h, M, 0, 0, np.arange(0, 2 * M + 2))
        if np.any(np.diff(c) > 0):
            found = True
            break
    assert found


def test_workload_targets():
    assert [synth.WORKLOADS[i].target for i in range(1, 6)] == [26, 128, 720, 307, 128]


def _rn32_exact(D, N):
    """D/N rounded to the nearest fp32, ties to even, decided with exact
    rationals among the float32 neighbours of a first guess."""
    from fractions import Fraction
    x = Fraction(D, N)
    g = np.float32(D / N)
    cands = [np.nextafter(g, np.float32(-np.inf)), g, np.nextafter(g, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - x), int(np.float32(c).view(np.uint32)) & 1))
    return np.float32(best)


def test_score_is_the_correctly_rounded_quotient():
    """The novelty score D / 2M (Eq. 2) rounded once to fp32, for 2M below
    and far above 2^24 (4K frames per channel: 2M = 6 * 3840 * 2160), against
    exact rational rounding; below 2^24 it equals one IEEE division of the
    exact operands."""
    rng = np.random.default_rng([2609, 3675, 66])
    for N in (2 * 64 * 64, 2 * 3 * 448 * 448, (1 << 24) - 2, 1 << 24, 6 * 3840 * 2160, (1 << 31) - 2, 12345679):
        Ds = list(rng.integers(0, N + 2, 300)) + [0, 1, 2, N - 1, N, N + 1]
        for D in Ds:
            got = oracle.score(int(D), N)
            assert got.view(np.uint32) == _rn32_exact(int(D), N).view(np.uint32), (D, N)
            if N < (1 << 24):
                assert got == np.float32(np.float32(D) / np.float32(N))


def test_score_ties_round_to_even():
    """Quotients exactly halfway between two fp32 values: the fp32 spacing in
    [2^-2, 2^-1) is 2^-25, so D / 2^26 with D odd in [2^24, 2^25) lies on a
    midpoint; ties go to the even significand."""
    N = 1 << 26
    for D in ((1 << 24) + 1, (1 << 24) + 3, (1 << 25) - 1):
        got = oracle.score(D, N)
        assert got.view(np.uint32) == _rn32_exact(D, N).view(np.uint32)
        assert got.view(np.uint32) & 1 == 0
