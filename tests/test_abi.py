"""The C ABI without a GPU: the library loads, exports every function the
header declares, its host helpers match the paper's printed values, and every
host-side validation error is reported before any GPU work."""
import ctypes
import os

import numpy as np
import pytest

from paper_2609_03675_amd import binding as B

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return True


@pytest.fixture(scope="module")
def L():
    return B.lib()


def test_exports_every_declared_symbol(L):
    names = B.declared_functions()
    assert len(names) >= 16
    for n in names:
        assert hasattr(L, n), n


def test_version(L):
    assert b"gfx950" in L.cofie_version()


def test_drop_ratio_compositions_printed_in_paper():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "drop_ratio_compositions.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 12
    for r in rows:
        dn, dq, printed = float(r[0]) / 100, float(r[1]) / 100, float(r[2])
        total = 100 * B.cofie_drop_total(dn, dq)
        assert abs(total - printed) <= 0.5 + 1e-9, r
    assert B.cofie_drop_total(0.2, 0.375) == pytest.approx(0.5, abs=1e-15)


def test_paper_defaults(L):
    vals = {l.split()[0]: l.split()[1] for l in open(os.path.join(GOLDEN, "paper_defaults.txt"))
            if l.strip() and not l.startswith("#")}
    r = B.KeepRule()
    L.cofie_keep_rule_default(ctypes.byref(r))
    assert r.M_min == int(vals["M_min"]) and r.L_max == int(vals["L_max"])
    assert r.tau_h == np.float32(float(vals["tau_h"]))
    assert r.hist_mode == B.GRAY and r.segment_len == 0
    assert B.cofie_ngff_nbins("gray", int(vals["bins"])) == 32


def test_k_from_ratio_eq8():
    """k = max(1, round(rho |S_c|)) (Eq. 8), half to even."""
    assert B.cofie_qer_k_from_ratio(0.5, 256) == 128
    assert B.cofie_qer_k_from_ratio(0.3, 1024) == 307
    assert B.cofie_qer_k_from_ratio(0.01, 10) == 1
    assert B.cofie_qer_k_from_ratio(0.5, 5) == 2     # 2.5 -> 2
    assert B.cofie_qer_k_from_ratio(0.5, 7) == 4     # 3.5 -> 4
    assert B.cofie_qer_k_from_ratio(0.4, 0) == 0
    assert B.cofie_qer_k_from_ratio(-0.1, 10) == -1


def test_nbins():
    assert B.cofie_ngff_nbins("per_channel", 32) == 96
    assert B.cofie_ngff_nbins("joint3d", 8) == 512
    assert B.cofie_ngff_nbins("gray", 32) == 32
    assert B.cofie_ngff_nbins(7, 32) == 0
    assert B.cofie_ngff_nbins("framediff", 32) == 1024   # G x G cell means
    assert B.cofie_ngff_nbins("dhash", 8) == 64           # 64 hash bits


def test_workspace_sizes_are_host_only():
    r = B.keep_rule("per_channel", L_max=30, segment_len=512)
    ws = B.ngff_workspace_bytes(16384, 448, 448, 3, 32, r)
    assert ws >= 16384 * (96 + 30 + 1) * 4  # hist + band + next
    assert B.ngff_workspace_bytes(16, 448, 448, 3, 33, r) == 0   # invalid bins
    d = B.qer_desc(32, 32768, 128, 28, 28, 128)
    assert B.qer_workspace_bytes(d, 16) >= 32768 * 4
    g = B.qer_desc(48, 58800, 300, 28, 4, 128)
    assert B.qer_workspace_bytes(g, 24) >= 58800 * 4 + 3 * 48 * 512 * 2
    assert B.qer_workspace_bytes(B.qer_desc(32, 10, 2, 28, 5, 128), 4) == 0  # H_q % H_kv


# Every case below is rejected by host validation before any HIP call; the
# fake pointer is never dereferenced.  Skipped where a GPU exists so that a
# validation bug can never turn into a device access.
FAKE = 0x1000


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
@pytest.mark.parametrize("args,code", [
    ((None, 4, 8, 8, 3, 32, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),        # frames NULL
    ((FAKE, -1, 8, 8, 3, 32, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),       # n < 0
    ((FAKE, 4, 0, 8, 3, 32, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),        # H = 0
    ((FAKE, 4, 8, 8, 2, 32, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),        # C = 2
    ((FAKE, 4, 8, 8, 1, 32, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),        # C = 1 needs GRAY
    ((FAKE, 4, 8, 8, 3, 32, 9, FAKE), B.COFIE_EINVAL),                     # bad mode
    ((FAKE, 4, 8, 8, 3, 1, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),         # bins < 2
    ((FAKE, 4, 8, 8, 3, 512, B.PER_CHANNEL, FAKE), B.COFIE_EINVAL),       # bins > 256
    ((FAKE, 4, 8, 8, 3, 24, B.PER_CHANNEL, FAKE), B.COFIE_EUNSUPPORTED),  # not a power of two
    ((FAKE, 4, 8, 8, 3, 32, B.JOINT3D, FAKE), B.COFIE_EUNSUPPORTED),      # 32^3 bins
    ((FAKE, 4, 20000, 20000, 3, 32, B.PER_CHANNEL, FAKE), B.COFIE_EUNSUPPORTED),  # 2M >= 2^31
    ((FAKE, 4, 8, 8, 3, 32, B.PER_CHANNEL, None), B.COFIE_EINVAL),        # out NULL
    ((FAKE, 4, 64, 64, 3, 24, B.FRAMEDIFF, FAKE), B.COFIE_EUNSUPPORTED),  # grid not a power of two
    ((FAKE, 4, 64, 64, 3, 128, B.FRAMEDIFF, FAKE), B.COFIE_EUNSUPPORTED), # grid above 64
    ((FAKE, 4, 16, 64, 3, 32, B.FRAMEDIFF, FAKE), B.COFIE_EINVAL),        # grid finer than H
    ((FAKE, 4, 7, 64, 3, 8, B.DHASH, FAKE), B.COFIE_EINVAL),              # dHash needs H >= 8
    ((FAKE, 4, 64, 8, 3, 8, B.DHASH, FAKE), B.COFIE_EINVAL),              # and W >= 9
    ((FAKE, 4, 64, 20000, 3, 8, B.DHASH, FAKE), B.COFIE_EUNSUPPORTED),    # W above 16384
])
def test_histogram_validation(L, args, code):
    assert L.cofie_ngff_histogram(*args, None) == code
    assert L.cofie_last_error()


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
def test_filter_validation(L):
    r = B.KeepRule()
    L.cofie_keep_rule_default(ctypes.byref(r))
    assert L.cofie_ngff_filter(FAKE, 4, 8, 8, 3, 32, None, FAKE, FAKE, None) == B.COFIE_EINVAL
    r.tau_h = float("nan")
    assert L.cofie_ngff_filter(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), FAKE, FAKE, None) == B.COFIE_EINVAL
    r.tau_h = 0.3
    r.M_min = -1
    assert L.cofie_ngff_filter(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), FAKE, FAKE, None) == B.COFIE_EINVAL
    r.M_min = 4
    r.segment_len = -5
    assert L.cofie_ngff_filter(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), FAKE, FAKE, None) == B.COFIE_EINVAL
    r.segment_len = 0
    assert L.cofie_ngff_filter(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), None, FAKE, None) == B.COFIE_EINVAL
    # n = 0 is a valid no-op that touches nothing
    assert L.cofie_ngff_filter(None, 0, 8, 8, 3, 32, ctypes.byref(r), None, None, None) == B.COFIE_OK
    r.L_max = 0
    assert L.cofie_ngff_calibrate(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), 2, FAKE, None) == B.COFIE_EUNSUPPORTED
    # the keep rule on given histograms validates the same way
    r.L_max = 30
    assert L.cofie_ngff_filter_hist(FAKE, 4, 8, 8, 3, 32, None, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_ngff_filter_hist(None, 4, 8, 8, 3, 32, ctypes.byref(r), FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_ngff_filter_hist(FAKE, 4, 8, 8, 3, 32, ctypes.byref(r), FAKE, None, None) == B.COFIE_EINVAL
    assert L.cofie_ngff_filter_hist(FAKE, 4, 8, 8, 3, 24, ctypes.byref(r), FAKE, FAKE, None) == B.COFIE_EUNSUPPORTED
    assert L.cofie_ngff_filter_hist(None, 0, 8, 8, 3, 32, ctypes.byref(r), None, None, None) == B.COFIE_OK


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
@pytest.mark.parametrize("field,value,code", [
    ("n_q", 0, B.COFIE_EINVAL),
    ("n_vis", -1, B.COFIE_EINVAL),
    ("H_kv", 3, B.COFIE_EINVAL),          # 28 % 3
    ("d", 24, B.COFIE_EUNSUPPORTED),      # not a multiple of 16
    ("dtype", 5, B.COFIE_EINVAL),
    ("score_mode", 7, B.COFIE_EINVAL),
])
def test_qer_validation(L, field, value, code):
    d = B.qer_desc(32, 64, 4, 28, 28, 128)
    setattr(d, field, value)
    assert L.cofie_qer_rank(FAKE, FAKE, FAKE, ctypes.byref(d), 2, FAKE, FAKE, None) == code


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
def test_qer_null_and_alignment_validation(L):
    d = B.qer_desc(32, 64, 4, 28, 28, 128)
    assert L.cofie_qer_rank(None, FAKE, FAKE, ctypes.byref(d), 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE, None, FAKE, ctypes.byref(d), 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE, FAKE, None, ctypes.byref(d), 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE, FAKE, FAKE, ctypes.byref(d), 2, FAKE, None, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE, FAKE, FAKE, ctypes.byref(d), -1, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE + 4, FAKE, FAKE, ctypes.byref(d), 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank(FAKE, FAKE, FAKE, None, 2, FAKE, FAKE, None) == B.COFIE_EINVAL


def test_diag_copy_validation(L):
    assert L.cofie_diag_stream_copy(FAKE, FAKE, 0, None) == B.COFIE_OK
    if _no_gpu():
        assert L.cofie_diag_stream_copy(FAKE, FAKE + 8, 32, None) == B.COFIE_EINVAL


def test_stream_checkpoint_validation(L):
    assert L.cofie_ngff_stream_state_bytes(None) == 0
    buf = ctypes.create_string_buffer(64)
    assert L.cofie_ngff_stream_save(None, buf, 64, None) == B.COFIE_EINVAL
    assert L.cofie_ngff_stream_restore(None, buf, 64, None) == B.COFIE_EINVAL


def test_softmax_workspace_holds_per_wave_statistics(L):
    """SOFTMAX with heads of whole 128-byte key segments runs both passes in
    the score kernel; its workspace holds one (max, sum) pair per wave, round
    and (head, query row), rows in blocks of 16.  Without a GPU the planner
    takes 256 CUs: the 1 fps stream's 2048 tiles give 256 workgroups x 8 waves
    in one round, 28 x 32 rows."""
    soft = B.qer_workspace_bytes(B.qer_desc(32, 32768, 128, 28, 28, 128, score_mode=B.SOFTMAX), 16)
    logit = B.qer_workspace_bytes(B.qer_desc(32, 32768, 128, 28, 28, 128), 16)
    assert soft >= 256 * 8 * (28 * 32) * 8 > logit > 0
    # heads of 32 bf16 elements take the per-head kernels: per 32-token block statistics
    small = B.qer_workspace_bytes(B.qer_desc(32, 32768, 128, 28, 28, 32, score_mode=B.SOFTMAX), 16)
    assert small >= (32768 // 32) * 28 * 32 * 8


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
def test_batched_softmax_workspace_and_refusal(L):
    """Several queries in SOFTMAX mode keep one (max, sum) pair per wave,
    round and stacked (head, query row): four queries of 32 rows over the
    1 fps stream's 2048 tiles take 256 workgroups x 8 waves x 28 x 128 rows.
    Heads that are not whole 128-byte key segments are refused for several
    queries (the per-head fallback has no per-query key range)."""
    d = B.qer_desc(32, 32768, 128, 28, 28, 128, score_mode=B.SOFTMAX)
    four = B.lib().cofie_qer_batched_workspace_bytes(ctypes.byref(d), 4, 16)
    one = B.lib().cofie_qer_batched_workspace_bytes(ctypes.byref(d), 1, 16)
    assert four >= 256 * 8 * (28 * 4 * 32) * 8 > one > 0
    d32 = B.qer_desc(16, 64, 4, 2, 2, 32, score_mode=B.SOFTMAX)
    nf = (ctypes.c_int32 * 2)(4, 3)
    assert L.cofie_qer_rank_batched(FAKE, FAKE, FAKE, ctypes.byref(d32), 2, nf, 2, FAKE, FAKE,
                                    None) == B.COFIE_EUNSUPPORTED


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
def test_batched_qer_validation(L):
    d = B.qer_desc(16, 64, 4, 2, 2, 32)
    nf = (ctypes.c_int32 * 2)(4, 5)   # 5 > n_frames
    assert L.cofie_qer_rank_batched(FAKE, FAKE, FAKE, ctypes.byref(d), 2, nf, 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    nf[1] = 3
    assert L.cofie_qer_rank_batched(FAKE, FAKE, FAKE, ctypes.byref(d), 0, nf, 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    assert L.cofie_qer_rank_batched(FAKE, FAKE, FAKE, ctypes.byref(d), 2, None, 2, FAKE, FAKE, None) == B.COFIE_EINVAL
    d20 = B.qer_desc(20, 64, 4, 2, 2, 32)
    assert L.cofie_qer_rank_batched(FAKE, FAKE, FAKE, ctypes.byref(d20), 2, nf, 2, FAKE, FAKE,
                                    None) == B.COFIE_EUNSUPPORTED
    assert B.lib().cofie_qer_batched_workspace_bytes(ctypes.byref(d), 3, 2) > \
        B.lib().cofie_qer_workspace_bytes(ctypes.byref(d), 2)


@pytest.mark.skipif(not _no_gpu(), reason="host-only validation checks")
def test_streams_qer_validation(L):
    """cofie_qer_rank_streams refuses inconsistent sequence tables, prefixes
    past a sequence's frames, SOFTMAX and query widths it does not tile, all
    before any GPU work; its workspace holds one m row per query as long as
    the longest sequence."""
    lay = B.StreamsLayout([40, 0, 24], [3, 0, 2], [2, 1, 1], [3, 1, 0, 2])
    d = B.qer_desc(16, 64, 5, 2, 2, 32)

    def call(desc, layout, k=2):
        return L.cofie_qer_rank_streams(FAKE, FAKE, FAKE, ctypes.byref(desc), *layout.args(), k, FAKE, FAKE, None)

    ws = B.qer_streams_workspace_bytes(d, lay, 2)
    assert ws >= 4 * 40 * 4
    bad = B.StreamsLayout([40, 0, 24], [3, 0, 2], [2, 1, 1], [3, 1, 0, 3])   # 3 > the third sequence's 2 frames
    assert call(d, bad) == B.COFIE_EINVAL
    assert B.qer_streams_workspace_bytes(d, bad, 2) == 0
    short = B.StreamsLayout([40, 0, 20], [3, 0, 2], [2, 1, 1], [3, 1, 0, 2])  # keys end at 60 != n_vis 64
    assert call(d, short) == B.COFIE_EINVAL
    none = B.StreamsLayout([40, 0, 24], [3, 0, 2], [0, 0, 0], [])
    assert call(d, none) == B.COFIE_EINVAL
    soft = B.qer_desc(16, 64, 5, 2, 2, 32, score_mode=B.SOFTMAX)
    assert call(soft, lay) == B.COFIE_EUNSUPPORTED
    assert call(B.qer_desc(20, 64, 5, 2, 2, 32), lay) == B.COFIE_EUNSUPPORTED   # n_q not a multiple of 16
    assert call(B.qer_desc(144, 64, 5, 2, 2, 32), lay) == B.COFIE_EUNSUPPORTED  # more than 128 rows
    assert call(B.qer_desc(80, 64, 5, 4, 2, 32), lay) == B.COFIE_EUNSUPPORTED   # grouped heads: at most 64
    assert L.cofie_qer_rank_streams(FAKE, FAKE, FAKE, ctypes.byref(d), 0, None, None, None, None, 2, FAKE, FAKE,
                                    None) == B.COFIE_EINVAL


def test_online_state_refuses_the_table5_signals(L):
    """The online NGFF state keeps histogram rows only."""
    st = ctypes.c_void_p()
    for mode in (B.FRAMEDIFF, B.DHASH):
        r = B.keep_rule(mode, 0.3, 30, 4)
        assert L.cofie_ngff_stream_create(2, 64, 64, 3, 8, ctypes.byref(r), ctypes.byref(st)) == \
            B.COFIE_EUNSUPPORTED
