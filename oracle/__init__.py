"""CPU oracle for CoFiE's NGFF and QER stages (test infrastructure only).

Only the test-suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  It wraps the plain C oracle in
``cofie_oracle.c`` (built with gcc by :func:`build`) and shares nothing with
the HIP implementation in ``paper_2609_03675_amd``.

Paper sections followed: Sec. 3.2 (NGFF: histogram, total-variation distance,
Eqs. 2-5 and the gap-aware safeguards), Sec. 3.3 (QER: Eqs. 6-8) and the glue
between them (the candidate set S_c as frame indices, Sec. 3.1-3.2; removal of
the frames outside S_e from a token sequence, chronological, Sec. 3.3).

Parity status: every function here is pinned by the CPU tests under
``tests/test_oracle_*.py`` (closed forms, invariants, brute force, library
routines, the paper's printed drop-ratio compositions).  The retention-target
calibration (``ngff_calibrate``) is not in the paper; it is pinned by a brute
force over every integer threshold on small inputs.  The glue functions are
pinned by hand-built cases, numpy's flatnonzero and a row-by-row brute force
(``tests/test_oracle_glue.py``).  The online reading of the keep rule
(``ngff_scan_open`` / ``ngff_finish``: decisions as frames arrive, the two
end-of-stream safeguards when the stream ends) is pinned by a hand-computed
stream, causality, and equality with the one-shot rule
(``tests/test_oracle_ngff_stream.py``).  The evidence-preservation metrics of
the appendix are pinned by hand-computed cases and a numpy brute force
(``tests/test_oracle_evidence.py``).  The causal attention whose QK^T tiles
QER reads (``attention``) is pinned by closed forms (the first row, uniform
logits giving prefix means, a two-key sigmoid, the hard-attention limit) and
invariants (causality, key shifts, grouped heads as repeated heads, weights
that sum to one) in ``tests/test_oracle_attention.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cofie_oracle.c")
_LIB = os.path.join(_HERE, "libcofie_oracle.so")

GRAY, PER_CHANNEL, JOINT3D = 0, 1, 2
FRAMEDIFF, DHASH = 3, 4  # alternative pre-encoder signals (Table 5)
F32, BF16 = 0, 1
LOGIT, SOFTMAX = 0, 1

_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP).  Returns the library path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=False)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, f32, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    lib.orc_num_threads.restype = ctypes.c_int
    lib.orc_set_num_threads.argtypes = [ctypes.c_int]
    lib.orc_set_num_threads.restype = None
    lib.orc_nbins.argtypes = [i32, i32]
    lib.orc_nbins.restype = i64
    lib.orc_mass.argtypes = [i32, i32, i32]
    lib.orc_mass.restype = i64
    lib.orc_histogram.argtypes = [P, i64, i32, i32, i32, i32, i32, P]
    lib.orc_histogram.restype = ctypes.c_int
    lib.orc_signature.argtypes = [P, i64, i32, i32, i32, i32, i32, P]
    lib.orc_signature.restype = i64
    lib.orc_signal_two_m.argtypes = [i32, i32]
    lib.orc_signal_two_m.restype = i64
    lib.orc_score.argtypes = [i64, i64]
    lib.orc_score.restype = f32
    lib.orc_l1.argtypes = [P, P, i64]
    lib.orc_l1.restype = i64
    lib.orc_ngff_select.argtypes = [P, i64, i64, i64, P, i64, i32, i32, i64, P, P, P]
    lib.orc_ngff_select.restype = ctypes.c_int
    lib.orc_ngff_calibrate.argtypes = [P, i64, i64, i64, i32, i32, i64, i64, P, P]
    lib.orc_ngff_calibrate.restype = ctypes.c_int
    lib.orc_qer_scores.argtypes = [P, P, i32, P, i32, i32, i32, i32, i32, i32, i32, f64, P]
    lib.orc_qer_scores.restype = ctypes.c_int
    lib.orc_topk.argtypes = [P, i32, i32, P]
    lib.orc_topk.restype = ctypes.c_int
    lib.orc_ngff_scan_open.argtypes = [P, i64, i64, i64, f32, i32, P, P, P]
    lib.orc_ngff_scan_open.restype = i64
    lib.orc_ngff_finish.argtypes = [P, i64, i32, P]
    lib.orc_ngff_finish.restype = i64
    lib.orc_evidence_preservation.argtypes = [P, P, i32, f64, ctypes.POINTER(f64), ctypes.POINTER(f64)]
    lib.orc_evidence_preservation.restype = ctypes.c_int
    lib.orc_attention_rows.argtypes = [P, P, P, i32, i32, i32, i32, i32, f64, P, i32, P]
    lib.orc_attention_rows.restype = ctypes.c_int
    lib.orc_mask_compact.argtypes = [P, i64, i64, P, P]
    lib.orc_mask_compact.restype = i64
    lib.orc_gather_frames.argtypes = [P, i64, i64, P, i32, P, i32, P, i64, P, P]
    lib.orc_gather_frames.restype = i64
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    """OpenMP threads the oracle uses."""
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's later calls (timing; results do not depend on it)."""
    _load().orc_set_num_threads(int(n))


def nbins(mode: int, bins: int) -> int:
    return int(_load().orc_nbins(mode, bins))


def mass(mode: int, H: int, W: int) -> int:
    """Histogram mass M (count total); h_t = counts / M sums to 1."""
    return int(_load().orc_mass(mode, H, W))


def histogram(frames: np.ndarray, bins: int, mode: int) -> np.ndarray:
    """Counts [n][nbins] uint32 for uint8 frames [n][H][W][C] (Sec. 3.2)."""
    f = np.ascontiguousarray(frames, dtype=np.uint8)
    if f.ndim == 3:
        f = f[..., None]
    n, H, W, C = f.shape
    out = np.zeros((n, nbins(mode, bins)), dtype=np.uint32)
    rc = _load().orc_histogram(_ptr(f), n, H, W, C, bins, mode, _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle histogram rejected C={C} mode={mode}")
    return out


def signature(frames: np.ndarray, kind: int, grid: int = 32) -> np.ndarray:
    """Rows [n][nsig] uint32 of an alternative signal (Table 5): the G x G
    low-resolution luma image (FRAMEDIFF, G = grid) or the 64 dHash bits
    (DHASH, grid unused); the L1 distance of two rows over signal_two_m() is
    the signal's distance in [0, 1]."""
    f = np.ascontiguousarray(frames, dtype=np.uint8)
    if f.ndim == 3:
        f = f[..., None]
    n, H, W, C = f.shape
    nsig = grid * grid if kind == FRAMEDIFF else 64
    out = np.zeros((n, nsig), dtype=np.uint32)
    got = _load().orc_signature(_ptr(f), n, H, W, C, kind, grid, _ptr(out))
    if got != nsig:
        raise ValueError(f"oracle signature rejected shape {f.shape} kind={kind} grid={grid}")
    return out


def signal_two_m(kind: int, grid: int = 32) -> int:
    """2M of a signal: 255 G^2 (frame difference) or 64 (dHash)."""
    return int(_load().orc_signal_two_m(kind, grid))


def score(D: int, two_m: int) -> np.float32:
    """The novelty score of an integer distance: D / 2M rounded once to the
    nearest fp32, ties to even (Eq. 2's total variation)."""
    return np.float32(_load().orc_score(int(D), int(two_m)))


def l1(ci: np.ndarray, cj: np.ndarray) -> int:
    """Exact integer sum_b |c_i[b]-c_j[b]| = 2M * d(h_i, h_j) (Eq. 2)."""
    a = np.ascontiguousarray(ci, dtype=np.uint32)
    b = np.ascontiguousarray(cj, dtype=np.uint32)
    return int(_load().orc_l1(_ptr(a), _ptr(b), a.size))


def ngff_select(counts: np.ndarray, mass_: int, tau, L_max: int = 30, M_min: int = 4,
                seg_len: int = 0):
    """Keep rule (Eqs. 3-5 and safeguards) over histograms [n][nbins].

    ``tau`` is one float (all streams) or one per stream of ``seg_len`` frames.
    Returns (scores fp32 [n], mask uint8 [n], kept count per stream int64)."""
    c = np.ascontiguousarray(counts, dtype=np.uint32)
    n, nb = c.shape
    taus = np.atleast_1d(np.asarray(tau, dtype=np.float32))
    seg = seg_len if 0 < seg_len <= n else max(n, 1)
    nseg = (n + seg - 1) // seg if n > 0 else 0
    scores = np.zeros(n, dtype=np.float32)
    mask = np.zeros(n, dtype=np.uint8)
    kept = np.zeros(max(nseg, 1), dtype=np.int64)
    rc = _load().orc_ngff_select(_ptr(c), n, nb, mass_, _ptr(taus), taus.size, L_max, M_min,
                                 seg_len, _ptr(scores), _ptr(mask), _ptr(kept))
    assert rc == 0
    return scores, mask, kept[:nseg]


def ngff_calibrate(counts: np.ndarray, mass_: int, target: int, L_max: int = 30, M_min: int = 4,
                   seg_len: int = 0):
    """Smallest candidate threshold keeping at most ``target`` frames per stream.

    Returns (theta int64 [nseg], tau fp32 [nseg]) with tau = fl32(theta)/fl32(2M)."""
    c = np.ascontiguousarray(counts, dtype=np.uint32)
    n, nb = c.shape
    seg = seg_len if 0 < seg_len <= n else max(n, 1)
    nseg = (n + seg - 1) // seg if n > 0 else 0
    theta = np.zeros(max(nseg, 1), dtype=np.int64)
    tau = np.zeros(max(nseg, 1), dtype=np.float32)
    rc = _load().orc_ngff_calibrate(_ptr(c), n, nb, mass_, L_max, M_min, seg_len, target,
                                    _ptr(theta), _ptr(tau))
    if rc != 0:
        raise ValueError("oracle calibration needs L_max >= 1")
    return theta[:nseg], tau[:nseg]


def qer_scores(Q: np.ndarray, K: np.ndarray, frame_offsets: np.ndarray, H_q: int, H_kv: int,
               d: int, mode: int = LOGIT, scale: float = 0.0) -> np.ndarray:
    """w_f in fp64 (Eqs. 6-7).  Q [n_q][H_q][d], K [n_vis][H_kv][d], either
    float32 or bf16 bit patterns stored as uint16."""
    Q = np.ascontiguousarray(Q)
    K = np.ascontiguousarray(K)
    if Q.dtype == np.float32 and K.dtype == np.float32:
        dt = F32
    elif Q.dtype == np.uint16 and K.dtype == np.uint16:
        dt = BF16
    else:
        raise TypeError("Q and K must both be float32 or both bf16 bits (uint16)")
    n_q = Q.size // (H_q * d)
    n_vis = K.size // (H_kv * d)
    offs = np.ascontiguousarray(frame_offsets, dtype=np.int32)
    n_frames = offs.size - 1
    w = np.zeros(max(n_frames, 1), dtype=np.float64)
    rc = _load().orc_qer_scores(_ptr(Q), _ptr(K), dt, _ptr(offs), n_frames, n_q, n_vis, H_q, H_kv,
                                d, mode, float(scale), _ptr(w))
    assert rc == 0
    return w[:n_frames]


def topk(w: np.ndarray, k_top: int) -> np.ndarray:
    """S_e (Eq. 8): k best by (score desc, index asc), chronological, -1 padded."""
    a = np.ascontiguousarray(w, dtype=np.float64)
    idx = np.full(max(k_top, 1), -1, dtype=np.int32)
    rc = _load().orc_topk(_ptr(a), a.size, k_top, _ptr(idx))
    assert rc == 0
    return idx[:k_top]


def mask_compact(mask: np.ndarray, seg_len: int = 0):
    """S_c as frame indices (increasing) and per-segment starts [nseg+1]."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    n = m.size
    nseg = -(-n // seg_len) if seg_len > 0 else 1
    idx = np.full(max(n, 1), -1, dtype=np.int32)
    seg_start = np.zeros(nseg + 1, dtype=np.int32)
    total = _load().orc_mask_compact(_ptr(m), n, seg_len, _ptr(idx), _ptr(seg_start))
    return idx[:total], seg_start


def gather_frames(src: np.ndarray, frame_offsets: np.ndarray, sel: np.ndarray, capacity: int = -1):
    """Rows of the selected frames, in the order of ``sel`` (Sec. 3.3 frame
    refinement).  ``src`` is [n_rows][...] (any dtype; rows are byte blocks).
    Returns (dst [min(total, capacity)][...], out_offs int32 [k+1],
    out_rows int32 [min(total, capacity)])."""
    s = np.ascontiguousarray(src)
    n_rows = s.shape[0]
    row_bytes = s.nbytes // n_rows if n_rows else (s.itemsize * int(np.prod(s.shape[1:])))
    offs = np.ascontiguousarray(frame_offsets, dtype=np.int32)
    sel_ = np.ascontiguousarray(sel, dtype=np.int32)
    k = sel_.size
    lengths = []
    for f in sel_:
        if 0 <= f < offs.size - 1:
            lo = min(max(int(offs[f]), 0), n_rows)
            hi = max(lo, min(max(int(offs[f + 1]), 0), n_rows))
            lengths.append(hi - lo)
    total = int(sum(lengths))
    cap = total if capacity < 0 else capacity
    dst = np.zeros((max(min(total, cap), 1),) + s.shape[1:], dtype=s.dtype)
    out_offs = np.zeros(k + 1, dtype=np.int32)
    out_rows = np.full(max(min(total, cap), 1), -1, dtype=np.int32)
    got = _load().orc_gather_frames(_ptr(s), n_rows, row_bytes, _ptr(offs), offs.size - 1, _ptr(sel_), k,
                                    _ptr(dst), cap, _ptr(out_offs), _ptr(out_rows))
    assert got == total
    m = min(total, cap)
    return dst[:m], out_offs, out_rows[:m]


def ngff_scan_open(counts: np.ndarray, mass_: int, tau: float, L_max: int = 30):
    """The keep rule as frames arrive (one stream so far, no end-of-stream
    safeguards).  Returns (scores fp32 [T], mask uint8 [T], last kept r)."""
    c = np.ascontiguousarray(counts, dtype=np.uint32)
    T, nb = c.shape
    scores = np.zeros(max(T, 1), dtype=np.float32)
    mask = np.zeros(max(T, 1), dtype=np.uint8)
    r = ctypes.c_int64(0)
    _load().orc_ngff_scan_open(_ptr(c), T, nb, mass_, float(np.float32(tau)), L_max, _ptr(scores),
                               _ptr(mask), ctypes.byref(r))
    return scores[:T], mask[:T], int(r.value)


def ngff_finish(mask: np.ndarray, M_min: int = 4):
    """End-of-stream safeguards on an open mask: (mask, frames added [M_min+1] -1 padded)."""
    m = np.array(mask, dtype=np.uint8, copy=True)
    added = np.full(max(M_min, 0) + 1, -1, dtype=np.int32)
    _load().orc_ngff_finish(_ptr(m), m.size, M_min, _ptr(added))
    return m, added


def evidence_preservation(w: np.ndarray, mask: np.ndarray, p: float = 0.2):
    """(Attention Preservation Ratio, Top-Evidence Recall@p) of an NGFF mask
    against full-video QER scores w (appendix, evidence preservation)."""
    a = np.ascontiguousarray(w, dtype=np.float64)
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    apr, rec = ctypes.c_double(0), ctypes.c_double(0)
    rc = _load().orc_evidence_preservation(_ptr(a), _ptr(m), a.size, float(p), ctypes.byref(apr),
                                           ctypes.byref(rec))
    assert rc == 0
    return apr.value, rec.value


def attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float = 0.0, rows=None) -> np.ndarray:
    """Causal softmax attention in fp64 of the given query rows (default: all),
    every head: Q [L][H_q][d], K and V [L][H_kv][d] (float32, or bf16 bit
    patterns as uint16).  Returns [len(rows)][H_q][d] float64."""
    Q = np.ascontiguousarray(Q)
    K = np.ascontiguousarray(K)
    V = np.ascontiguousarray(V)
    L, H_q, d = Q.shape
    H_kv = K.shape[1]
    if not (Q.dtype == K.dtype == V.dtype) or Q.dtype not in (np.float32, np.uint16):
        raise TypeError("Q, K, V must all be float32 or all bf16 bits (uint16)")
    assert K.shape == (L, H_kv, d) and V.shape == (L, H_kv, d)
    dtype = F32 if Q.dtype == np.float32 else BF16
    r = np.arange(L, dtype=np.int32) if rows is None else np.ascontiguousarray(rows, dtype=np.int32)
    out = np.zeros((max(r.size, 1), H_q, d), dtype=np.float64)
    rc = _load().orc_attention_rows(_ptr(Q), _ptr(K), _ptr(V), dtype, L, H_q, H_kv, d, float(scale),
                                    _ptr(r), r.size, _ptr(out))
    if rc != 0:
        raise ValueError(f"orc_attention_rows failed ({rc})")
    return out[:r.size]
