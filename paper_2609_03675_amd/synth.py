"""Seeded synthetic video streams and query/key tensors.

This module is the only code that the HIP path and the CPU oracle share: it
draws inputs and holds none of the method's arithmetic (no histogram, no
distance, no score).  Every buffer is a pure function of
``numpy.random.default_rng([2609, 3675, config, stream, purpose, ...])``.

The paper evaluates on public streaming/offline video benchmarks that are not
available here; these streams stand in for them, shaped like the five
workloads the library is measured on:

1. tiny: 64 RGB frames of 64x64, six piecewise-constant colour scenes with
   five distinct random cut points, uniform integer noise in [-8, 8].
2. 1 fps stream: 256 frames of 448x448, scene cuts as a discrete Poisson
   process (a cut before frame t with probability 1/12), scene colour uniform,
   Gaussian noise sigma 10 rounded half-to-even.
3. hour-long stream: 3600 frames of 448x448, mean cut gap 30, plus one-frame
   "flash" events (probability 0.02, a random solid colour, no noise).
4. high-res: 1024 frames of 1920x1080, mean cut gap 20, a global brightness
   random walk of +/-1 per frame added to every channel, noise sigma 10.
5. multi-stream: 32 independent streams of 512 frames of 448x448, each with
   its own mean cut gap drawn uniformly from [5, 40].

Per-pixel noise is read from a per-stream pool of pre-drawn noise values at a
random pixel-aligned window per frame, so that gigabyte streams are generated
at memory speed: every pixel's noise is a draw of the stated distribution,
and consecutive frames see different windows of the pool.

Query/key tensors are N(0, 1), fp32 for the tiny workload and bf16 (fp32 draws
rounded to nearest-even) otherwise; bf16 tensors are carried as their uint16
bit patterns, which are the input of record.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

SEED0 = (2609, 3675)
PURPOSE_FRAMES, PURPOSE_QK, PURPOSE_TIMESTAMPS, PURPOSE_NOISE, PURPOSE_QUERY, PURPOSE_ATTN = 0, 1, 2, 3, 4, 5
_POOL_WINDOWS = 65536


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    n_streams: int
    T: int                  # frames per stream
    H: int
    W: int
    bins: int               # per channel (per axis for the joint histogram)
    hist_mode: str          # "per_channel" | "joint3d" | "gray"
    retain: float           # retention ratio the keep threshold is calibrated for
    cut_gap: Optional[float]  # mean cut gap (None: fixed number of cuts)
    n_cuts: int = 0
    noise: str = "gauss10"  # "gauss10" | "uniform8"
    flash_p: float = 0.0
    drift: bool = False
    gap_range: Optional[tuple] = None  # per-stream mean gap ~ U(lo, hi)
    # QER shape
    qk_dtype: str = "bf16"  # "f32" | "bf16"
    n_q: int = 32
    H_q: int = 28
    H_kv: int = 28
    d: int = 128
    n_frames: int = 128     # candidate frames (C5: per query, from the NGFF mask)
    tokens: int = 256       # visual tokens per frame
    k_top: int = 16
    queries_per_stream: int = 0

    @property
    def frame_bytes(self) -> int:
        return self.H * self.W * 3

    @property
    def n(self) -> int:
        return self.n_streams * self.T

    @property
    def target(self) -> int:
        """Kept frames per stream the threshold is calibrated for: max(1, round(rho*T))."""
        return max(1, int(round(self.retain * self.T)))


WORKLOADS = {
    1: Workload(1, "tiny", 1, 64, 64, 64, 16, "per_channel", 0.40, None, n_cuts=5,
                noise="uniform8", qk_dtype="f32", n_q=8, H_q=4, H_kv=4, d=32, n_frames=32,
                tokens=16, k_top=8),
    2: Workload(2, "1fps_stream", 1, 256, 448, 448, 32, "per_channel", 0.50, 12.0,
                n_q=32, H_q=28, H_kv=28, d=128, n_frames=128, tokens=256, k_top=16),
    3: Workload(3, "hour_stream", 1, 3600, 448, 448, 32, "per_channel", 0.20, 30.0,
                flash_p=0.02, n_q=64, H_q=28, H_kv=28, d=128, n_frames=720, tokens=64,
                k_top=32),
    4: Workload(4, "highres", 1, 1024, 1080, 1920, 8, "joint3d", 0.30, 20.0, drift=True,
                n_q=48, H_q=28, H_kv=4, d=128, n_frames=300, tokens=196, k_top=24),
    5: Workload(5, "multistream", 32, 512, 448, 448, 32, "per_channel", 0.25, None,
                gap_range=(5.0, 40.0), n_q=32, H_q=28, H_kv=28, d=128, n_frames=0,
                tokens=144, k_top=16, queries_per_stream=4),
}


def _gen_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def rng(cfg: int, stream: int, purpose: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng([*SEED0, cfg, stream, purpose, *extra])


class StreamPlan:
    """Per-frame scene colour, flash, brightness offset and noise window of one stream."""

    def __init__(self, cfg: int, stream: int = 0):
        wl = WORKLOADS[cfg]
        self.wl = wl
        T = wl.T
        r = rng(cfg, stream, PURPOSE_FRAMES)
        if wl.gap_range is not None:
            gap = float(r.uniform(*wl.gap_range))
        else:
            gap = wl.cut_gap
        self.mean_gap = gap
        if gap is None:
            cuts = np.sort(r.choice(np.arange(1, T), size=wl.n_cuts, replace=False))
            scene = np.searchsorted(cuts, np.arange(T), side="right")
        else:
            cut = r.random(T) < 1.0 / gap
            cut[0] = False
            scene = np.cumsum(cut)
        self.scene = scene.astype(np.int64)
        n_scenes = int(self.scene[-1]) + 1
        self.colours = r.integers(0, 256, size=(n_scenes, 3))
        if wl.flash_p > 0:
            self.flash = r.random(T) < wl.flash_p
            self.flash_colour = r.integers(0, 256, size=(T, 3))
        else:
            self.flash = np.zeros(T, dtype=bool)
            self.flash_colour = np.zeros((T, 3), dtype=np.int64)
        if wl.drift:
            steps = r.choice(np.array([-1, 1]), size=T)
            steps[0] = 0
            self.brightness = np.cumsum(steps)
        else:
            self.brightness = np.zeros(T, dtype=np.int64)
        self.window = r.integers(0, _POOL_WINDOWS, size=T) * 3
        nr = rng(cfg, stream, PURPOSE_NOISE)
        F = wl.frame_bytes
        P = F + 3 * _POOL_WINDOWS
        if wl.noise == "gauss10":
            v = np.rint(nr.standard_normal(P, dtype=np.float32) * np.float32(10.0))
            v = np.clip(v, -128, 127).astype(np.int32)
        else:
            v = nr.integers(-8, 9, size=P).astype(np.int32)
        chan = np.arange(P, dtype=np.int64) % 3
        # pool entry = index into a per-frame 768-entry lookup: channel*256 + (noise+128)
        self.pool = ((v + 128) + 256 * chan).astype(np.uint16)

    def _lut(self, t: int) -> np.ndarray:
        u = np.arange(256, dtype=np.int64) - 128
        base = self.colours[self.scene[t]] + self.brightness[t]
        lut = np.empty(768, dtype=np.uint8)
        for c in range(3):
            lut[c * 256:(c + 1) * 256] = np.clip(base[c] + u, 0, 255)
        return lut

    def frames(self, start: int = 0, count: Optional[int] = None,
               out: Optional[np.ndarray] = None) -> np.ndarray:
        """uint8 frames [count][H][W][3] for frame indices start .. start+count-1."""
        wl = self.wl
        if count is None:
            count = wl.T - start
        F = wl.frame_bytes
        if out is None:
            out = np.empty((count, wl.H, wl.W, 3), dtype=np.uint8)
        flat = out.reshape(count, F)

        def one(i: int) -> None:
            t = start + i
            if self.flash[t]:
                flat[i].reshape(-1, 3)[:] = self.flash_colour[t].astype(np.uint8)
            else:
                o = int(self.window[t])
                np.take(self._lut(t), self.pool[o:o + F], out=flat[i])

        if count * F < (64 << 20):
            for i in range(count):
                one(i)
        else:  # np.take releases the GIL: fill frames on a few threads
            with ThreadPoolExecutor(_gen_threads()) as ex:
                list(ex.map(one, range(count)))
        return out


def frames(cfg: int, stream: int = 0, start: int = 0, count: Optional[int] = None) -> np.ndarray:
    return StreamPlan(cfg, stream).frames(start, count)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if not np.all(np.isfinite(x)):
        raise ValueError("bf16_bits expects finite values")
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal(r: np.random.Generator, shape, dtype: str) -> np.ndarray:
    x = r.standard_normal(shape, dtype=np.float32)
    return x if dtype == "f32" else bf16_bits(x)


def frame_offsets(tokens_per_frame) -> np.ndarray:
    """CSR offsets [n_frames+1] (int32) from per-frame visual-token counts."""
    t = np.asarray(tokens_per_frame, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(t)]).astype(np.int32)


def qer_inputs(cfg: int, stream: int = 0):
    """(Q [n_q][H_q][d], K [n_frames*tokens][H_kv][d], frame_offsets) for workloads 1-4."""
    wl = WORKLOADS[cfg]
    r = rng(cfg, stream, PURPOSE_QK)
    Q = _normal(r, (wl.n_q, wl.H_q, wl.d), wl.qk_dtype)
    K = _normal(r, (wl.n_frames * wl.tokens, wl.H_kv, wl.d), wl.qk_dtype)
    offs = frame_offsets(np.full(wl.n_frames, wl.tokens))
    return Q, K, offs


def attn_layout(cfg: int):
    """(L, vis_begin, vis_end) of the last-layer prefill sequence of workloads
    1-4: a quarter of the text tokens (a system prompt) before the candidate
    frames' visual tokens, the rest (the question) after them."""
    wl = WORKLOADS[cfg]
    n_vis = wl.n_frames * wl.tokens
    n_pre = wl.n_q // 4
    return wl.n_q + n_vis, n_pre, n_pre + n_vis


def attn_inputs(cfg: int):
    """bf16 Q [L][H_q][d], K and V [L][H_kv][d] of the whole prefill sequence
    (standard normal, rounded to bf16) and the visual frames' offsets."""
    wl = WORKLOADS[cfg]
    L, _, _ = attn_layout(cfg)
    r = rng(cfg, 0, PURPOSE_ATTN)
    Q = _normal(r, (L, wl.H_q, wl.d), "bf16")
    K = _normal(r, (L, wl.H_kv, wl.d), "bf16")
    V = _normal(r, (L, wl.H_kv, wl.d), "bf16")
    return Q, K, V, frame_offsets(np.full(wl.n_frames, wl.tokens))


def multistream_queries(cfg: int, stream: int):
    """Query timestamps (frame indices in [0, T)) of one stream of workload 5."""
    wl = WORKLOADS[cfg]
    r = rng(cfg, stream, PURPOSE_TIMESTAMPS)
    return np.sort(r.integers(0, wl.T, size=wl.queries_per_stream))


def multistream_q(cfg: int, stream: int, query: int) -> np.ndarray:
    wl = WORKLOADS[cfg]
    return _normal(rng(cfg, stream, PURPOSE_QUERY, query), (wl.n_q, wl.H_q, wl.d), wl.qk_dtype)


def multistream_k(cfg: int, stream: int, frame_ids) -> np.ndarray:
    """Visual keys of the given frames of one stream, concatenated in order
    ([len(frame_ids)*tokens][H_kv][d]); frame f's keys depend only on (stream, f)."""
    wl = WORKLOADS[cfg]
    blocks = [_normal(rng(cfg, stream, PURPOSE_QK, int(f)), (wl.tokens, wl.H_kv, wl.d), wl.qk_dtype)
              for f in frame_ids]
    if not blocks:
        shape = (0, wl.H_kv, wl.d)
        return np.zeros(shape, dtype=np.float32 if wl.qk_dtype == "f32" else np.uint16)
    return np.concatenate(blocks, axis=0)


def random_qk(seed: int, n_q: int, n_vis: int, H_q: int, H_kv: int, d: int, dtype: str = "bf16"):
    """Free-shape N(0,1) Q/K for edge-case tests."""
    r = np.random.default_rng([*SEED0, 99, seed])
    return _normal(r, (n_q, H_q, d), dtype), _normal(r, (n_vis, H_kv, d), dtype)


def random_frames(seed: int, n: int, H: int, W: int, C: int = 3, scenes: int = 4) -> np.ndarray:
    """Free-shape piecewise-constant noisy frames for edge-case tests."""
    r = np.random.default_rng([*SEED0, 98, seed])
    sid = np.sort(r.integers(0, scenes, size=n))
    col = r.integers(0, 256, size=(scenes, C))
    base = col[sid][:, None, None, :]
    noise = r.integers(-12, 13, size=(n, H, W, C))
    return np.clip(base + noise, 0, 255).astype(np.uint8)
