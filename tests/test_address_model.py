"""Host-side address check of the kernels' index arithmetic, without a GPU.

The library's dry run (cofie_debug_dry_run) makes an entry point validate and
plan exactly as on the device, launch nothing, and walk instead every global
and LDS address of the kernels that have an address model: the QER score
kernels (LOGIT and both SOFTMAX passes, grouped-query folds, split
contractions, several key sequences), the operand-order query copy and the
sequence kernel of the multi-stream step, the frame means and their top-k
trees, the fused prefill attention (its DMA stages, fragments, text row
groups and merge), the NGFF histogram kernel's clamped unit loads and pixel
tails, the signature kernel of the alternative signals, the keep-rule
kernel's staged rows, and the frame gather.  The addresses come from the same __host__ __device__
index functions the kernels call, and each is checked against fake device
buffers of the sizes a caller passes (the inputs, the outputs and the
workspace the library asks for).

Every plan below is one the GPU parity tests or the benchmark produce: the
five workloads at full size (the multi-stream step exactly as the benchmark
launches it, all 32 sequences in one call), and the shapes of the GPU tests
(ragged tiles, tails of the contraction, query rows past 64 and 128, grouped
heads, split contractions, several rounds per workgroup, prefixes, empty
sequences).  Each must report zero violations over a nonzero number of
checked accesses; the negative controls show that a buffer one access too
short is reported."""
import numpy as np
import pytest

from paper_2609_03675_amd import binding as B
from paper_2609_03675_amd import synth

torch = pytest.importorskip("torch")

DT = {"bf16": (torch.bfloat16, B.BF16), "f32": (torch.float32, B.F32)}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    B.lib()


def clean(dr, what=""):
    v, n, msg = dr.result()
    assert v == 0, f"{what}: {v} violations, first: {msg}"
    assert n > 0, f"{what}: nothing was checked"
    return n


# ---- QER ----------------------------------------------------------------------------

def qer_single(dr, n_q, H_q, H_kv, d, tokens, dtype, k, mode=B.LOGIT, trim_k=0, noalloc=False):
    tdt, cdt = DT[dtype]
    offs = synth.frame_offsets(tokens).astype(np.int32)
    n_vis, nf = int(offs[-1]), len(tokens)
    Q = dr.buffer((n_q, H_q, d), tdt, "Q")
    K = dr.buffer((n_vis, H_kv, d), tdt, "K", trim=trim_k)
    od = dr.buffer(nf + 1, torch.int32, "frame offsets", data=offs)
    out = dr.buffer(max(nf, 1), torch.float32, "scores")
    idx = dr.buffer(max(k, 1), torch.int32, "top-k")
    if noalloc:
        B.cofie_qer_rank_noalloc(Q, K, od, k, out, idx, score_mode=mode, stream=0)
        return
    desc = B.qer_desc(n_q, n_vis, nf, H_q, H_kv, d, cdt, mode)
    ws = dr.buffer(B.qer_workspace_bytes(desc, k), torch.uint8, "workspace")
    B.cofie_qer_rank(Q, K, od, k, score_mode=mode, out_scores=out, out_idx=idx, workspace=ws, stream=0)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
@pytest.mark.parametrize("mode", [B.LOGIT, B.SOFTMAX])
def test_qer_workloads(cfg, mode):
    wl = synth.WORKLOADS[cfg]
    with B.DryRun() as dr:
        qer_single(dr, wl.n_q, wl.H_q, wl.H_kv, wl.d, [wl.tokens] * wl.n_frames, wl.qk_dtype, wl.k_top, mode)
        clean(dr, f"C{cfg} mode {mode}")


SHAPES = [(20, 4, 4, 32), (80, 2, 2, 64), (16, 8, 2, 32), (48, 28, 4, 128), (3, 1, 1, 16), (5, 3, 3, 16),
          (7, 5, 5, 16), (9, 2, 2, 48), (10, 7, 7, 16), (33, 28, 28, 128)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d", SHAPES)
def test_qer_shapes(dtype, n_q, H_q, H_kv, d):
    """The parity tests' head shapes: ragged and empty frames, contraction
    tails of 16 to 48 elements, query chunks past 64 rows, grouped heads."""
    with B.DryRun() as dr:
        for k in (0, 1, 9, 12):
            qer_single(dr, n_q, H_q, H_kv, d, [17, 0, 40, 1, 33, 64, 5, 0, 29], dtype, k)
        qer_single(dr, n_q, H_q, H_kv, d, [12, 30, 0, 7, 64, 19], dtype, 3, B.SOFTMAX)
        clean(dr, "shapes")


# SOFTMAX with grouped bf16 heads of d = 128 (one query) takes the grouped-head
# kernel: every instance, ragged rows and tiles, fewer tiles than key ranges
SOFT_GRP = [(48, 28, 4, [222] * 8 + [224]),   # the high-res heads
            (40, 28, 4, [17, 0, 40, 1, 33]),   # rows past the last full block, ragged last tile
            (1, 28, 4, [5]),                   # one row, one partial tile
            (64, 32, 4, [100] * 7),            # four row blocks
            (16, 8, 4, [16] * 33),             # 33 whole tiles: one pair short of a full last pair
            (33, 8, 2, [3001]),                # G = 4
            (5, 16, 2, [64] * 60),             # G = 8, many tiles per range
            (100, 28, 4, [160] * 9 + [77]),    # 7 row blocks: two sets of four, the last set one block short
            (70, 8, 4, [300, 1, 299])]         # G = 2: 5 row blocks in two sets


@pytest.mark.parametrize("n_q,H_q,H_kv,tokens", SOFT_GRP)
def test_softmax_grouped_heads(n_q, H_q, H_kv, tokens):
    with B.DryRun() as dr:
        for k in (0, 3):
            qer_single(dr, n_q, H_q, H_kv, 128, tokens, "bf16", k, B.SOFTMAX)
        qer_single(dr, n_q, H_q, H_kv, 128, tokens, "bf16", 3, B.SOFTMAX, noalloc=True)
        clean(dr, "grouped SOFTMAX")


def test_softmax_grouped_heads_short_keys_reported():
    with B.DryRun() as dr:
        qer_single(dr, 48, 28, 4, 128, [222] * 8 + [224], "bf16", 4, B.SOFTMAX, trim_k=16)
        v, n, msg = dr.result()
    assert v > 0 and "soft grp: keys" in msg, msg


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d,tokens", [
    (32, 28, 28, 128, [333] * 8 + [337]),   # ragged last tile
    (48, 28, 4, 128, [222] * 8 + [224]),    # seven query heads per key head
    (70, 4, 4, 64, [166] * 8 + [172]),      # two query chunks
    (16, 2, 1, 64, [7288] * 8 + [7296]),    # > 4096 tiles: several rounds per workgroup
    (1, 2, 2, 64, [1]), (17, 4, 2, 64, [0, 5, 0, 3]), (3, 1, 1, 128, [16, 16]), (2, 6, 3, 64, [300, 0, 41]),
])
def test_qer_softmax_score_kernel(dtype, n_q, H_q, H_kv, d, tokens):
    with B.DryRun() as dr:
        for k in (0, 4):
            qer_single(dr, n_q, H_q, H_kv, d, tokens, dtype, k, B.SOFTMAX)
        clean(dr, "softmax")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H,d,tokens", [
    (20, 8, 64, [97] * 99), (20, 8, 64, [100] * 81 + [3]), (32, 28, 128, [144] * 49 + [7]),
    (4, 32, 128, [10000] * 7),              # many rounds per workgroup, several query phases
])
def test_qer_split_and_rounds(dtype, n_q, H, d, tokens):
    with B.DryRun() as dr:
        qer_single(dr, n_q, H, H, d, tokens, dtype, 16)
        clean(dr, "split")


def test_qer_noalloc_static_scratch():
    """The allocation-free entry point's plans stay inside its static scratch."""
    wl = synth.WORKLOADS[2]
    with B.DryRun() as dr:
        qer_single(dr, wl.n_q, wl.H_q, wl.H_kv, wl.d, [wl.tokens] * wl.n_frames, "bf16", wl.k_top, noalloc=True)
        qer_single(dr, 20, 4, 4, 32, [17, 0, 40, 1, 33], "bf16", 3, noalloc=True)
        clean(dr, "noalloc")


def qer_batched(dr, n_queries, n_q, H_q, H_kv, d, tokens, nf, dtype, k, mode=B.LOGIT):
    tdt, cdt = DT[dtype]
    offs = synth.frame_offsets(tokens).astype(np.int32)
    n_vis, n_frames = int(offs[-1]), len(tokens)
    Q = dr.buffer((n_queries, n_q, H_q, d), tdt, "Q")
    K = dr.buffer((n_vis, H_kv, d), tdt, "K")
    od = dr.buffer(n_frames + 1, torch.int32, "frame offsets", data=offs)
    out = dr.buffer((n_queries, max(n_frames, 1)), torch.float32, "scores")
    idx = dr.buffer((n_queries, max(k, 1)), torch.int32, "top-k")
    desc = B.qer_desc(n_q, n_vis, n_frames, H_q, H_kv, d, cdt, mode)
    ws = dr.buffer(B.qer_batched_workspace_bytes(desc, n_queries, k), torch.uint8, "workspace")
    B.cofie_qer_rank_batched(Q, K, od, nf, k, score_mode=mode, out_scores=out, out_idx=idx, workspace=ws, stream=0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_queries,n_q,H_q,H_kv,d,n_frames,max_tokens", [
    (3, 16, 4, 4, 32, 40, 40), (5, 48, 2, 2, 64, 70, 40), (4, 32, 8, 2, 32, 33, 40), (6, 16, 28, 4, 128, 150, 40),
    (2, 64, 1, 1, 16, 9, 40), (1, 20, 4, 4, 32, 30, 40), (3, 16, 4, 4, 64, 40, 24), (5, 32, 28, 4, 128, 30, 60),
    (4, 32, 8, 8, 64, 48, 900), (5, 48, 28, 4, 128, 64, 24), (5, 32, 28, 28, 128, 64, 24),
    (5, 32, 8, 8, 64, 64, 300), (5, 32, 8, 8, 64, 64, 700),
])
def test_qer_batched(dtype, n_queries, n_q, H_q, H_kv, d, n_frames, max_tokens):
    """The batched tests' shapes: queries sharing the keys, each on a prefix
    of the frames (the full set, empty and random prefixes)."""
    rng = np.random.default_rng([2609, 3675, 97, n_queries, n_q, n_frames, max_tokens])
    tokens = rng.integers(0, max_tokens + 1, n_frames)
    nf = rng.integers(0, n_frames + 1, n_queries).astype(np.int32)
    nf[0] = n_frames
    with B.DryRun() as dr:
        for mode in (B.LOGIT, B.SOFTMAX) if d % 64 == 0 else (B.LOGIT,):  # several SOFTMAX queries: whole segments
            qer_batched(dr, n_queries, n_q, H_q, H_kv, d, tokens, nf, dtype, 6, mode)
        clean(dr, "batched")


def streams_call(dr, keys, frames, nq, nf, n_q, H_q, H_kv, d, dtype, k, short=""):
    tdt, cdt = DT[dtype]
    lay = B.StreamsLayout(keys, frames, nq, nf)
    nk, nfr, nQ = sum(keys), sum(frames), sum(nq)
    offs = np.concatenate([[0], np.cumsum(np.full(nfr, 1))])  # values are read on the device only
    Q = dr.buffer((nQ, n_q, H_q, d), tdt, "Q", trim=16 * (short == "Q"))
    K = dr.buffer((nk, H_kv, d), tdt, "K", trim=16 * (short == "K"))
    od = dr.buffer(nfr + 1, torch.int32, "frame offsets", data=offs.astype(np.int32), trim=4 * (short == "offs"))
    desc = B.qer_desc(n_q, nk, nfr, H_q, H_kv, d, cdt)
    ws = dr.buffer(B.qer_streams_workspace_bytes(desc, lay, k), torch.uint8, "workspace")
    out = dr.buffer((nQ, lay.max_frames), torch.float32, "scores")
    idx = dr.buffer((nQ, max(k, 1)), torch.int32, "top-k")
    B.cofie_qer_rank_streams(Q, K, od, lay, k, out_scores=out, out_idx=idx, workspace=ws, stream=0)


def multistream_layout(seed=1):
    """The multi-stream step's layout: per stream the calibrated number of
    candidates (frame 0 and a seeded draw of the rest), its queries'
    timestamps and prefixes, 144 keys per candidate."""
    wl = synth.WORKLOADS[5]
    rng = np.random.default_rng([2609, 3675, 98, seed])
    keys, frames, nq, nf = [], [], [], []
    for s in range(wl.n_streams):
        kept = np.sort(np.concatenate([[0], rng.choice(np.arange(1, wl.T), wl.target - 1, replace=False)]))
        stamps = synth.multistream_queries(5, s)
        cand = kept[kept <= stamps.max()]
        keys.append(cand.size * wl.tokens)
        frames.append(cand.size)
        nq.append(len(stamps))
        nf += [int((kept <= t).sum()) for t in stamps]
    return keys, frames, nq, nf


def test_multistream_step():
    """The benchmark's QER step: 32 sequences, 128 queries, one launch of the
    sequence kernel (after the operand-order query copy) and the frame means."""
    wl = synth.WORKLOADS[5]
    with B.DryRun() as dr:
        for seed in (1, 2):
            streams_call(dr, *multistream_layout(seed), wl.n_q, wl.H_q, wl.H_kv, wl.d, "bf16", wl.k_top)
        n = clean(dr, "multistream")
    assert n > 10_000_000  # every key tile of every round was walked


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d,streams", [
    (32, 4, 4, 64, [(12, 4), (0, 2), (7, 0), (20, 3), (1, 1)]),
    (16, 2, 2, 64, [(30, 9), (5, 1)]),
    (48, 4, 4, 32, [(25, 3), (9, 2)]),
    (32, 8, 2, 64, [(18, 3), (6, 2), (11, 1)]),
    (16, 28, 28, 128, [(40, 4), (3, 4), (60, 2)]),
])
def test_streams_shapes(dtype, n_q, H_q, H_kv, d, streams):
    """The streams tests' layouts: empty sequences, sequences without
    queries, chunks of several 128-row pieces, 96-row chunks, grouped heads."""
    rng = np.random.default_rng([2609, 3675, 99, n_q, len(streams)])
    keys, frames, nq, nf = [], [], [], []
    for nfr, q in streams:
        keys.append(int(rng.integers(0, 41, nfr).sum()))
        frames.append(nfr)
        nq.append(q)
        p = rng.integers(0, nfr + 1, q)
        if q:
            p[0] = nfr
        nf += p.tolist()
    with B.DryRun() as dr:
        for k in (0, 3, 50):
            streams_call(dr, keys, frames, nq, nf, n_q, H_q, H_kv, d, dtype, k)
        clean(dr, "streams")


@pytest.mark.parametrize("frames", [33288, 33289])
def test_streams_keys_near_int32_offsets(frames):
    """A sequence whose keys reach the 32-bit 16-byte offsets of the sequence
    kernel (2^31 units = 4 793 490.3 rows of 7168 bytes): 33 288 frames of
    144 keys stay below, the sequence kernel runs with every offset inside
    its sequence; 33 289 frames pass it, the call takes the general score
    kernel (64-bit offsets).  Both walk clean."""
    tokens = 144
    nk = frames * tokens
    with B.DryRun() as dr:
        streams_call(dr, [nk, 2880], [frames, 20], [4, 4], [frames, frames // 2, 7, frames, 20, 10, 1, 0],
                     32, 28, 28, 128, "bf16", 16)
        clean(dr, "keys near 2^31 units")


@pytest.mark.parametrize("short", ["K", "Q", "offs"])
def test_short_buffers_are_reported(short):
    """Negative control: the same multi-stream step with one buffer 16 (4)
    bytes short of its size reports a violation."""
    wl = synth.WORKLOADS[5]
    with B.DryRun() as dr:
        streams_call(dr, *multistream_layout(), wl.n_q, wl.H_q, wl.H_kv, wl.d, "bf16", wl.k_top, short=short)
        v, n, msg = dr.result()
    assert v > 0 and msg, short


def test_short_keys_reported_in_score_kernel():
    with B.DryRun() as dr:
        qer_single(dr, 33, 28, 28, 128, [17, 0, 40, 1, 33, 64, 5, 0, 29], "bf16", 4, trim_k=16)
        v, _, msg = dr.result()
    assert v > 0 and "score: key" in msg, msg


# ---- fused attention -------------------------------------------------------------------

def attn_call(dr, n_pre, n_vis, n_post, H_q, H_kv, n_frames, k=4, trim_v=0):
    L = n_pre + n_vis + n_post
    Q = dr.buffer((L, H_q, 128), torch.bfloat16, "Q")
    K = dr.buffer((L, H_kv, 128), torch.bfloat16, "K")
    V = dr.buffer((L, H_kv, 128), torch.bfloat16, "V", trim=trim_v)
    offs = np.linspace(0, n_vis, n_frames + 1).astype(np.int32)
    od = dr.buffer(n_frames + 1, torch.int32, "frame offsets", data=offs)
    out = dr.buffer((L, H_q, 128), torch.bfloat16, "out")
    w = dr.buffer(max(n_frames, 1), torch.float32, "scores")
    idx = dr.buffer(max(k, 1), torch.int32, "top-k")
    ws = dr.buffer(B.attn_qer_workspace_bytes(B.attn_desc(L, H_q, H_kv, 128, n_pre, n_pre + n_vis, n_frames)),
                   torch.uint8, "workspace")
    B.cofie_attn_qer(Q, K, V, od, n_pre, n_pre + n_vis, k, out=out, out_scores=w, out_idx=idx, workspace=ws,
                     stream=0)


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_attention_workloads(cfg):
    """The last-layer prefill of the 1 fps, hour and high-res workloads."""
    wl = synth.WORKLOADS[cfg]
    L, vb, ve = synth.attn_layout(cfg)
    with B.DryRun() as dr:
        attn_call(dr, vb, ve - vb, L - ve, wl.H_q, wl.H_kv, wl.n_frames, wl.k_top)
        clean(dr, f"attention C{cfg}")


@pytest.mark.parametrize("n_pre,n_vis,n_post,H_q,H_kv,n_frames", [
    (5, 30, 5, 2, 2, 3), (7, 650, 43, 4, 2, 9), (0, 536, 64, 3, 1, 5), (64, 300, 0, 2, 1, 4), (0, 1000, 1, 2, 2, 7),
    (3, 256, 2, 1, 1, 1), (1, 1, 1, 2, 2, 1), (40, 100, 40, 2, 2, 3), (100, 700, 100, 4, 2, 9),
    (0, 300, 300, 2, 1, 4), (129, 520, 0, 2, 2, 5), (20, 0, 0, 2, 2, 3),
])
def test_attention_shapes(n_pre, n_vis, n_post, H_q, H_kv, n_frames):
    """The attention parity tests' shapes (ragged blocks and chunks, text
    rows before and after the video, several row groups, no visual token)."""
    with B.DryRun() as dr:
        attn_call(dr, n_pre, n_vis, n_post, H_q, H_kv, n_frames)
        clean(dr, "attention shapes")


def test_attention_short_values_reported():
    with B.DryRun() as dr:
        attn_call(dr, 7, 650, 43, 4, 2, 9, trim_v=16)
        v, _, msg = dr.result()
    assert v > 0 and "V" in msg, msg


# ---- NGFF ---------------------------------------------------------------------------

def ngff_filter(dr, n, H, W, C, mode, bins, misalign=0, trim=0, seg=0):
    frames = dr.buffer((n, H, W, C), torch.uint8, "frames", misalign=misalign, trim=trim)
    rule = B.keep_rule(mode, 0.3, 30, 4, seg)
    ws = dr.buffer(max(B.ngff_workspace_bytes(n, H, W, C, bins, rule), 1), torch.uint8, "workspace")
    rule = B.keep_rule(mode, 0.3, 30, 4, seg, workspace=ws)
    scores = dr.buffer(max(n, 1), torch.float32, "scores")
    mask = dr.buffer(max(n, 1), torch.uint8, "mask")
    B.cofie_ngff_filter(frames, bins, rule, out_scores=scores, out_mask=mask, stream=0)
    hist = dr.buffer((n, B.cofie_ngff_nbins(mode, bins)), torch.int32, "histograms")
    B.cofie_ngff_histogram(frames, bins, mode, out=hist, stream=0)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_ngff_workloads(cfg):
    wl = synth.WORKLOADS[cfg]
    mode = {"per_channel": "per_channel", "joint3d": "joint3d", "gray": "gray"}[wl.hist_mode]
    with B.DryRun() as dr:
        ngff_filter(dr, wl.n, wl.H, wl.W, 3, mode, wl.bins, seg=wl.T if wl.n_streams > 1 else 0)
        clean(dr, f"NGFF C{cfg}")


RGB_SHAPES = [(3, 64, 64, 3), (2, 40, 40, 3), (3, 37, 53, 3), (5, 448, 448, 3), (1, 1, 1, 3), (2, 2160, 3840, 3),
              (2, 1464, 1920, 3)]
ONE_CHANNEL_SHAPES = [(4, 64, 64, 1), (3, 37, 53, 1), (2, 448, 448, 1)]
MODES = [("per_channel", 32), ("per_channel", 2), ("per_channel", 64), ("joint3d", 8), ("joint3d", 16), ("gray", 32),
         ("gray", 256)]


# one-channel frames take the gray mode only
@pytest.mark.parametrize("shape,mode,bins", [(s, m, b) for s in RGB_SHAPES for m, b in MODES] +
                         [(s, m, b) for s in ONE_CHANNEL_SHAPES for m, b in MODES if m == "gray"])
def test_ngff_shapes(shape, mode, bins):
    n, H, W, C = shape
    with B.DryRun() as dr:
        ngff_filter(dr, n, H, W, C, mode, bins)
        ngff_filter(dr, n, H, W, C, mode, bins, misalign=1)  # byte path of a frame at an odd address
        clean(dr, "NGFF shapes")


@pytest.mark.parametrize("name", ["framediff", "dhash"])
@pytest.mark.parametrize("shape,G", [((5, 33, 47, 3), 4), ((3, 64, 64, 1), 16), ((2, 90, 160, 3), 32),
                                     ((3, 37, 29, 3), 2), ((2, 64, 64, 3), 64), ((4, 448, 448, 3), 32),
                                     ((2, 1080, 1920, 3), 32), ((200, 448, 448, 3), 32)])
def test_signal_shapes(name, shape, G):
    """The alternative signals (Table 5) with the signal tests' shapes: the
    signature kernel's vector and byte paths (W not a multiple of 4, a frame
    at an odd address), then the keep rule on their rows."""
    n, H, W, C = shape
    if name == "dhash" and (H < 8 or W < 9):
        pytest.skip("dHash needs an 8 x 9 grid")
    with B.DryRun() as dr:
        ngff_filter(dr, n, H, W, C, name, G)
        ngff_filter(dr, n, H, W, C, name, G, misalign=1)
        ngff_filter(dr, n, H, W, C, name, G, seg=100 if n >= 200 else 0)
        clean(dr, "signals")


def test_ngff_million_frames():
    """2^20 small frames in streams of 4096: frame and histogram offsets past
    2^31 bytes, 256 streams of keep words."""
    with B.DryRun() as dr:
        ngff_filter(dr, 1 << 20, 40, 48, 3, "per_channel", 32, seg=4096)
        clean(dr, "a million frames")


def test_short_frames_reported():
    with B.DryRun() as dr:
        ngff_filter(dr, 5, 448, 448, 3, "per_channel", 32, trim=1)
        v, _, msg = dr.result()
    assert v > 0 and "hist" in msg, msg


# ---- frame gather -------------------------------------------------------------------

def gather(dr, src_rows, row_bytes, offs, sel, capacity, misalign=0, dst_trim=0):
    src = dr.buffer((src_rows, row_bytes), torch.uint8, "src", misalign=misalign)
    od = dr.buffer(offs.size, torch.int32, "frame offsets", data=offs.astype(np.int32))
    sd = dr.buffer(sel.size, torch.int32, "sel", data=sel.astype(np.int32))
    dst = dr.buffer((max(capacity, 1), row_bytes), torch.uint8, "dst", trim=dst_trim)
    oo = dr.buffer(sel.size + 1, torch.int32, "out offsets")
    rows = dr.buffer(max(capacity, 1), torch.int32, "out rows")
    B.cofie_gather_frames(src, od, sd, dst=dst, capacity=capacity, out_offsets=oo, out_rows=rows, stream=0)


@pytest.mark.parametrize("row_bytes", [7, 30, 4, 7168])
def test_gather_frames(row_bytes):
    """The gather tests' cases: repeated and invalid entries, capacities
    below, at and above the rows; byte, 4-byte and 16-byte lanes."""
    rng = np.random.default_rng([2609, 3675, 100, row_bytes])
    sizes = rng.integers(0, 9, 60)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    sel = np.sort(rng.choice(60, 20, replace=False))
    sel = np.concatenate([sel, [sel[0], -1, 60, -7]])
    with B.DryRun() as dr:
        for cap in (int(offs[-1]), 0, 9, 3 * int(offs[-1])):
            gather(dr, int(offs[-1]), row_bytes, offs, sel, cap)
        gather(dr, int(offs[-1]), row_bytes, offs, sel, int(offs[-1]), misalign=1)
        clean(dr, "gather")


@pytest.mark.parametrize("k", [4096, 5000])
def test_gather_many_frames(k):
    """One-kernel gather (<= 4096 frames) and the offsets kernel first."""
    rng = np.random.default_rng([2609, 3675, 92, k])
    sizes = rng.integers(0, 4, 6000)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    sel = np.sort(rng.choice(6000, k, replace=False))
    with B.DryRun() as dr:
        for cap in (int(offs[-1]), int(offs[-1]) // 3):
            gather(dr, int(offs[-1]), 16, offs, sel, cap)
        clean(dr, "gather many")


def test_gather_malformed_offsets_and_short_dst():
    offs = np.array([-5, 3, 2, 60, 7, 7, 40])
    sel = np.array([0, 1, 2, 3, 5, -1])
    with B.DryRun() as dr:
        gather(dr, 40, 6, offs, sel, 40)
        clean(dr, "malformed")
    with B.DryRun() as dr:
        gather(dr, 40, 6, offs, sel, 40, dst_trim=1)
        v, _, msg = dr.result()
    assert v > 0 and "gather: destination" in msg, msg


def test_gather_offsets_saturate_past_int32():
    """A selection that repeats a frame until its running row count passes
    2^31 (5000 entries of a 2^20-row frame: the offsets kernel path): every
    copy stays inside dst, because the stored offsets saturate at 2^31 - 1
    and the frames placed past the capacity are skipped (int32 offsets that
    wrapped would have placed them before dst)."""
    rows = 1 << 20
    offs = np.array([0, rows])
    sel = np.zeros(5000, np.int32)
    with B.DryRun() as dr:
        gather(dr, rows, 16, offs, sel, (1 << 31) - 1)
        clean(dr, "saturated offsets")


def test_gather_capacity_beyond_int32_refused():
    with B.DryRun() as dr:
        with pytest.raises(B.CofieError):
            gather(dr, 4, 16, np.array([0, 4]), np.array([0]), 1 << 31)


def test_dry_run_allocates_nothing():
    """A dry run makes no HIP call: a call that would allocate its scratch is
    refused (a workspace must be given), the online filter (device state) is
    refused, and the dry run ends cleanly."""
    with B.DryRun() as dr:
        Q = dr.buffer((16, 2, 32), torch.bfloat16, "Q")
        K = dr.buffer((64, 2, 32), torch.bfloat16, "K")
        od = dr.buffer(5, torch.int32, "frame offsets", data=np.arange(0, 80, 16, dtype=np.int32))
        out = dr.buffer(4, torch.float32, "scores")
        idx = dr.buffer(2, torch.int32, "top-k")
        with pytest.raises(B.CofieError) as e:
            B.cofie_qer_rank(Q, K, od, 2, out_scores=out, out_idx=idx, stream=0)
        assert e.value.code == B.COFIE_EINVAL and "workspace" in str(e.value)
        with pytest.raises(B.CofieError) as e:
            B.cofie_ngff_stream_create(2, 16, 16, 3, 32, B.keep_rule("per_channel"))
        assert e.value.code == B.COFIE_EUNSUPPORTED
    # outside the dry run the refusals are gone (no GPU here: the sizing call works)
    assert B.qer_workspace_bytes(B.qer_desc(16, 64, 4, 2, 2, 32), 2) > 0

