"""GPU parity of QER (Sec. 3.3, Eqs. 6-8) against the fp64 CPU oracle through
the C ABI.  Frame scores within 1e-5 relative (fp32 inputs) or 2e-2 relative
(bf16 MFMA path); top-k index sets identical except inside a group of
reference scores tied within 1e-6."""
import numpy as np
import pytest

import oracle
from paper_2609_03675_amd import binding as B
from paper_2609_03675_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import BF16_REGRESSION, check_topk, qk_dev, rel_err, require_gpu, to_dev  # noqa: E402

TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    B.lib()


def run_case(Q, K, offs, H_q, H_kv, d, k_top, mode=B.LOGIT, scale=0.0, dtype="bf16", regression=False):
    print(f"qer n_q={Q.shape[0]} n_vis={K.shape[0]} frames={len(offs)-1} H={H_q}/{H_kv} d={d} "
          f"k={k_top} mode={mode} {dtype}", flush=True)
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs.astype(np.int32)), k_top,
                              score_mode=mode, scale=scale)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    idx = idx.cpu().numpy()
    ref = oracle.qer_scores(Q, K, offs, H_q, H_kv, d, mode, scale)
    err = rel_err(w, ref)
    print(f"  max rel err {err:.3e}", flush=True)
    assert err <= TOL[dtype], err
    if regression and dtype == "bf16":  # scores well away from zero (workload shapes)
        assert err <= BF16_REGRESSION, err
    assert np.array_equal(np.isneginf(w), np.isneginf(ref)), "empty-frame scores differ"
    check_topk(idx, ref, k_top)
    return w, idx, ref


@pytest.mark.parametrize("cfg", [1, 2])
def test_workload_scores_and_topk(cfg):
    wl = synth.WORKLOADS[cfg]
    Q, K, offs = synth.qer_inputs(cfg)
    run_case(Q, K, offs, wl.H_q, wl.H_kv, wl.d, wl.k_top, dtype=wl.qk_dtype, regression=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d", [(20, 4, 4, 32),     # query rows not a multiple of 16
                                            (80, 2, 2, 64),     # two query chunks (> 64 rows)
                                            (16, 8, 2, 32),     # GQA fold
                                            (48, 28, 4, 128),   # GQA, high-res workload heads
                                            (3, 1, 1, 16),      # single head, d = 16
                                            (5, 3, 3, 16),      # contraction 48: tail only
                                            (7, 5, 5, 16),      # 80: one segment + 16 tail
                                            (9, 2, 2, 48),      # 96: one segment + 32 tail
                                            (10, 7, 7, 16),     # 112: one segment + 48 tail
                                            (33, 28, 28, 128)]) # long contraction (k-split)
def test_shapes(dtype, n_q, H_q, H_kv, d):
    tokens = [17, 0, 40, 1, 33, 64, 5, 0, 29]
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(n_q * 7 + d, n_q, int(offs[-1]), H_q, H_kv, d, dtype)
    for k in (0, 1, 4, 9, 12):
        run_case(Q, K, offs, H_q, H_kv, d, k, dtype=dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d", [(8, 4, 4, 32), (40, 4, 2, 16), (70, 2, 2, 32)])
def test_softmax_mode(dtype, n_q, H_q, H_kv, d):
    offs = synth.frame_offsets([12, 30, 0, 7, 64, 19])
    Q, K = synth.random_qk(n_q + 3 * d, n_q, int(offs[-1]), H_q, H_kv, d, dtype)
    run_case(Q, K, offs, H_q, H_kv, d, 3, mode=B.SOFTMAX, dtype=dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d,n_tok", [
    (32, 28, 28, 128, 3001),   # the 1 fps stream's heads, ragged last tile
    (48, 28, 4, 128, 2000),    # the high-res heads (bf16: the grouped-head kernel)
    (48, 12, 4, 128, 2000),    # three query heads per key head: no grouped-head instance
    (70, 4, 4, 64, 1500),      # two query chunks (> 64 rows)
    (16, 2, 1, 64, 65600),     # > 4096 tiles: two rounds in some workgroups, one in others
])
def test_softmax_through_score_kernel(dtype, n_q, H_q, H_kv, d, n_tok):
    """SOFTMAX mode where every head is whole 128-byte segments of a key row:
    both passes run in the LDS-staged score kernel (per-head statistics per
    wave, merged, then the head mean of the probabilities), or, for bf16
    grouped heads of d = 128 with an instance, in the grouped-head kernel."""
    per = max(1, n_tok // 9)
    tokens = [per] * 8 + [n_tok - 8 * per]
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(n_q * 31 + H_q + n_tok, n_q, int(offs[-1]), H_q, H_kv, d, dtype)
    w, idx, ref = run_case(Q, K, offs, H_q, H_kv, d, 4, mode=B.SOFTMAX, dtype=dtype)
    w2, idx2 = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs.astype(np.int32)), 4, score_mode=B.SOFTMAX)
    torch.cuda.synchronize()
    assert np.array_equal(w, w2.cpu().numpy()), "SOFTMAX scores differ between two calls"


@pytest.mark.parametrize("n_q,H_q,H_kv,tokens", [
    (48, 28, 4, [222] * 8 + [224]),    # the high-res heads
    (40, 28, 4, [17, 0, 40, 1, 33]),   # rows past the last full block, ragged last tile
    (1, 28, 4, [5]),                   # one row, one partial tile
    (64, 32, 4, [100] * 7),            # four row blocks
    (16, 8, 4, [16] * 33),             # 33 whole tiles
    (33, 8, 2, [3001]),                # G = 4
    (5, 16, 2, [64] * 60),             # G = 8
    (48, 28, 4, [196] * 60),           # several pairs per wave
    (100, 28, 4, [160] * 9 + [77]),    # 7 row blocks: pass 1 in two sets of four, the last one block short
    (70, 8, 4, [300, 1, 299]),         # G = 2: 5 row blocks in two sets
])
def test_softmax_grouped_heads(n_q, H_q, H_kv, tokens):
    """SOFTMAX with bf16 grouped heads of d = 128 through the grouped-head
    kernel (per-head statistics per lane over its own keys, merged over lanes,
    waves and key ranges; then the head mean of the probabilities and its max
    over the rows): every instance, ragged rows and tiles, fewer tiles than key
    ranges.  Scores within the bf16 regression bound (the products are exact
    bf16 values, accumulated in fp32), and two calls bit-identical."""
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(n_q * 37 + H_q + len(tokens), n_q, int(offs[-1]), H_q, H_kv, 128, "bf16")
    for k in (0, 4):
        w, idx, ref = run_case(Q, K, offs, H_q, H_kv, 128, k, mode=B.SOFTMAX, regression=True)
    w2, idx2 = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs.astype(np.int32)), 4, score_mode=B.SOFTMAX)
    torch.cuda.synchronize()
    assert np.array_equal(w, w2.cpu().numpy()), "SOFTMAX scores differ between two calls"


@pytest.mark.parametrize("n_q,H_q,H_kv", [(48, 28, 4), (33, 8, 2), (20, 12, 4)])
@pytest.mark.parametrize("rising", [True, False])
def test_softmax_scores_of_very_different_scale(n_q, H_q, H_kv, rising):
    """Key rows scaled by powers of two that grow (or shrink) along the
    sequence, up to 2^6: a row's scores later in the keys exceed the running
    maximum by far more than 2^64 allows (grouped-head kernel: the pair is
    summed again against its own max and the earlier sum rescaled), or fall
    far below it (their exponentials underflow).  The scaling is exact in
    bf16, so the oracle sees the same inputs; the (48, 28, 4) and (33, 8, 2)
    shapes take the grouped-head kernel, (20, 12, 4) the score kernel."""
    tokens = [64] * 24 + [37]
    offs = synth.frame_offsets(tokens)
    n_vis = int(offs[-1])
    Q, K = synth.random_qk(n_q * 41 + H_q, n_q, n_vis, H_q, H_kv, 128, "bf16")
    e = np.floor(np.linspace(0, 6, n_vis)).astype(np.uint16)
    e = (e if rising else e[::-1])[:, None, None]
    # times 2^e on the bf16 bits: e added to the exponent field of every normal value
    normal = (K & 0x7F80) != 0
    K = np.where(normal, K + (e << 7), K).astype(np.uint16)
    w, idx, ref = run_case(Q, K, offs, H_q, H_kv, 128, 5, mode=B.SOFTMAX)
    err = rel_err(w, ref)
    assert err <= 1e-3, err  # fp32 exponents of scores up to ~2^9 in size


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,d,tokens", [
    (1, 2, 2, 64, [1]),               # one query row, one token
    (17, 4, 2, 64, [0, 5, 0, 3]),     # grouped heads, empty frames, a ragged tile
    (3, 1, 1, 128, [16, 16]),         # one head, whole tiles
    (2, 6, 3, 64, [300, 0, 41]),      # several tiles per wave group
])
def test_softmax_score_kernel_edges(dtype, n_q, H_q, H_kv, d, tokens):
    """Edge shapes of SOFTMAX through the score kernel (heads of whole
    128-byte segments)."""
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(n_q * 13 + d + len(tokens), n_q, int(offs[-1]), H_q, H_kv, d, dtype)
    for k in (0, 1, 3):
        run_case(Q, K, offs, H_q, H_kv, d, k, mode=B.SOFTMAX, dtype=dtype)


@pytest.mark.parametrize("H_q,H_kv", [(4, 4), (8, 2)])
def test_softmax_identical_keys_tie(H_q, H_kv):
    """Identical keys: every probability is 1/n_vis in both passes of the
    score kernel, so every frame scores the same bits and the top-k is the
    lowest frame indices (Eq. 8's tie rule)."""
    n_q, d = 20, 64
    tokens = [7, 30, 1, 64, 12, 5]
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(4711, n_q, int(offs[-1]), H_q, H_kv, d, "bf16")
    K[:] = K[0]
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs.astype(np.int32)), 3, score_mode=B.SOFTMAX)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    assert np.all(w.view(np.uint32) == w[0].view(np.uint32)), w
    assert idx.cpu().tolist() == [0, 1, 2]
    ref = oracle.qer_scores(Q, K, offs, H_q, H_kv, d, B.SOFTMAX)
    assert rel_err(w, ref) <= TOL["bf16"]


def test_explicit_scale():
    offs = synth.frame_offsets([16] * 6)
    Q, K = synth.random_qk(5, 16, 96, 4, 4, 32, "bf16")
    run_case(Q, K, offs, 4, 4, 32, 2, scale=0.25)
    run_case(Q, K, offs, 4, 4, 32, 2, mode=B.SOFTMAX, scale=0.25)


def test_planted_frame_and_ties():
    """A frame whose keys align with the mean query ranks first; identical
    frames tie and resolve to the lower index."""
    d, H = 32, 4
    Q, K = synth.random_qk(9, 16, 160, H, H, d, "f32")
    qbar = Q.mean(axis=0)
    K[48:64] = 3.0 * qbar / np.linalg.norm(qbar, axis=-1, keepdims=True)
    K[96:112] = K[0:16]  # frames 6 and 0 identical
    offs = synth.frame_offsets([16] * 10)
    w, idx, ref = run_case(Q, K, offs, H, H, d, 1, dtype="f32")
    assert idx.tolist() == [3]
    assert w[6] == w[0]


def test_no_frames_no_tokens():
    Q, K = synth.random_qk(1, 4, 8, 2, 2, 16, "bf16")
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(np.zeros(1, np.int32)), 3)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [-1, -1, -1]
    offs = np.array([0, 0, 0], np.int32)
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K[:0]), to_dev(offs), 1)
    torch.cuda.synchronize()
    assert np.isneginf(w.cpu().numpy()).all() and idx.cpu().tolist() == [0]


def test_malformed_offsets_are_clamped():
    """Offsets outside [0, n_vis] or inverted ranges read nothing out of bounds:
    frame f covers [clamp(off[f]), max(that, clamp(off[f+1])))."""
    Q, K = synth.random_qk(2, 4, 40, 2, 2, 16, "bf16")
    offs = np.array([-5, 10, 4, 40, 1000], np.int32)
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs), 4)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    spans = [(0, 10), (10, 10), (4, 40), (40, 40)]
    ref = np.array([oracle.qer_scores(Q, K, np.array(sp, np.int32), 2, 2, 16)[0] for sp in spans])
    assert rel_err(w, ref) <= 2e-2 and np.isneginf(w[1]) and np.isneginf(w[3])
    check_topk(idx.cpu().numpy(), ref, 4)


def test_deterministic_and_workspace():
    Q, K, offs = synth.qer_inputs(2)
    Qd, Kd, od = qk_dev(Q), qk_dev(K), to_dev(offs)
    w1, i1 = B.cofie_qer_rank(Qd, Kd, od, 16)
    desc = B.qer_desc(32, K.shape[0], 128, 28, 28, 128)
    ws = torch.empty(B.qer_workspace_bytes(desc, 16), dtype=torch.uint8, device="cuda")
    w2, i2 = B.cofie_qer_rank(Qd, Kd, od, 16, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(w1, w2) and torch.equal(i1, i2)


def test_poisoned_workspace():
    """The frame-mean kernel's arrival counters live in the workspace: fill it
    with 0xFF, then rank twice with it (single query and several queries)."""
    Q, K, offs = synth.qer_inputs(1)
    wl = synth.WORKLOADS[1]
    Qd, Kd, od = qk_dev(Q), qk_dev(K), to_dev(offs)
    w1, i1 = B.cofie_qer_rank(Qd, Kd, od, wl.k_top)
    desc = B.qer_desc(wl.n_q, K.shape[0], len(offs) - 1, wl.H_q, wl.H_kv, wl.d, dtype=B.F32)
    ws = torch.full((B.qer_workspace_bytes(desc, wl.k_top),), 255, dtype=torch.uint8, device="cuda")
    for _ in range(2):
        w2, i2 = B.cofie_qer_rank(Qd, Kd, od, wl.k_top, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(w1, w2) and torch.equal(i1, i2)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H,d,tokens", [
    (20, 8, 64, [97] * 99),        # ~600 tiles: contraction split 2 ways
    (20, 8, 64, [100] * 81 + [3]),   # 507 tiles: split 4 ways, two tiles per workgroup, ragged last tile
    (32, 28, 128, [144] * 49 + [7]),  # multi-stream heads, a short candidate prefix: split 4 ways
])
def test_split_contraction(dtype, n_q, H, d, tokens):
    """Inputs with fewer 16-token tiles than waves on the chip: the score
    kernel splits each tile's contraction over several waves and adds their
    partial sums before the maximum over the query rows."""
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(777 + len(tokens), n_q, int(offs[-1]), H, H, d, dtype)
    run_case(Q, K, offs, H, H, d, 16, dtype=dtype)


def test_many_tokens_per_workgroup():
    """More 16-token tiles than one pass of a workgroup's waves covers (the
    score kernel loops over rounds of tiles, refilling the query phases), with
    a contraction of several query phases."""
    n_q, H, d = 4, 32, 128
    tokens = [10000] * 7
    offs = synth.frame_offsets(tokens)
    Q, K = synth.random_qk(4242, n_q, int(offs[-1]), H, H, d, "bf16")
    run_case(Q, K, offs, H, H, d, 3)


@pytest.mark.parametrize("n_frames", [1, 7, 128, 129, 1000, 8192, 8193, 20000])
@pytest.mark.parametrize("k", [1, 16, 300])
def test_topk_selection_exact(n_frames, k):
    """The selection itself, bit for bit: the GPU's top-k indices equal the
    oracle's top-k of the GPU's own frame scores.  One token per frame drawn
    from 5 distinct key rows, so scores tie exactly in large groups, and every
    13th frame is empty (score -inf); covers the counting path (<= 128 frames),
    the radix select on LDS-staged keys (<= 8192) and on keys in memory."""
    H, d, n_q = 1, 16, 4
    Q, base = synth.random_qk(77, n_q, 5, H, H, d, "bf16")
    tokens = np.where(np.arange(n_frames) % 13 == 12, 0, 1)
    rows = (np.flatnonzero(tokens) * 7919) % 5
    K = base[rows]
    offs = synth.frame_offsets(tokens)
    print(f"topk n_frames={n_frames} k={k}", flush=True)
    w, idx = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs), k)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    assert np.array_equal(idx.cpu().numpy(), oracle.topk(w.astype(np.float64), k))
