"""GPU parity of the last-layer prefill attention with QER taken from its
own QK^T tiles (Sec. 3.3) through the C ABI: the attention output against
the fp64 oracle's causal attention, the frame scores against the oracle's
QER over the text rows (all non-visual tokens) and the visual rows, the
top-k exact.

Attention tolerance, from the arithmetic: the probabilities enter the value
product rounded to bf16 (relative 2^-9 each; the visual rows' row sums add
the same rounded values, the text rows' chunk sums keep them in fp32), so
the normalised weights are off by at most about 2 * 2^-9 relative, and the
output is rounded to bf16 (2^-9 relative); together at most 3 * 2^-9 of the
largest |v| the row attends to, plus the output rounding, so
|o - o_ref| <= 2^-7 max|v| + 2^-8 |o_ref| per element.  Frame scores within
2e-2 relative as for cofie_qer_rank (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest

import oracle
from paper_2609_03675_amd import binding as B
from paper_2609_03675_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import bf16_dev, check_topk, rel_err, require_gpu, to_dev  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    B.lib()


def dec(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


def make_case(seed, n_pre, n_vis, n_post, H_q, H_kv, n_frames, scale=1.0):
    rng = np.random.default_rng([2609, 3675, 96, seed])
    L = n_pre + n_vis + n_post
    bits = lambda shape: synth.bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))
    Q, K, V = bits((L, H_q, 128)), bits((L, H_kv, 128)), bits((L, H_kv, 128))
    if n_frames:
        cuts = np.sort(rng.integers(0, n_vis + 1, n_frames - 1))
        offs = np.concatenate([[0], cuts, [n_vis]]).astype(np.int32)
    else:
        offs = np.zeros(1, np.int32)
    return Q, K, V, offs


def check(Q, K, V, offs, vb, ve, k_top, rows=None, scale=0.0):
    L, H_q, _ = Q.shape
    H_kv = K.shape[1]
    print(f"attn_qer L={L} vis=[{vb},{ve}) H={H_q}/{H_kv} frames={len(offs)-1} k={k_top} "
          f"rows={'all' if rows is None else len(rows)}", flush=True)
    out, w, idx = B.cofie_attn_qer(bf16_dev(Q), bf16_dev(K), bf16_dev(V), to_dev(offs), vb, ve, k_top, scale=scale)
    torch.cuda.synchronize()
    o = out.view(torch.int16).cpu().numpy().view(np.uint16)
    w, idx = w.cpu().numpy(), idx.cpu().numpy()
    r = np.arange(L, dtype=np.int32) if rows is None else np.asarray(rows, np.int32)
    ref = oracle.attention(Q, K, V, scale=scale, rows=r)
    got = dec(o[r]).astype(np.float64)
    g = np.arange(H_q) * H_kv // H_q
    vmax = np.abs(dec(V)).max(axis=(0, 2))[g]                    # per query head
    bound = 2.0 ** -7 * vmax[None, :, None] + 2.0 ** -8 * np.abs(ref)
    err = np.abs(got - ref)
    print(f"  attention max |err| {err.max():.3e}, worst err/bound {np.max(err / bound):.3f}", flush=True)
    assert np.all(err <= bound)
    # QER: text rows = every non-visual token, in sequence order
    Qt = np.concatenate([Q[:vb], Q[ve:]])
    wref = oracle.qer_scores(Qt, K[vb:ve], offs, H_q, H_kv, 128, oracle.LOGIT, scale)
    e = rel_err(w, wref)
    print(f"  qer max rel err {e:.3e}", flush=True)
    assert e <= 2e-2
    assert np.array_equal(np.isneginf(w), np.isneginf(wref))
    check_topk(idx, wref, k_top)
    return out, w, idx


@pytest.mark.parametrize("n_pre,n_vis,n_post,H_q,H_kv,n_frames", [
    (5, 30, 5, 2, 2, 3),        # one block, one chunk, partial tiles
    (7, 650, 43, 4, 2, 9),      # 3 query blocks (ragged), 2 chunks, grouped heads
    (0, 536, 64, 3, 1, 5),      # 64 text rows, all after the video
    (64, 300, 0, 2, 1, 4),      # all text before the video
    (0, 1000, 1, 2, 2, 7),      # a single text token
    (3, 256, 2, 1, 1, 1),       # exactly one query block
    (1, 1, 1, 2, 2, 1),         # one visual token
    (40, 100, 40, 2, 2, 3),     # 80 text rows: one text workgroup's 128 rows
    (100, 700, 100, 4, 2, 9),   # 200 text rows: two row groups, their m_j maxima combined
    (0, 300, 300, 2, 1, 4),     # 300 text rows, all after the video: three row groups
    (129, 520, 0, 2, 2, 5),     # 129 text rows before the video: a group of one row
])
def test_shapes_against_oracle(n_pre, n_vis, n_post, H_q, H_kv, n_frames):
    Q, K, V, offs = make_case(n_pre * 1000 + n_vis + n_post, n_pre, n_vis, n_post, H_q, H_kv, n_frames)
    check(Q, K, V, offs, n_pre, n_pre + n_vis, 4)


def test_no_visual_tokens_and_empty_frames():
    Q, K, V, _ = make_case(1, 20, 0, 0, 2, 2, 0)
    out, w, idx = check(Q, K, V, np.zeros(4, np.int32), 20, 20, 3)
    assert np.all(np.isneginf(w)) and idx.tolist() == [0, 1, 2]


def test_peaked_logits_and_explicit_scale():
    # large logits: the running max moves often and the weights are peaked
    Q, K, V, offs = make_case(2, 4, 700, 12, 2, 2, 6, scale=3.0)
    check(Q, K, V, offs, 4, 704, 3, scale=0.2)


@pytest.mark.parametrize("H_q,H_kv", [(2, 2), (4, 2)])
def test_outlier_keys_beyond_the_first_lane_group(H_q, H_kv):
    """Keys whose logit exceeds the rest of their 32-key step by about 231
    in base 2 (exp2 of that overflows fp32): a visual row's running max must
    see every key of the step; a max over the first lane group's keys only
    (offsets 0-3 and 16-19 of the step) would leave exp2 to overflow.  The
    outliers sit at offsets 5, 10, 29, 23, 26 and 21 of their steps, i.e. in
    lane groups 1, 2, 3, 1, 2 and 1; positive queries and constant outlier
    keys make every row prefer them.  MHA and two query heads per key head."""
    n_pre, n_vis, n_post = 6, 700, 10
    Q, K, V, offs = make_case(6, n_pre, n_vis, n_post, H_q, H_kv, 7)
    rng = np.random.default_rng([2609, 3675, 97])
    q = np.abs(rng.standard_normal(Q.shape)).astype(np.float32) * 0.5 + 0.5
    Q = synth.bf16_bits(q)
    Kf = dec(K).copy()
    outl = [37, 106, 189, 247, 410, 629]          # offsets 5, 10, 29, 23, 26, 21
    Kf[outl] = 16.0
    K = synth.bf16_bits(Kf)
    rows = np.arange(n_pre + n_vis + n_post, dtype=np.int32)
    check(Q, K, V, offs, n_pre, n_pre + n_vis, 3, rows=rows)


def test_workload_sampled_rows():
    """The 1 fps stream's last layer: 128 candidate frames of 256 tokens and
    32 text tokens (L = 32800, 28 heads); attention checked on sampled rows
    (text rows, block edges, the last rows), QER on every frame."""
    wl = synth.WORKLOADS[2]
    L, vb, ve = synth.attn_layout(2)
    Q, K, V, offs = synth.attn_inputs(2)
    rows = [0, vb - 1, vb, vb + 255, vb + 256, vb + 4095, ve - 257, ve - 1, ve, L - 1]
    check(Q, K, V, offs, vb, ve, wl.k_top, rows=rows)


def test_qer_equals_separate_ranking():
    """The scores from the attention's tiles equal cofie_qer_rank's over the
    same text rows and visual keys up to fp32 summation order."""
    Q, K, V, offs = make_case(3, 6, 900, 26, 4, 4, 12)
    vb, ve = 6, 906
    _, w, idx = B.cofie_attn_qer(bf16_dev(Q), bf16_dev(K), bf16_dev(V), to_dev(offs), vb, ve, 5)
    Qt = np.concatenate([Q[:vb], Q[ve:]])
    w2, idx2 = B.cofie_qer_rank(bf16_dev(Qt), bf16_dev(K[vb:ve]), to_dev(offs), 5)
    torch.cuda.synchronize()
    w, w2 = w.cpu().numpy(), w2.cpu().numpy()
    assert np.max(np.abs(w - w2) / np.maximum(np.abs(w2), 1e-3 * np.abs(w2).max())) <= 1e-4
    assert np.array_equal(idx.cpu().numpy(), idx2.cpu().numpy())


def test_workspace_and_determinism():
    Q, K, V, offs = make_case(4, 2, 520, 9, 2, 2, 5)
    d = B.attn_desc(531, 2, 2, 128, 2, 522, 5)
    nbytes = B.attn_qer_workspace_bytes(d)
    assert nbytes > 0
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    a = B.cofie_attn_qer(bf16_dev(Q), bf16_dev(K), bf16_dev(V), to_dev(offs), 2, 522, 3, workspace=ws)
    b = B.cofie_attn_qer(bf16_dev(Q), bf16_dev(K), bf16_dev(V), to_dev(offs), 2, 522, 3)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)
    small = torch.empty(nbytes // 2, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.CofieError) as e:
        B.cofie_attn_qer(bf16_dev(Q), bf16_dev(K), bf16_dev(V), to_dev(offs), 2, 522, 3, workspace=small)
    assert e.value.code == B.COFIE_ENOMEM


def test_rejects_unsupported():
    Q, K, V, offs = make_case(5, 4, 100, 4, 2, 2, 3)
    with pytest.raises(B.CofieError) as e:  # head dimension 64: only 128 is built
        B.cofie_attn_qer(bf16_dev(Q[..., :64]).contiguous(), bf16_dev(K[..., :64]).contiguous(),
                         bf16_dev(V[..., :64]).contiguous(), to_dev(offs), 4, 104, 3)
    assert e.value.code == B.COFIE_EUNSUPPORTED
    with pytest.raises(B.CofieError) as e:  # no text token: nothing to score with
        B.cofie_attn_qer(bf16_dev(Q[4:104]), bf16_dev(K[4:104]), bf16_dev(V[4:104]), to_dev(offs), 0, 100, 3)
    assert e.value.code == B.COFIE_EINVAL
