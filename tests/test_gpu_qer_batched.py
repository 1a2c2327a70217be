"""GPU parity of QER for several queries sharing one key sequence (Sec. 3.3,
Eqs. 6-8; each query of a stream ranks the prefix of candidates it has seen,
Sec. 3.1) against the fp64 CPU oracle through the C ABI.  Every query's
scores within the single-query tolerances and its top-k exact; the batched
call also equals one single-query call per query, bit for bit, since grouping
the queries changes neither a dot product's order nor a frame's mean."""
import numpy as np
import pytest

import oracle
from paper_2609_03675_amd import binding as B
from paper_2609_03675_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import check_topk, qk_dev, rel_err, require_gpu, to_dev  # noqa: E402

TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    B.lib()


def make_case(seed, n_queries, n_q, H_q, H_kv, d, n_frames, dtype, max_tokens=24):
    rng = np.random.default_rng([2609, 3675, 93, seed])
    sizes = rng.integers(0, max_tokens + 1, n_frames)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    n_vis = int(offs[-1])

    def normal(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return x if dtype == "f32" else (x.view(np.uint32) >> 16).astype(np.uint16)

    Q = normal((n_queries, n_q, H_q, d))
    K = normal((n_vis, H_kv, d))
    nf = rng.integers(0, n_frames + 1, n_queries).astype(np.int32)
    nf[0] = n_frames  # one query sees the whole sequence
    return Q, K, offs, nf


def run_batched(Q, K, offs, nf, H_q, H_kv, d, k_top, dtype, mode=B.LOGIT):
    n_queries, n_q = Q.shape[:2]
    n_frames = len(offs) - 1
    print(f"qer batched queries={n_queries} n_q={n_q} n_vis={K.shape[0]} frames={n_frames} "
          f"H={H_q}/{H_kv} d={d} k={k_top} {dtype} mode={mode} nf={nf.tolist()}", flush=True)
    w, idx = B.cofie_qer_rank_batched(qk_dev(Q), qk_dev(K), to_dev(offs), nf, k_top, score_mode=mode)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    idx = idx.cpu().numpy()
    worst = 0.0
    for g in range(n_queries):
        f = int(nf[g])
        # the oracle on the prefix: the first f frames and their tokens only
        ref = oracle.qer_scores(Q[g], K[:offs[f]], offs[:f + 1], H_q, H_kv, d, mode)
        worst = max(worst, rel_err(w[g, :f], ref))
        assert np.array_equal(np.isneginf(w[g, :f]), np.isneginf(ref)), f"query {g}: empty-frame scores differ"
        assert np.all(np.isneginf(w[g, f:])), f"query {g}: scores past its prefix are not -inf"
        check_topk(idx[g], ref, k_top)
    print(f"  max rel err {worst:.3e}", flush=True)
    assert worst <= TOL[dtype], worst
    return w, idx


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_queries,n_q,H_q,H_kv,d,n_frames", [
    (3, 16, 4, 4, 32, 40),      # one 64-row chunk holds all queries
    (5, 48, 2, 2, 64, 70),      # queries straddle 64-row chunks
    (4, 32, 8, 2, 32, 33),      # GQA fold
    (6, 16, 28, 4, 128, 150),   # GQA, high-res workload heads, 96 rows
    (2, 64, 1, 1, 16, 9),       # one query per chunk
    (1, 20, 4, 4, 32, 30),      # a single query may have any n_q
])
def test_batched_against_oracle(dtype, n_queries, n_q, H_q, H_kv, d, n_frames):
    Q, K, offs, nf = make_case(n_queries * 100 + n_q + d, n_queries, n_q, H_q, H_kv, d, n_frames, dtype)
    run_batched(Q, K, offs, nf, H_q, H_kv, d, 8, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_queries,n_q,H_q,H_kv,d,n_frames,max_tokens", [
    (3, 16, 4, 4, 64, 40, 24),        # one 64-row chunk holds all queries
    (5, 32, 28, 4, 128, 30, 60),      # grouped heads, queries straddle 64-row chunks
    (4, 32, 8, 8, 64, 48, 900),       # ~1500 tiles
])
def test_batched_softmax(dtype, n_queries, n_q, H_q, H_kv, d, n_frames, max_tokens):
    """SOFTMAX for several queries: query g's softmax runs over the keys of
    its own prefix (pass 1 counts no key past offs[nf[g]]), so every query
    matches the oracle on its prefix, and a single-query call on the prefix to
    rounding (the work split, which orders the sums, follows the key count)."""
    Q, K, offs, nf = make_case(n_queries * 10 + d, n_queries, n_q, H_q, H_kv, d, n_frames, dtype, max_tokens)
    w, idx = run_batched(Q, K, offs, nf, H_q, H_kv, d, 6, dtype, mode=B.SOFTMAX)
    Kd, od = qk_dev(K), to_dev(offs)
    for g in range(n_queries):
        f = int(nf[g])
        if f == 0:
            continue
        w1, _ = B.cofie_qer_rank(qk_dev(Q[g]), Kd[:int(offs[f])].contiguous(), od[:f + 1].contiguous(), 6,
                                 score_mode=B.SOFTMAX)
        torch.cuda.synchronize()
        assert rel_err(w[g, :f], w1.cpu().numpy().astype(np.float64)) <= 1e-5, g


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_batched_wide_pass(dtype):
    """128 query rows (four queries of 32) over more tiles than a split would
    take: the score kernel multiplies all of them in one pass over K."""
    Q, K, offs, nf = make_case(11, 4, 32, 8, 8, 64, 48, dtype, max_tokens=900)
    assert K.shape[0] > 16 * 1024
    run_batched(Q, K, offs, nf, 8, 8, 64, 10, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_q,H_q,H_kv,max_tokens", [
    (48, 28, 4, 24),     # GQA fold (three query terms)
    (32, 28, 28, 24),    # multi-stream heads: few tiles, contraction split 4 ways
    (32, 8, 8, 300),     # 512-long contraction split 2 ways (~590 tiles)
    (32, 8, 8, 700),     # ~1400 tiles, no split: 160 rows as one 128-row pass and one of 32
])
def test_batched_equals_single_query_calls(dtype, n_q, H_q, H_kv, max_tokens):
    """Per-query calls over the same keys add in the same order as the
    batched call (also when the score kernel splits the contraction, whose
    split depends on the keys and heads only), so the scores are equal bit for
    bit."""
    n_queries, d, n_frames = 5, 128 if H_q == 28 else 64, 64
    Q, K, offs, nf = make_case(7, n_queries, n_q, H_q, H_kv, d, n_frames, dtype, max_tokens)
    w, idx = run_batched(Q, K, offs, nf, H_q, H_kv, d, 12, dtype)
    Kd, od = qk_dev(K), to_dev(offs)
    for g in range(n_queries):
        f = int(nf[g])
        w1, i1 = B.cofie_qer_rank(qk_dev(Q[g]), Kd, od[:f + 1].contiguous(), 12)
        torch.cuda.synchronize()
        assert np.array_equal(w1.cpu().numpy().view(np.uint32), w[g, :f].view(np.uint32)), g
        assert np.array_equal(i1.cpu().numpy(), idx[g]), g


@pytest.mark.parametrize("mode", [B.LOGIT, B.SOFTMAX])
def test_stream_queries_on_candidate_prefixes(mode):
    """The multi-stream use: the queries of one stream of the multi-stream
    workload (T = 512, 144 tokens per frame), each ranking the candidates
    that precede its timestamp (in SOFTMAX mode, each query's softmax over the
    keys of its own prefix)."""
    wl = synth.WORKLOADS[5]
    rng = np.random.default_rng([2609, 3675, 94])
    cands = np.sort(rng.choice(wl.T, 40, replace=False))
    ts = synth.multistream_queries(5, 0)
    nf = np.searchsorted(cands, ts, side="right").astype(np.int32)
    Q = np.stack([synth.multistream_q(5, 0, g) for g in range(len(ts))])
    K = synth.multistream_k(5, 0, cands)
    offs = np.arange(0, (len(cands) + 1) * wl.tokens, wl.tokens, dtype=np.int32)
    run_batched(Q, K, offs, nf, wl.H_q, wl.H_kv, wl.d, wl.k_top, wl.qk_dtype, mode)


def test_empty_prefixes_and_no_topk():
    Q, K, offs, nf = make_case(3, 3, 16, 2, 2, 32, 12, "bf16")
    nf[:] = [0, 12, 0]
    w, idx = run_batched(Q, K, offs, nf, 2, 2, 32, 5, "bf16")
    assert np.all(idx[0] == -1) and np.all(idx[2] == -1)
    w0, _ = B.cofie_qer_rank_batched(qk_dev(Q), qk_dev(K), to_dev(offs), nf, 0)
    torch.cuda.synchronize()
    assert np.array_equal(w0.cpu().numpy().view(np.uint32), w.view(np.uint32))


def test_batched_rejects_unsupported():
    Q, K, offs, nf = make_case(5, 2, 20, 2, 2, 32, 10, "bf16")
    Qd, Kd, od = qk_dev(Q), qk_dev(K), to_dev(offs)
    with pytest.raises(B.CofieError) as e:           # several queries of 20 rows
        B.cofie_qer_rank_batched(Qd, Kd, od, nf, 4)
    assert e.value.code == B.COFIE_EUNSUPPORTED
    Q16 = qk_dev(Q[:, :16].copy())
    with pytest.raises(B.CofieError) as e:           # several queries in softmax mode, 32-element heads
        B.cofie_qer_rank_batched(Q16, Kd, od, nf, 4, score_mode=B.SOFTMAX)
    assert e.value.code == B.COFIE_EUNSUPPORTED
    with pytest.raises(B.CofieError) as e:           # a prefix longer than the sequence
        B.cofie_qer_rank_batched(Q16, Kd, od, np.array([3, 11], np.int32), 4)
    assert e.value.code == B.COFIE_EINVAL
