"""GPU parity of cofie_qer_rank_streams, several independent key sequences
ranked in one launch (Sec. 3.1's streaming setting: each stream's queries
rank prefixes of that stream's candidates; Eqs. 6-8 per query), against the
fp64 oracle through the C ABI: every query's scores over its own sequence's
prefix within the tolerances of cofie_qer_rank (and the 1e-5 regression
bound where the scores are well away from zero), its top-k exact outside
1e-6 ties, frame indices within its sequence.  The edge cases cover empty
sequences, sequences without queries, empty prefixes, ragged and empty
frames, sequences whose queries take several 128-row chunks, chunks that
are not whole 16-row blocks of eight (48-row queries), grouped-query heads
(64-row chunks of three query terms), fp32 inputs and k_top beyond the
frames."""
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


def make_streams(seed, n_q, H_q, H_kv, d, streams, dtype, max_tokens=40):
    """streams: (frames, queries) per sequence.  Returns per-sequence Q, K,
    local CSR and prefixes, plus the concatenated device inputs."""
    rng = np.random.default_rng([2609, 3675, 94, seed])
    per = []
    for nfr, nq in streams:
        sizes = rng.integers(0, max_tokens + 1, nfr)
        offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        Q, K = synth.random_qk(int(rng.integers(1 << 30)), n_q * max(nq, 1), int(offs[-1]), H_q, H_kv, d, dtype)
        Q = Q.reshape(max(nq, 1), n_q, H_q, d)[:nq]
        nf = rng.integers(0, nfr + 1, nq).astype(np.int32)
        if nq:
            nf[0] = nfr
        per.append((Q, K, offs, nf))
    return per


def run_streams(per, n_q, H_q, H_kv, d, k_top, dtype, regression=False):
    Ks = [p[1] for p in per]
    keys = [k.shape[0] for k in Ks]
    frames = [p[2].size - 1 for p in per]
    nq = [p[0].shape[0] for p in per]
    nf = np.concatenate([p[3] for p in per]).astype(np.int32)
    base = np.concatenate([[0], np.cumsum(keys)])
    offs = np.concatenate([[0]] + [p[2][1:] + base[i] for i, p in enumerate(per)]).astype(np.int32)
    K = np.concatenate(Ks, axis=0)
    Q = np.concatenate([p[0] for p in per], axis=0)
    lay = B.StreamsLayout(keys, frames, nq, nf)
    print(f"qer streams keys={keys} frames={frames} queries={nq} n_q={n_q} H={H_q}/{H_kv} d={d} k={k_top} "
          f"{dtype}", flush=True)
    w, idx = B.cofie_qer_rank_streams(qk_dev(Q), qk_dev(K), to_dev(offs), lay, k_top)
    torch.cuda.synchronize()
    w = w.cpu().numpy()
    idx = idx.cpu().numpy()
    assert w.shape == (Q.shape[0], max(1, max(frames)))
    worst = 0.0
    g = 0
    for s, (Qs, Ks_, offs_s, nf_s) in enumerate(per):
        for qi in range(Qs.shape[0]):
            f = int(nf_s[qi])
            ref = oracle.qer_scores(Qs[qi], Ks_[:offs_s[f]], offs_s[:f + 1], H_q, H_kv, d)
            err = rel_err(w[g, :f], ref)
            worst = max(worst, err)
            assert np.array_equal(np.isneginf(w[g, :f]), np.isneginf(ref)), f"query {g}: empty-frame scores differ"
            assert np.all(np.isneginf(w[g, f:frames[s]])), f"query {g}: scores past its prefix are not -inf"
            check_topk(idx[g], ref, k_top)
            g += 1
    print(f"  max rel err {worst:.3e}", flush=True)
    assert worst <= TOL[dtype], worst
    if regression:
        assert worst <= BF16_REGRESSION, worst
    return w, idx


STREAM_SHAPES = [
    (32, 4, 4, 64, [(12, 4), (0, 2), (7, 0), (20, 3), (1, 1)]),   # empty sequence, sequence without queries
    (16, 2, 2, 64, [(30, 9), (5, 1)]),                             # 9 x 16 rows: chunks of 128 + 16
    (48, 4, 4, 32, [(25, 3), (9, 2)]),                             # 96-row chunks: two of eight blocks unused
    (32, 8, 2, 64, [(18, 3), (6, 2), (11, 1)]),                    # grouped heads: 64-row chunks
    (16, 28, 28, 128, [(40, 4), (3, 4), (60, 2)]),                 # workload heads, many tiles
]


# the grouped-head shape in bf16 only: in fp32 its fold is one query term,
# chunked as MHA, which the fp32 MHA shapes cover
@pytest.mark.parametrize("dtype,n_q,H_q,H_kv,d,streams",
                         [("bf16",) + c for c in STREAM_SHAPES] +
                         [("f32",) + c for c in STREAM_SHAPES if not (c[1] != c[2] and c[0] > 16)])
def test_streams_shapes(dtype, n_q, H_q, H_kv, d, streams):
    per = make_streams(n_q + 7 * d + len(streams), n_q, H_q, H_kv, d, streams, dtype)
    for k in (0, 3, 50):
        run_streams(per, n_q, H_q, H_kv, d, k, dtype)


def test_streams_empty_keys_everywhere():
    """No sequence has keys: every frame is empty (-inf) and the top-k lists the
    lowest frame indices of each prefix (all scores tie at -inf)."""
    per = []
    rng = np.random.default_rng(5)
    for nfr, nq in [(3, 2), (0, 1)]:
        offs = np.zeros(nfr + 1, np.int32)
        Q, K = synth.random_qk(int(rng.integers(1000)), 16 * nq, 0, 2, 2, 32, "bf16")
        per.append((Q.reshape(nq, 16, 2, 32), K, offs, np.array([nfr] * nq, np.int32)))
    run_streams(per, 16, 2, 2, 32, 2, "bf16")
