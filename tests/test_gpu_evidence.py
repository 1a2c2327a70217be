"""GPU parity of the selection on given scores (cofie_topk, bit for bit) and
of the evidence-preservation metrics (APR within 1e-12 relative, the fp64 sum
order differs; recall exactly) against the oracle."""
import numpy as np
import pytest

import oracle
from paper_2609_03675_amd import binding as B
from paper_2609_03675_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import qk_dev, require_gpu, to_dev  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    B.lib()


def scores(n, seed):
    rng = np.random.default_rng([2609, 3675, 94, n, seed])
    w = np.round(rng.normal(size=n), 2).astype(np.float32)   # many exact ties
    if n > 3:
        w[rng.integers(0, n, 3)] = [np.nan, -np.inf, -0.0]
    return w


@pytest.mark.parametrize("n", [0, 1, 5, 128, 129, 3000, 8193, 20000])
@pytest.mark.parametrize("k", [0, 1, 16, 500])
def test_topk(n, k):
    w = scores(n, k)
    idx = B.cofie_topk(to_dev(w) if n else torch.empty(0, device="cuda"), k)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), oracle.topk(w.astype(np.float64), k))


@pytest.mark.parametrize("n", [1, 10, 1000, 50000])
@pytest.mark.parametrize("p", [0.0, 0.2, 0.5])
def test_evidence_preservation(n, p):
    rng = np.random.default_rng([2609, 3675, 95, n])
    w = (rng.random(n) * (rng.random(n) < 0.9)).astype(np.float32)
    mask = (rng.random(n) < 0.3).astype(np.uint8)
    out = B.cofie_evidence_preservation(to_dev(w), to_dev(mask), p)
    torch.cuda.synchronize()
    apr, rec = out.cpu().numpy()
    apr_o, rec_o = oracle.evidence_preservation(w.astype(np.float64), mask, p)
    assert abs(apr - apr_o) <= 1e-12 * max(1.0, abs(apr_o)) and rec == rec_o


def test_evidence_of_qer_softmax_scores():
    """Full-video QER in SOFTMAX mode (an attention mass) on the tiny workload,
    and a coarse mask: the metrics over the GPU's own scores."""
    wl = synth.WORKLOADS[1]
    Q, K, offs = synth.qer_inputs(1)
    w, _ = B.cofie_qer_rank(qk_dev(Q), qk_dev(K), to_dev(offs), 0, score_mode=B.SOFTMAX)
    mask = to_dev((np.arange(wl.n_frames) % 3 != 1).astype(np.uint8))
    out = B.cofie_evidence_preservation(w, mask, 0.2)
    torch.cuda.synchronize()
    apr, rec = out.cpu().numpy()
    apr_o, rec_o = oracle.evidence_preservation(w.cpu().numpy().astype(np.float64), mask.cpu().numpy(), 0.2)
    assert abs(apr - apr_o) <= 1e-12 and rec == rec_o and 0 < apr < 1
