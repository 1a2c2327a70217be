"""Pins of the oracle's evidence-preservation metrics (appendix, Preservation
of Answer-Relevant Evidence): Attention Preservation Ratio and Top-Evidence
Recall@20%, against hand-computed cases and a numpy brute force."""
import numpy as np
import pytest

import oracle


def test_hand_computed():
    w = np.array([1.0, 2.0, 3.0, 4.0, 10.0])
    assert oracle.evidence_preservation(w, np.array([0, 1, 0, 1, 1]), 0.4) == (0.8, 1.0)
    # k = round(0.2 * 5) = 1: frame 4 (score 10) is dropped
    assert oracle.evidence_preservation(w, np.array([1, 1, 1, 1, 0]), 0.2) == (0.5, 0.0)
    assert oracle.evidence_preservation(w, np.ones(5), 0.2) == (1.0, 1.0)
    assert oracle.evidence_preservation(w, np.zeros(5), 0.2) == (0.0, 0.0)
    # k = round(0.5 * 5) = round(2.5) = 2 (half to even); ties go to the lower index
    w2 = np.array([5.0, 5.0, 5.0, 1.0, 1.0])
    assert oracle.evidence_preservation(w2, np.array([1, 0, 1, 0, 0]), 0.5)[1] == 0.5


@pytest.mark.parametrize("n", [1, 7, 100, 1000])
def test_matches_brute_force(n):
    rng = np.random.default_rng([2609, 3675, 93, n])
    w = rng.random(n) * (rng.random(n) < 0.8)          # zeros tie
    mask = (rng.random(n) < 0.4).astype(np.uint8)
    for p in (0.0, 0.2, 0.5, 1.0):
        apr, rec = oracle.evidence_preservation(w, mask, p)
        k = max(1, min(n, int(np.round(p * n))))         # numpy rounds half to even
        top = np.lexsort((np.arange(n), -w))[:k]          # score desc, index asc
        assert rec == mask[top].sum() / k
        assert abs(apr - (w[mask == 1].sum() / w.sum() if w.sum() else 0.0)) <= 1e-12
