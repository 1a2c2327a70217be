"""Helpers for the GPU parity tests: device transfer and the comparison rules."""
import numpy as np

import torch


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    """bf16 bit patterns (uint16) -> torch.bfloat16 GPU tensor with those bits."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def qk_dev(x: np.ndarray) -> torch.Tensor:
    return bf16_dev(x) if x.dtype == np.uint16 else to_dev(x.astype(np.float32))


def hist_np(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


# Regression bound of the bf16 MFMA paths, beside the 2e-2 contract: the
# operands the matrix cores multiply are exact (bf16 inputs; a folded
# grouped-query sum carried as three bf16 terms), products are exact in fp32,
# and only the fp32 accumulation order differs from the fp64 oracle, which
# leaves ~1e-7 relative.  An operand rounded to a single bf16 term (relative
# error 2^-9 per element) moves the scores by ~1e-4 and fails it.
BF16_REGRESSION = 1e-5


def rel_err(w_gpu: np.ndarray, w_ref: np.ndarray) -> float:
    """max_f |w - w_ref| / max(|w_ref|, 1e-3 max|w_ref|) over finite reference scores."""
    fin = np.isfinite(w_ref)
    if not fin.any():
        return 0.0
    ref = w_ref[fin]
    floor = 1e-3 * np.abs(ref).max()
    den = np.maximum(np.abs(ref), floor if floor > 0 else 1.0)
    return float(np.max(np.abs(w_gpu[fin].astype(np.float64) - ref) / den))


def check_topk(idx_gpu: np.ndarray, w_ref: np.ndarray, k_top: int, tie_rel: float = 1e-6):
    """Top-k parity: exact set equality, except inside a group of reference
    scores within tie_rel (relative) of the k-th score when the k-th and
    (k+1)-th reference scores are that close.  Output must be chronological
    and -1 padded."""
    n = w_ref.size
    k = min(k_top, n)
    got = idx_gpu[:k].tolist()
    assert got == sorted(got), "top-k not in chronological order"
    assert np.all(idx_gpu[k:k_top] == -1), "top-k not padded with -1"
    key = np.where(np.isnan(w_ref), -np.inf, w_ref)
    order = np.lexsort((np.arange(n), -key))
    expect = set(order[:k].tolist())
    if k == 0:
        assert got == []
        return
    if k < n:
        kth, nxt = key[order[k - 1]], key[order[k]]
        scale = max(abs(kth), 1e-30)
        if np.isfinite(kth) and abs(kth - nxt) <= tie_rel * scale:
            tie = set(np.flatnonzero(np.abs(key - kth) <= tie_rel * scale).tolist())
            sure = expect - tie
            assert sure <= set(got), "a frame clearly in the top-k is missing"
            assert set(got) - sure <= tie, "a frame outside the tie group was selected"
            return
    assert set(got) == expect
