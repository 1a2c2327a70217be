"""GPU parity of the coarse-to-fine glue through the C ABI against the CPU
oracle, bit for bit: candidate compaction of an NGFF mask (Sec. 3.1-3.2) and
the chronological removal of the frames outside S_e from a token sequence
(Sec. 3.3)."""
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


@pytest.mark.parametrize("n,seg_len", [(0, 0), (0, 4), (1, 0), (5, 1), (16383, 0), (16384, 512),
                                       (16385, 1000), (100000, 0), (100000, 7), (70000, 100000)])
@pytest.mark.parametrize("p", [0.0, 0.25, 1.0])
def test_mask_compact(n, seg_len, p):
    rng = np.random.default_rng([2609, 3675, 90, n, seg_len, int(p * 100)])
    mask = ((rng.random(n) < p) * rng.integers(1, 256, n)).astype(np.uint8)
    print(f"compact n={n} seg_len={seg_len} p={p}", flush=True)
    idx, seg = B.cofie_mask_compact(to_dev(mask) if n else torch.empty(0, dtype=torch.uint8, device="cuda"),
                                    seg_len)
    torch.cuda.synchronize()
    ref_idx, ref_seg = oracle.mask_compact(mask, seg_len)
    seg = seg.cpu().numpy()
    assert np.array_equal(seg, ref_seg)
    assert np.array_equal(idx.cpu().numpy()[:seg[-1]], ref_idx)


def test_compact_of_ngff_mask():
    """NGFF on the GPU, then the candidate list of every stream."""
    frames = synth.random_frames(11, 96, 24, 32, scenes=6)
    rule = B.keep_rule("per_channel", 0.05, 8, 3, 32)
    _, mask = B.cofie_ngff_filter(to_dev(frames), 16, rule)
    idx, seg = B.cofie_mask_compact(mask, 32)
    torch.cuda.synchronize()
    h = oracle.histogram(frames, 16, oracle.PER_CHANNEL)
    _, mo, _ = oracle.ngff_select(h, oracle.mass(oracle.PER_CHANNEL, 24, 32), 0.05, 8, 3, 32)
    ref_idx, ref_seg = oracle.mask_compact(mo, 32)
    assert np.array_equal(seg.cpu().numpy(), ref_seg)
    assert np.array_equal(idx.cpu().numpy()[:ref_seg[-1]], ref_idx)


def random_case(seed, n_frames, row_shape, dtype):
    rng = np.random.default_rng([2609, 3675, 91, seed])
    sizes = rng.integers(0, 12, n_frames)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    n_rows = int(offs[-1])
    src = rng.integers(0, 30000, (n_rows,) + row_shape).astype(dtype)
    sel = np.sort(rng.choice(n_frames, min(n_frames, 20), replace=False)).astype(np.int32)
    sel = np.concatenate([sel, [sel[0], -1, n_frames, -7]]).astype(np.int32)  # a repeat and invalid entries
    return src, offs, sel


def check_gather(src, offs, sel, capacity):
    dst, out_offs, out_rows = B.cofie_gather_frames(to_dev(src), to_dev(offs), to_dev(sel), capacity=capacity)
    torch.cuda.synchronize()
    rdst, roffs, rrows = oracle.gather_frames(src, offs, sel, capacity)
    m = rrows.size
    assert np.array_equal(out_offs.cpu().numpy(), roffs)
    assert np.array_equal(out_rows.cpu().numpy()[:m], rrows)
    assert np.array_equal(dst.cpu().numpy()[:m], rdst)


@pytest.mark.parametrize("row_shape,dtype", [((7,), np.uint8),       # byte lanes
                                             ((3, 5), np.int16),     # 30-byte rows: byte lanes
                                             ((1,), np.float32),     # 4-byte lanes
                                             ((28, 128), np.int16)])  # 7168-byte rows: 16-byte lanes
def test_gather_frames(row_shape, dtype):
    src, offs, sel = random_case(len(row_shape) * 10 + np.dtype(dtype).itemsize, 60, row_shape, dtype)
    print(f"gather rows={src.shape} dtype={dtype}", flush=True)
    for cap in (src.shape[0], 0, 9, 3 * src.shape[0]):
        check_gather(src, offs, sel, cap)


@pytest.mark.parametrize("k", [4096, 5000])
def test_gather_many_frames(k):
    """Up to 4096 selected frames one kernel copies them (each workgroup sums
    the row counts before its frame); more take the offsets kernel first."""
    rng = np.random.default_rng([2609, 3675, 92, k])
    n_frames = 6000
    sizes = rng.integers(0, 4, n_frames)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    src = rng.integers(0, 30000, (int(offs[-1]), 8)).astype(np.int16)
    sel = np.sort(rng.choice(n_frames, k, replace=False)).astype(np.int32)
    print(f"gather {k} of {n_frames} frames, {src.shape[0]} rows", flush=True)
    for cap in (src.shape[0], src.shape[0] // 3):
        check_gather(src, offs, sel, cap)


def test_gather_malformed_offsets_and_misaligned_rows():
    src = np.arange(40 * 6, dtype=np.uint8).reshape(40, 6)
    offs = np.array([-5, 3, 2, 60, 7, 7, 40], np.int32)
    sel = np.array([0, 1, 2, 3, 5, -1], np.int32)
    check_gather(src, offs, sel, 40)
    # a source view at an odd byte address takes the byte path
    base = torch.from_numpy(np.arange(41 * 6, dtype=np.uint8)).cuda()
    view = base[1:1 + 40 * 6].view(40, 6)
    dst, out_offs, out_rows = B.cofie_gather_frames(view, to_dev(offs), to_dev(sel), capacity=40)
    torch.cuda.synchronize()
    rdst, roffs, rrows = oracle.gather_frames(view.cpu().numpy(), offs, sel, 40)
    assert np.array_equal(out_offs.cpu().numpy(), roffs)
    assert np.array_equal(dst.cpu().numpy()[:rrows.size], rdst)


def test_qer_then_gather_keys():
    """QER top-k on the GPU, then the selected frames' keys in chronological
    order: the shortened key sequence the remaining layers would read."""
    wl = synth.WORKLOADS[1]
    Q, K, offs = synth.qer_inputs(1)
    Kd = qk_dev(K)
    od = to_dev(offs)
    w, idx = B.cofie_qer_rank(qk_dev(Q), Kd, od, wl.k_top)
    dst, out_offs, out_rows = B.cofie_gather_frames(Kd, od, idx)
    torch.cuda.synchronize()
    sel = idx.cpu().numpy()
    rdst, roffs, rrows = oracle.gather_frames(K, offs, sel)
    assert np.array_equal(out_offs.cpu().numpy(), roffs)
    assert np.array_equal(out_rows.cpu().numpy()[:rrows.size], rrows)
    assert np.array_equal(dst.cpu().numpy()[:rrows.size].view(np.uint8), rdst.view(np.uint8))
    assert np.all(np.diff(rrows) > 0)  # chronological
