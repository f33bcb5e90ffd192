"""Dense W4A8 products of M activation rows (q4q8_gemm) against the oracle's
W4A8 product row by row (GPU).

Each output row m must agree with the oracle's fp64 product of xq[m] within
1e-5 times the sum of the magnitudes of its scaled block terms (the fp32
rounding of one scaling and one add per block); with every scale 1.0 the
result is the exact integer sum and must match bit for bit."""
import numpy as np
import pytest

import oracle
import paper_2606_24031_amd as w4
from paper_2606_24031_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def _rows_check(y, w, xq, N, K, rows, cols=None):
    for m in rows:
        ref, R = oracle.gemv(w if cols is None else w[cols], xq[m], N if cols is None else len(cols),
                             K)
        got = y[m] if cols is None else y[m, cols]
        assert np.all(np.abs(got.astype(np.float64) - ref) <= 1e-5 * R), f"row {m}"


# K <= 2048 and M <= 128: the VALU kernel of the small groups, the rows in
# chunks of 8 (2 one partial chunk, 8 one full, 17 a 1-row chunk last, 128
# sixteen full); M = 129 and K = 4096: the MFMA tiles (33 one tile, both
# 32-row halves; 64 and 65 a full tile, then a 1-row tile; 96 a full and a
# 32-row tile; 2-32 the 32-row tiles of a few rows).  N: ragged past a
# 128-row slice; K: 512 (codes resident, several slices per workgroup), 768
# (three staged groups), 2048, 4096.
@pytest.mark.parametrize("M", [2, 8, 17, 32, 33, 64, 65, 96, 128, 129])
@pytest.mark.parametrize("N,K", [(1000, 2048), (4096, 512), (333, 768), (40, 256), (300, 4096)])
def test_gemm_matches_oracle(M, N, K):
    print(f"gemm M={M} N={N} K={K}", flush=True)
    g = synth.rng(10 * M + N + K)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, -1)
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (M, K))).reshape(M, -1)
    y = w4.q4q8_gemm(dev(w), dev(xq), M, N, K).cpu().numpy()
    _rows_check(y, w, xq, N, K, range(M))


def test_gemm_prefill_rows_sampled():
    """947 rows (14 full tiles and a 51-row tile) at the dense layer shape
    N = 2048, K = 2048: 40 sampled rows and the first and last."""
    M, N, K = 947, 2048, 2048
    g = synth.rng(947)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, -1)
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (M, K))).reshape(M, -1)
    y = w4.q4q8_gemm(dev(w), dev(xq), M, N, K).cpu().numpy()
    rows = np.unique(np.concatenate([[0, M - 1], g.choice(M, 40, replace=False)]))
    _rows_check(y, w, xq, N, K, rows)


def test_gemm_lm_head_shape_sampled():
    """The output projection at 32 rows (N = 151936 vocabulary rows, K =
    2048): 300 sampled columns of 8 sampled rows and the first and last."""
    M, N, K = 32, 151936, 2048
    g = synth.rng(151)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, -1)
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (M, K))).reshape(M, -1)
    y = w4.q4q8_gemm(dev(w), dev(xq), M, N, K).cpu().numpy()
    cols = np.unique(np.concatenate([[0, N - 1], g.choice(N, 300, replace=False)]))
    rows = np.unique(np.concatenate([[0, M - 1], g.choice(M, 6, replace=False)]))
    _rows_check(y, w, xq, N, K, rows, cols)


@pytest.mark.parametrize("M,N,K", [(70, 300, 2048), (40, 256, 512), (19, 300, 2048), (32, 200, 768),
                                   (70, 200, 4096), (19, 100, 4096)])
def test_gemm_unit_scales_exact(M, N, K):
    """Every scale 1.0: each block term and every partial sum is an integer
    below 2^24, so the fp32 result is the exact integer sum."""
    g = synth.rng(71 + M)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, K // 32, 18)
    w[:, :, 0:2] = np.array([0x3C00], np.uint16).view(np.uint8)
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (M, K))).reshape(M, K // 32, 34)
    xq[:, :, 0:2] = np.array([0x3C00], np.uint16).view(np.uint8)
    y = w4.q4q8_gemm(dev(w), dev(xq), M, N, K).cpu().numpy()
    for m in range(M):
        ref, _ = oracle.gemv(w, xq[m], N, K)
        assert np.array_equal(y[m].astype(np.float64), ref), f"row {m}"


def test_gemm_single_row_is_the_gemv():
    N, K = 777, 1024
    g = synth.rng(77)
    w = dev(synth.q4_0_random_blocks(g, N, K).reshape(N, -1))
    xq = dev(oracle.q8_0_quantize(synth.normal_f32(g, (1, K))).reshape(1, -1))
    a = w4.q4q8_gemm(w, xq, 1, N, K).cpu().numpy()
    b = w4.q4q8_gemv(w, xq, N, K).cpu().numpy()
    assert np.array_equal(a.ravel(), b.ravel())


def test_gemm_workspace_reused_and_output_rows_untouched_past_m():
    """One workspace for a larger then a smaller call; rows of y past M are
    never written."""
    N, K = 200, 1024
    g = synth.rng(88)
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, -1)
    ws = w4.gemm_workspace(80, K)
    for M in (80, 35, 20, 3):
        xq = oracle.q8_0_quantize(synth.normal_f32(g, (M, K))).reshape(M, -1)
        y = torch.full((M + 3, N), 7.0, device="cuda")
        w4.q4q8_gemm(dev(w), dev(xq), M, N, K, y=y, workspace=ws)
        yh = y.cpu().numpy()
        assert (yh[M:] == 7.0).all()
        _rows_check(yh[:M], w, xq, N, K, range(M))
