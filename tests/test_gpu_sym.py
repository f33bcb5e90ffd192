"""GPU parity for the paper's own block format (Sec. 2.3: symmetric 4-bit
weights in {-7..7} with an fp32 scale per group; Sec. 3.3: 8-bit activations
with an fp32 scale), called through the C ABI, against the CPU oracle on the
same seeded inputs.  Quantized bytes bit-exact; the product within 1e-5 of
sum |d_w d_a s| elementwise, and exact with unit scales."""
import numpy as np
import pytest

import oracle
from paper_2606_24031_amd import synth
import paper_2606_24031_amd as w4

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = "cuda"


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _special_rows(K):
    rows = []
    rows.append(np.zeros(K, np.float32))                                     # zero blocks
    t = np.zeros(K, np.float32)
    t[::32] = 127.0; t[1::32] = 2.5; t[2::32] = -2.5; t[3::32] = 0.5; t[4::32] = -126.5
    rows.append(t)                                                          # exact ties, d = 1 (Q8)
    u = np.zeros(K, np.float32)
    u[::32] = 7.0; u[1::32] = 2.5; u[2::32] = -0.5; u[5::32] = 3.5
    rows.append(u)                                                          # exact ties, d = 1 (Q4)
    rows.append(np.full(K, 1e-39, np.float32))                              # reciprocal overflows
    v = np.full(K, 2.0 ** -120, np.float32); v[::5] = -(2.0 ** -121)
    rows.append(v)                                                          # subnormal scale
    b = np.full(K, 3.0e37, np.float32); b[::3] = -1.0
    rows.append(b)                                                          # large scale
    return np.stack(rows)


def _rows(g, rows, K, std):
    x = synth.normal_f32(g, (rows, K), std)
    x *= (2.0 ** g.integers(-8, 8, size=(rows, 1))).astype(np.float32)
    x[g.random((rows, K)) < 0.01] = 0.0
    return np.concatenate([x, _special_rows(K), -_special_rows(K)])


@pytest.mark.parametrize("rows,K", [(1, 32), (3, 96), (7, 2048), (129, 512), (1000, 1024)])
def test_q8_f32_bit_exact(rows, K):
    g = synth.rng(600 + rows)
    x = _rows(g, rows, K, 1.0)
    assert np.array_equal(host(w4.q8_f32_quantize(dev(x))), oracle.q8_f32_quantize(x))


@pytest.mark.parametrize("rows,K", [(1, 32), (5, 160), (64, 2048), (1023, 512)])
def test_q4_sym_bit_exact(rows, K):
    g = synth.rng(700 + rows)
    w = _rows(g, rows, K, 0.02)
    assert np.array_equal(host(w4.q4_sym_quantize(dev(w))), oracle.q4_sym_quantize(w))


@pytest.mark.parametrize("N,K", [(1024, 1024), (1, 256), (7, 768), (333, 2048),
                                 (64, 16384), (5, 32768), (4097, 512)])
def test_gemv_sym_matches_oracle(N, K):
    g = synth.rng(800 + N)
    W = synth.normal_f32(g, (N, K), 0.02)
    x = synth.normal_f32(g, (K,))
    wq, xq = w4.q4_sym_quantize(dev(W)), w4.q8_f32_quantize(dev(x))
    wq_ref, xq_ref = oracle.q4_sym_quantize(W), oracle.q8_f32_quantize(x)
    assert np.array_equal(host(wq), wq_ref) and np.array_equal(host(xq), xq_ref)
    y = host(w4.q4sym_q8f32_gemv(wq, xq, N, K))
    y_ref, R = oracle.gemv_sym(wq_ref, xq_ref, N, K)
    assert np.all(np.abs(y - y_ref) <= 1e-5 * R)


def _random_sym_blocks(g, N, K):
    """Random bytes in the Q4_SYM layout: nibbles uniform in 1..15, fp32 scales
    of the magnitude N(0, 0.02^2) weights give (amax / 7)."""
    nb = K // 32
    blk = np.empty((N, nb, 20), np.uint8)
    blk[:, :, 4:] = (g.integers(1, 16, (N, nb, 16)) | (g.integers(1, 16, (N, nb, 16)) << 4))
    d = (g.uniform(0.03, 0.07, (N, nb)) / 7).astype(np.float32)
    blk[:, :, :4] = d[:, :, None].view(np.uint8)
    return blk


@pytest.mark.parametrize("N,K", [(256, 2048), (33, 1024)])
def test_gemv_sym_unit_scales_give_exact_integer_dots(N, K):
    """Every scale 1.0: each partial sum is an integer below 2^24, so the fp32
    result equals the int32 block-dot sum exactly, in any order."""
    g = synth.rng(900 + N)
    w = _random_sym_blocks(g, N, K)
    w[:, :, :4] = np.array([1.0], np.float32).view(np.uint8)
    xq = oracle.q8_f32_quantize(synth.normal_f32(g, (K,))).reshape(K // 32, 36)
    xq[:, :4] = np.array([1.0], np.float32).view(np.uint8)
    y = host(w4.q4sym_q8f32_gemv(dev(w), dev(xq), N, K))
    y_ref, _ = oracle.gemv_sym(w, xq, N, K)
    assert np.array_equal(y.astype(np.float64), y_ref)


def test_gemv_sym_lm_head_shape_sampled_rows():
    """The output projection's shape (N = 151936, K = 2048): 200 sampled rows
    and the first and last rows against the oracle."""
    N, K = 151936, 2048
    g = synth.rng(901)
    w = _random_sym_blocks(g, N, K).reshape(N, -1)
    xq = oracle.q8_f32_quantize(synth.normal_f32(g, (K,)))
    y = host(w4.q4sym_q8f32_gemv(dev(w), dev(xq), N, K))
    rows = np.unique(np.concatenate([[0, N - 1], g.choice(N, 200, replace=False)]))
    y_ref, R = oracle.gemv_sym(w[rows], xq, len(rows), K)
    assert np.all(np.abs(y[rows] - y_ref) <= 1e-5 * R)


def test_gemv_sym_zero_codes_give_zero():
    N, K = 100, 512
    w = np.zeros((N, K // 32, 20), np.uint8)
    w[:, :, :4] = np.array([0.1], np.float32).view(np.uint8)
    w[:, :, 4:] = 0x88
    g = synth.rng(902)
    xq = w4.q8_f32_quantize(dev(synth.normal_f32(g, (K,))))
    assert not host(w4.q4sym_q8f32_gemv(dev(w), xq, N, K)).any()
