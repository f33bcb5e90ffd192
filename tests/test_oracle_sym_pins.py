"""Pins for the oracle of the paper's own block format (Sec. 2.3: symmetric
4-bit weights in {-7..7} with an FP32 scale per group; Sec. 3.3: 8-bit
activations with an FP32 scale, the weight held as the unsigned value in
{1..15}): hand-built blocks (tests/golden/), brute-force search over every
code, the round-trip bound, sign and power-of-two invariants, an
independently written numpy dequantize-then-dot, and closed forms.  CPU only."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name_, vals, hexbytes = [c.strip() for c in line.split("|")]
            rows.append((name_, np.array([float(v) for v in vals.split()], dtype=np.float32),
                         bytes.fromhex(hexbytes)))
    return rows


def _scale(blocks, nbytes):
    """fp32 scales and raw payload of blocks [n, nbytes]."""
    b = np.ascontiguousarray(blocks.reshape(-1, nbytes))
    return b[:, :4].copy().view(np.float32)[:, 0], b[:, 4:]


def _nibbles(payload):
    """[n, 16] bytes -> [n, 32] unsigned nibbles in element order."""
    return np.concatenate([payload & 0x0F, payload >> 4], axis=1).astype(np.int64)


def _blocks(g, n, adversarial=True):
    """n blocks of 32 fp32 values: normal, wide-range, exact halves and ties."""
    x = g.normal(0.0, 1.0, (n, 32)).astype(np.float32)
    if adversarial:
        k = n // 4
        x[:k] *= np.float32(2.0) ** g.integers(-30, 30, (k, 1)).astype(np.float32)
        # values on the code grid and half-way between grid points
        d = np.float32(0.25)
        x[k:2 * k] = (g.integers(-14, 15, (k, 32)) * 0.5 * d).astype(np.float32)
        x[2 * k:2 * k + 4] = 0.0
    return x


# ------------------------------------------------------------ weights
def test_q4_sym_golden_blocks():
    for name, w, want in _golden("q4_sym_blocks.txt"):
        got = oracle.q4_sym_quantize(w).tobytes()
        assert got == want, (name, got.hex(" "), want.hex(" "))


def test_q4_sym_brute_force_codes():
    """Every code is the nearest of the 15 grid points {-7..7} * d to w (ties
    either way), against the stored fp32 scale, in fp64."""
    g = np.random.default_rng(11)
    w = _blocks(g, 4000)
    q = oracle.q4_sym_quantize(w)
    d, pay = _scale(q, oracle.Q4S_BYTES)
    codes = _nibbles(pay) - 8
    assert codes.min() >= -7 and codes.max() <= 7          # nibble 0 never used
    cand = np.arange(-7, 8, dtype=np.float64)
    for i in range(w.shape[0]):
        if d[i] == 0:
            assert np.all(codes[i] == 0)
            continue
        err = np.abs(w[i].astype(np.float64)[:, None] - cand[None, :] * float(d[i]))
        best = err.min(axis=1)
        mine = err[np.arange(32), codes[i] + 7]
        assert np.all(mine <= best + 1e-6 * float(d[i])), i


def test_q4_sym_roundtrip_and_extreme():
    """|w - q d| <= d/2 (plus the rounding of w * (1/d)), the largest |w| maps to
    +-7, and amax / 7 is the stored scale."""
    g = np.random.default_rng(12)
    w = _blocks(g, 4000)
    q = oracle.q4_sym_quantize(w)
    d, pay = _scale(q, oracle.Q4S_BYTES)
    codes = _nibbles(pay) - 8
    amax = np.abs(w).max(axis=1)
    assert np.array_equal(d, (amax / np.float32(7.0)).astype(np.float32))
    live = d > 0
    err = np.abs(w.astype(np.float64) - codes * d[:, None].astype(np.float64))
    assert np.all(err[live] <= d[live, None] * (0.5 + 2.0 ** -20))
    top = np.argmax(np.abs(w), axis=1)
    assert np.all(np.abs(codes[np.arange(len(w)), top])[live] == 7)


def test_q4_sym_invariants():
    """Q(-w) = (d, -q); Q(2^j w) = (2^j d, q); an all-zero block is d = 0 and
    nibble 8 everywhere."""
    g = np.random.default_rng(13)
    w = g.normal(0.0, 0.02, (500, 32)).astype(np.float32)
    q = oracle.q4_sym_quantize(w)
    d, pay = _scale(q, oracle.Q4S_BYTES)
    qn = oracle.q4_sym_quantize(-w)
    dn, payn = _scale(qn, oracle.Q4S_BYTES)
    assert np.array_equal(dn, d)
    assert np.array_equal(_nibbles(payn) - 8, -(_nibbles(pay) - 8))
    for j in (-6, 5):
        q2 = oracle.q4_sym_quantize((w * np.float32(2.0 ** j)).astype(np.float32))
        d2, pay2 = _scale(q2, oracle.Q4S_BYTES)
        assert np.array_equal(d2, (d * np.float32(2.0 ** j)).astype(np.float32))
        assert np.array_equal(pay2, pay)
    z = oracle.q4_sym_quantize(np.zeros((1, 64), np.float32)).reshape(2, -1)
    assert np.all(z[:, :4] == 0) and np.all(z[:, 4:] == 0x88)


def test_q4_sym_tiny_scale_gives_zero_codes():
    """A scale whose fp32 reciprocal overflows gives zero codes (the reading of
    the format for scales below 2^-128); a subnormal but invertible one
    quantizes normally."""
    w = np.zeros(32, np.float32)
    w[3] = np.float32(1e-39)
    q = oracle.q4_sym_quantize(w)
    d, pay = _scale(q, oracle.Q4S_BYTES)
    assert d[0] > 0 and np.all(_nibbles(pay) == 8)
    w[3] = np.float32(2.0 ** -120)
    q = oracle.q4_sym_quantize(w)
    d, pay = _scale(q, oracle.Q4S_BYTES)
    assert _nibbles(pay)[0, 3] == 15


# ------------------------------------------------------------ activations
def test_q8_f32_golden_blocks():
    for name, x, want in _golden("q8_f32_blocks.txt"):
        got = oracle.q8_f32_quantize(x).tobytes()
        assert got == want, (name, got.hex(" "), want.hex(" "))


def test_q8_f32_brute_force_and_bound():
    """Each code is the nearest of the 255 grid points to x (ties either way);
    |x - q d| <= d/2; amax maps to +-127; Q(-x) = (d, -q)."""
    g = np.random.default_rng(14)
    x = _blocks(g, 3000)
    q = oracle.q8_f32_quantize(x)
    d, pay = _scale(q, oracle.Q8F_BYTES)
    codes = pay.view(np.int8).astype(np.int64)
    assert np.array_equal(d, (np.abs(x).max(axis=1) / np.float32(127.0)).astype(np.float32))
    live = d > 0
    xd = x.astype(np.float64)
    err = np.abs(xd - codes * d[:, None].astype(np.float64))
    assert np.all(err[live] <= d[live, None] * (0.5 + 2.0 ** -20))
    # nearest grid point: any other code is at least as far (up to rounding)
    for delta in (-1, 1):
        alt = np.clip(codes + delta, -127, 127)
        erra = np.abs(xd - alt * d[:, None].astype(np.float64))
        assert np.all(err[live] <= erra[live] + 1e-6 * d[live, None])
    top = np.argmax(np.abs(x), axis=1)
    assert np.all(np.abs(codes[np.arange(len(x)), top])[live] == 127)
    qn = oracle.q8_f32_quantize(-x)
    dn, payn = _scale(qn, oracle.Q8F_BYTES)
    assert np.array_equal(dn, d) and np.array_equal(payn.view(np.int8), -pay.view(np.int8))


# ------------------------------------------------------------ products
def _dequant_dot(w, xq, N, K):
    """fp64 dequantize-then-dot written from the block layouts alone."""
    nb = K // 32
    dw, pw = _scale(w.reshape(N * nb, -1), oracle.Q4S_BYTES)
    da, pa = _scale(xq.reshape(nb, -1), oracle.Q8F_BYTES)
    wv = (_nibbles(pw) - 8).astype(np.float64) * dw[:, None].astype(np.float64)
    av = pa.view(np.int8).astype(np.float64) * da[:, None].astype(np.float64)
    return wv.reshape(N, K) @ av.reshape(K)


@pytest.mark.parametrize("N,K", [(1, 32), (7, 256), (33, 2048)])
def test_gemv_sym_matches_dequant_definition(N, K):
    g = np.random.default_rng(15 + K)
    w = oracle.q4_sym_quantize(g.normal(0.0, 0.02, (N, K)).astype(np.float32))
    xq = oracle.q8_f32_quantize(g.normal(0.0, 1.0, K).astype(np.float32))
    y, R = oracle.gemv_sym(w, xq, N, K)
    ref = _dequant_dot(w, xq, N, K)
    assert np.all(np.abs(y - ref) <= 1e-12 * R + 1e-300)
    assert np.all(R > 0)


def test_gemv_sym_closed_forms():
    """All weight nibbles 8 give exactly 0; a single nonzero weight code gives
    one exact product; the block dot equals the integer definition."""
    K, N = 64, 3
    g = np.random.default_rng(16)
    xq = oracle.q8_f32_quantize(g.normal(0.0, 1.0, K).astype(np.float32))
    w = np.zeros((N, K // 32, oracle.Q4S_BYTES), np.uint8)
    w[:, :, :4] = np.frombuffer(np.float32(0.75).tobytes(), np.uint8)
    w[:, :, 4:] = 0x88
    y, R = oracle.gemv_sym(w.reshape(N, -1), xq, N, K)
    assert np.all(y == 0) and np.all(R == 0)
    w[1, 1, 4 + 5] = 0x8F                      # element 32 + 5 of row 1: code +7
    y, R = oracle.gemv_sym(w.reshape(N, -1), xq, N, K)
    da, pa = _scale(xq.reshape(2, -1), oracle.Q8F_BYTES)
    want = 0.75 * float(da[1]) * 7 * int(pa[1].view(np.int8)[5])
    assert y[1] == want and y[0] == 0 and y[2] == 0
    s = oracle.blockdot_sym(w[1, 1], xq.reshape(2, -1)[1])
    assert s == 7 * int(pa[1].view(np.int8)[5])


# ------------------------------------------------------------ the MoE layer
def test_moe_sym_equals_q4_0_layer_on_exact_layers():
    """On a layer whose weights are codes in -7..7 with every scale 1.0 and
    whose activations and h are integers with a largest magnitude of 127 per
    block, both formats describe the same numbers (a Q4_0 block of scale 1.0
    and a symmetric block of scale 1.0 with the same nibbles; Q8_0 and Q8_F32
    both give scale 1.0 and the values as codes), so the layer in the paper's
    format must reproduce the pinned Q4_0 layer exactly: gate/up sums, h, the
    codes of h and the output (routed slots with weights 0.5/1/2, a skipped
    slot, the shared expert)."""
    from tests.exact_layers import ExactLayer
    H, I, E, k = 512, 256, 6, 3
    L = ExactLayer(31, H, I, E, k, [(3, [0, 4, -1])], shared=True, lo=1)
    r0 = oracle.moe(L.x, L.ids, L.wts, L.w_gu, L.w_d, L.ws_gu, L.ws_d, H, I, E, k)
    w_gu, w_d, ws_gu, ws_d = L.sym()
    r1 = oracle.moe_sym(L.x, L.ids, L.wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    assert np.array_equal(r0.out, r1.out) and np.array_equal(r0.R, r1.R)
    assert np.array_equal(r0.gu, r1.gu) and np.array_equal(r0.h, r1.h)
    P = L.x.shape[0] * (k + 1)
    q0 = r0.hq.reshape(P, I // 32, 34)
    q1 = r1.hq.reshape(P, I // 32, 36)
    live = [p for p in range(P) if p >= 3 * k or L.ids.ravel()[p] >= 0]
    assert np.array_equal(q0[live, :, 2:], q1[live, :, 4:])           # the codes
    assert (q0[live, :, 0:2].copy().view(np.uint16) == 0x3C00).all()  # Q8_0 scale 1.0
    assert (q1[live, :, 0:4].copy().view(np.float32) == 1.0).all()    # Q8_F32 scale 1.0
    assert np.abs(r1.out).max() > 1000                                 # not a trivial layer


def _sym_layer(seed, H, I, E, T, k, shared=True):
    from paper_2606_24031_amd import synth
    g = synth.rng(seed)
    w = dict(w_gu=synth.q4_sym_random_blocks(g, E * 2 * I, H),
             w_d=synth.q4_sym_random_blocks(g, E * H, I),
             ws_gu=synth.q4_sym_random_blocks(g, 2 * I, H) if shared else None,
             ws_d=synth.q4_sym_random_blocks(g, H, I) if shared else None)
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, k)
    return w, x, ids, wts


def test_moe_sym_slot_order_and_linearity():
    """Routing invariants of the layer: permuting a token's slots (ids and
    weights together) leaves its output unchanged up to the order of the fp64
    sums; an expert named in two slots with weights a and b equals one slot
    of weight a + b (exact in fp32) and a skipped slot; a skipped slot is
    the same as weight 0."""
    H, I, E, T, k = 256, 256, 5, 3, 3
    w, x, ids, wts = _sym_layer(51, H, I, E, T, k)
    args = (w["w_gu"], w["w_d"], w["ws_gu"], w["ws_d"], H, I, E, k)
    r = oracle.moe_sym(x, ids, wts, *args)
    perm = np.array([2, 0, 1])
    rp = oracle.moe_sym(x, ids[:, perm], wts[:, perm], *args)
    assert np.all(np.abs(rp.out - r.out) <= 1e-12 * r.R)
    ids2 = ids.copy()
    wts2 = wts.copy()
    ids2[:, 1] = ids2[:, 0]
    wts2[:, 0], wts2[:, 1] = 0.25, 0.5
    ra = oracle.moe_sym(x, ids2, wts2, *args)
    ids3, wts3 = ids2.copy(), wts2.copy()
    ids3[:, 1] = -1
    wts3[:, 0] = 0.75
    rb = oracle.moe_sym(x, ids3, wts3, *args)
    assert np.all(np.abs(ra.out - rb.out) <= 1e-12 * ra.R)
    wts4 = wts3.copy()
    wts4[:, 1] = 0.0
    ids4 = ids3.copy()
    ids4[:, 1] = ids2[:, 1]
    rc = oracle.moe_sym(x, ids4, wts4, *args)
    assert np.all(np.abs(rc.out - rb.out) <= 1e-12 * rb.R)
