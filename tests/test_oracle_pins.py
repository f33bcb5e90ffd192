"""Pins for the CPU oracle: each oracle function is tied to something other
than itself -- a library routine (numpy's IEEE fp16 conversion, BLAS matmul),
exact rational arithmetic, brute-force search over all codes, hand-built
blocks (tests/golden/), closed forms and invariants.  CPU only."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2606_24031_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _f16(bits):
    return np.array([bits], dtype=np.uint16).view(np.float16).astype(np.float64)[0]


# ------------------------------------------------------------------ fp16
def test_f16_to_f32_exhaustive():
    """Every one of the 65536 binary16 patterns decodes like numpy's float16."""
    bits = np.arange(65536, dtype=np.uint16)
    got = oracle.f16_bits_to_f32(bits)
    ref = bits.view(np.float16).astype(np.float32)
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite].view(np.uint32), ref[finite].view(np.uint32))
    assert np.all(np.isnan(got[np.isnan(ref)]))
    assert np.array_equal(np.isinf(got), np.isinf(ref))


def test_f32_to_f16_matches_numpy_rne():
    """binary32 -> binary16 RNE (subnormals, ties, overflow) equals numpy's."""
    g = np.random.default_rng(1)
    # random bit patterns across the whole exponent range of interest
    exps = g.integers(90, 150, size=20000).astype(np.uint32)
    mant = g.integers(0, 1 << 23, size=20000).astype(np.uint32)
    sign = g.integers(0, 2, size=20000).astype(np.uint32)
    x = ((sign << 31) | (exps << 23) | mant).view(np.float32)
    # exact ties and boundaries
    specials = [0.0, -0.0, 1.0 + 2**-11, 1.0 + 3 * 2**-11, 2**-25, 3 * 2**-26, 2**-24,
                2**-14 - 2**-26, 65504.0, 65519.99, 65520.0, 1e30, -1e30, 5.96e-8,
                np.inf, -np.inf]
    x = np.concatenate([x, np.array(specials, dtype=np.float32)])
    got = oracle.f32_to_f16_bits(x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


# ------------------------------------------------------------------ Q8_0
def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([c.strip() for c in line.split("|")])
    return rows


def test_q8_0_golden_blocks():
    for name, xs, dbits, codes in _read_golden("q8_0_blocks.txt"):
        x = np.array([float(v) for v in xs.split()], dtype=np.float32)
        out = oracle.q8_0_quantize(x)[0]
        d, q = oracle.q8_0_split(out)
        assert int(d[0]) == int(dbits, 16), name
        assert q[0].tolist() == [int(c) for c in codes.split()], name


def test_q8_0_golden_ramp_exact_rational():
    """Re-derive the ramp codes with exact rational arithmetic (no fp32)."""
    x = [Fraction(i - 16) for i in range(32)]
    d = Fraction(_f16(0x3008))          # fp16(16/127), checked against numpy
    assert np.float16(np.float32(16) / np.float32(127)).view(np.uint16) == 0x3008
    codes = []
    for v in x:
        r = v / d
        n = int(abs(r) + Fraction(1, 2)) * (1 if r >= 0 else -1)   # half away
        codes.append(max(-127, min(127, n)))
    out = oracle.q8_0_quantize(np.array([float(v) for v in x], dtype=np.float32))[0]
    assert oracle.q8_0_split(out)[1][0].tolist() == codes


def _rand_blocks(g, n, scale_exp_range=(-6, 6)):
    """Blocks with widely varying magnitudes, including some exact zeros."""
    x = g.standard_normal((n, 32)).astype(np.float32)
    x *= (2.0 ** g.integers(*scale_exp_range, size=(n, 1))).astype(np.float32)
    x[g.random((n, 32)) < 0.02] = 0.0
    return x


def test_q8_0_invariants():
    g = np.random.default_rng(2)
    x = _rand_blocks(g, 4000)
    out = oracle.q8_0_quantize(x.reshape(1, -1)).reshape(4000, 34)
    d, q = oracle.q8_0_split(out)
    d = d[:, 0]
    q = q[:, 0, :].astype(np.int64)
    df = d.view(np.float16).astype(np.float64)
    assert np.all(np.abs(q) <= 127)
    # amax element maps to +-127
    imax = np.argmax(np.abs(x), axis=1)
    qm = q[np.arange(4000), imax]
    assert np.all(np.abs(qm) == 127)
    assert np.all(np.sign(qm) == np.sign(x[np.arange(4000), imax]))
    # round trip |x - q d| <= d/2, plus the fp32 error of x * fl(1/d)
    err = np.abs(x.astype(np.float64) - q * df[:, None])
    assert np.all(err <= df[:, None] * (0.5 + 127 * 2.0**-22))


def test_q8_0_symmetry_and_power_of_two_scaling():
    g = np.random.default_rng(3)
    x = _rand_blocks(g, 500, (-3, 3))
    base = oracle.q8_0_quantize(x.reshape(1, -1)).reshape(500, 34)
    neg = oracle.q8_0_quantize(-x.reshape(1, -1)).reshape(500, 34)
    db, qb = oracle.q8_0_split(base)
    dn, qn = oracle.q8_0_split(neg)
    assert np.array_equal(db, dn)
    assert np.array_equal(qn.astype(np.int16), -qb.astype(np.int16))
    for j in (-3, 2):
        s = oracle.q8_0_quantize((x * np.float32(2.0**j)).reshape(1, -1)).reshape(500, 34)
        ds, qs = oracle.q8_0_split(s)
        assert np.array_equal(qs, qb)
        assert np.array_equal(ds.view(np.float16).astype(np.float64),
                              db.view(np.float16).astype(np.float64) * 2.0**j)


def test_q8_0_brute_force_codes():
    """Each code is the integer in [-127,127] nearest x/d (either neighbour
    accepted within 1e-5 of a tie, the width of the fp32 rounding of x/d)."""
    g = np.random.default_rng(4)
    x = _rand_blocks(g, 300)
    out = oracle.q8_0_quantize(x.reshape(1, -1)).reshape(300, 34)
    d, q = oracle.q8_0_split(out)
    df = d[:, 0].view(np.float16).astype(np.float64)
    cand = np.arange(-127, 128, dtype=np.float64)
    for b in range(300):
        for i in range(32):
            v = float(x[b, i])
            dist = np.abs(v - cand * df[b])
            best = cand[np.argmin(dist)]
            got = float(q[b, 0, i])
            if got != best:
                r = v / df[b]
                assert abs(abs(r - np.trunc(r)) - 0.5) < 1e-5 and abs(got - best) == 1


def test_q8_0_zero_and_underflow():
    x = np.zeros((2, 32), dtype=np.float32)
    x[1, :] = 1e-9
    out = oracle.q8_0_quantize(x)
    assert not out.any()


# ------------------------------------------------------------------ Q4_0
def test_q4_0_golden_blocks():
    for name, ws, hexbytes in _read_golden("q4_0_blocks.txt"):
        w = np.array([float(v) for v in ws.split()], dtype=np.float32)
        out = oracle.q4_0_quantize(w)[0]
        assert out.tolist() == [int(h, 16) for h in hexbytes.split()], name


def test_q4_0_brute_force_and_extreme():
    """Codes equal the nearest of the 16 levels (q-8)*d (half rounds up, the
    top level clamps at q=15); the extreme element reconstructs to -8 d."""
    g = np.random.default_rng(5)
    w = _rand_blocks(g, 600)
    out = oracle.q4_0_quantize(w.reshape(1, -1)).reshape(600, 18)
    d, q = oracle.q4_0_split(out)
    df = d[:, 0].view(np.float16).astype(np.float64)
    q = q[:, 0, :].astype(np.int64)
    levels = np.arange(16) - 8
    for b in range(600):
        i_star = int(np.argmax(np.abs(w[b])))
        if df[b] != 0:
            assert q[b, i_star] == 0
            assert abs(-8 * df[b] - float(w[b, i_star])) <= abs(df[b]) * 8 * 2.0**-11 * 1.01
        for i in range(32):
            v = float(w[b, i])
            if df[b] == 0:
                assert q[b, i] == 8
                continue
            dist = np.abs(v - levels * df[b])
            best = int(np.argmin(dist))
            if q[b, i] != best:
                r = v / df[b] + 8.0
                near_tie = abs(r - np.floor(r) - 0.5) < 1e-5
                assert near_tie and abs(q[b, i] - best) == 1, (b, i)


def test_q4_0_matches_numpy_reference_on_bits():
    """Nibble order: byte j = element j (low) | element j+16 (high)."""
    g = np.random.default_rng(6)
    w = g.standard_normal((8, 64)).astype(np.float32) * np.float32(0.02)
    out = oracle.q4_0_quantize(w)
    d, q = oracle.q4_0_split(out)
    vals = (q.astype(np.float64) - 8) * d.view(np.float16).astype(np.float64)[..., None]
    err = np.abs(vals.reshape(8, 64) - w)
    bound = np.repeat(np.abs(d.view(np.float16).astype(np.float64)), 32, axis=1)
    assert np.all(err <= bound * (1 + 1e-6))   # <= d/2, or d at the clamped top level


# ------------------------------------------------------------------ dot + gemv
def test_blockdot_against_numpy_decoding():
    g = np.random.default_rng(7)
    wq = synth.q4_0_random_blocks(g, 50, 32)
    x = g.standard_normal((50, 32)).astype(np.float32)
    xq = oracle.q8_0_quantize(x)
    _, qw = oracle.q4_0_split(wq)
    _, qa = oracle.q8_0_split(xq)
    for r in range(50):
        ref = int(np.dot(qw[r, 0].astype(np.int64) - 8, qa[r, 0].astype(np.int64)))
        assert oracle.blockdot(wq[r], xq[r]) == ref


def test_blockdot_closed_forms():
    a = np.zeros(34, np.uint8)
    a[0:2] = np.array([0x3c00], np.uint16).view(np.uint8)
    a[2:] = np.arange(32, dtype=np.int8).view(np.uint8)
    w = np.zeros(18, np.uint8)
    w[2:] = 0x88                        # every code 8 -> weight 0
    assert oracle.blockdot(w, a) == 0
    w[2 + 3] = 0x8B                     # element 3 -> code 11 (+3)
    assert oracle.blockdot(w, a) == 3 * 3
    w[2 + 3] = 0x28                     # element 19 -> code 2 (-6)
    assert oracle.blockdot(w, a) == -6 * 19
    w[2:] = 0x00                        # every code 0 -> -8 each
    a[2:] = np.full(32, 127, np.int8).view(np.uint8)
    assert oracle.blockdot(w, a) == -8 * 127 * 32   # extreme magnitude -32512


@pytest.mark.parametrize("N,K", [(64, 256), (33, 2048), (1024, 1024)])
def test_gemv_matches_dequant_fp64(N, K):
    g = np.random.default_rng(8)
    w = oracle.q4_0_quantize(synth.normal_f32(g, (N, K), 0.02))
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (K,)))
    y, R = oracle.gemv(w, xq, N, K)
    ydq = oracle.gemv_dequant(w, xq, N, K)
    assert np.all(np.abs(y - ydq) <= 1e-12 * R)
    # and numpy's BLAS on the dequantized operands
    dw, qw = oracle.q4_0_split(w.reshape(N, -1))
    da, qa = oracle.q8_0_split(xq.reshape(1, -1))
    Wf = ((qw.astype(np.float64) - 8) * dw.view(np.float16).astype(np.float64)[..., None]).reshape(N, K)
    xf = (qa.astype(np.float64) * da.view(np.float16).astype(np.float64)[..., None]).reshape(K)
    assert np.all(np.abs(Wf @ xf - y) <= 1e-12 * R)


def test_gemv_unit_scale_is_exact_integer_sum():
    g = np.random.default_rng(9)
    N, K = 16, 2048
    w = synth.q4_0_random_blocks(g, N, K).reshape(N, K // 32, 18)
    w[:, :, 0:2] = np.array([0x3c00], np.uint16).view(np.uint8)   # d_w = 1
    xq = oracle.q8_0_quantize(synth.normal_f32(g, (K,))).reshape(K // 32, 34)
    xq[:, 0:2] = np.array([0x3c00], np.uint16).view(np.uint8)     # d_a = 1
    y, _ = oracle.gemv(w, xq, N, K)
    ref = [sum(oracle.blockdot(w[n, b], xq[b]) for b in range(K // 32)) for n in range(N)]
    assert y.tolist() == [float(v) for v in ref]


def test_gemv_all_zero_codes_and_single_term():
    N, K = 4, 256
    w = np.zeros((N, K // 32, 18), np.uint8)
    w[:, :, 0:2] = np.array([0x2e66], np.uint16).view(np.uint8)    # d_w = 0.1
    w[:, :, 2:] = 0x88
    xq = oracle.q8_0_quantize(np.linspace(-3, 3, K, dtype=np.float32))
    y, R = oracle.gemv(w, xq, N, K)
    assert np.all(y == 0) and np.all(R == 0)
    w[1, 3, 2 + 5] = 0x8F                       # row 1, block 3, element 5: +7
    y, _ = oracle.gemv(w, xq, N, K)
    da, qa = oracle.q8_0_split(xq.reshape(1, -1))
    expect = _f16(0x2e66) * float(_f16(int(da[0, 3]))) * 7 * int(qa[0, 3, 5])
    assert y[1] == expect and y[0] == 0 and y[2] == 0


# ------------------------------------------------------------------ MoE layer
def _layer(g, T, H, I, E, k, shared=True, bias=0.0):
    w_gu = oracle.q4_0_quantize(synth.normal_f32(g, (E * 2 * I, H), 0.02)).reshape(E, 2 * I, -1)
    w_d = oracle.q4_0_quantize(synth.normal_f32(g, (E * H, I), 0.02)).reshape(E, H, -1)
    ws_gu = ws_d = None
    if shared:
        ws_gu = oracle.q4_0_quantize(synth.normal_f32(g, (2 * I, H), 0.02))
        ws_d = oracle.q4_0_quantize(synth.normal_f32(g, (H, I), 0.02))
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, k, bias)
    return x, ids, wts, w_gu, w_d, ws_gu, ws_d


def _dequant(wq, rows, K):
    d, q = oracle.q4_0_split(np.asarray(wq).reshape(rows, -1))
    return ((q.astype(np.float64) - 8) * d.view(np.float16).astype(np.float64)[..., None]).reshape(rows, K)


def _deq8(xq, K):
    d, q = oracle.q8_0_split(np.asarray(xq).reshape(1, -1))
    return (q.astype(np.float64) * d.view(np.float16).astype(np.float64)[..., None]).reshape(K)


def _textbook_swiglu(x, Wgu, Wd, H, I):
    """W_d (silu(W_g x) * (W_u x)) with Q8_0 at both quantization points,
    every product in fp64 through numpy's BLAS on dequantized operands."""
    xq = oracle.q8_0_quantize(x)
    gu = (_dequant(Wgu, 2 * I, H) @ _deq8(xq, H)).astype(np.float32)
    g_, u_ = gu[:I].astype(np.float64), gu[I:].astype(np.float64)
    h = (g_ / (1.0 + np.exp(-g_)) * u_).astype(np.float32)
    hq = oracle.q8_0_quantize(h)
    return _dequant(Wd, H, I) @ _deq8(hq, I)


def test_moe_k1_no_shared_is_textbook_swiglu():
    g = np.random.default_rng(10)
    T, H, I, E, k = 3, 256, 256, 4, 1
    x, ids, _, w_gu, w_d, _, _ = _layer(g, T, H, I, E, k, shared=False)
    wts = np.ones((T, k), np.float32)
    r = oracle.moe(x, ids, wts, w_gu, w_d, None, None, H, I, E, k)
    for t in range(T):
        e = ids[t, 0]
        ref = _textbook_swiglu(x[t], w_gu[e], w_d[e], H, I)
        assert np.all(np.abs(r.out[t] - ref) <= 1e-12 * r.R[t])


def test_moe_tiny_brute_force_python_loops():
    """H=64, I=32, E=4, k=2, T=3: every operand dequantized, pure-Python fp64."""
    g = np.random.default_rng(11)
    T, H, I, E, k = 3, 64, 32, 4, 2
    x, ids, wts, w_gu, w_d, ws_gu, ws_d = _layer(g, T, H, I, E, k)
    r = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    for t in range(T):
        xv = _deq8(oracle.q8_0_quantize(x[t]), H).tolist()
        outs = [0.0] * H
        experts = [(int(ids[t, j]), float(wts[t, j])) for j in range(k)] + [(-2, 1.0)]
        for e, wj in experts:
            Wg = _dequant(ws_gu if e == -2 else w_gu[e], 2 * I, H).tolist()
            Wd = _dequant(ws_d if e == -2 else w_d[e], H, I).tolist()
            gu = [float(np.float32(sum(Wg[n][c] * xv[c] for c in range(H)))) for n in range(2 * I)]
            h = np.array([gu[i] / (1.0 + np.exp(-gu[i])) * gu[I + i] for i in range(I)], np.float32)
            hv = _deq8(oracle.q8_0_quantize(h), I).tolist()
            for n in range(H):
                outs[n] += wj * sum(Wd[n][c] * hv[c] for c in range(I))
        assert np.all(np.abs(r.out[t] - np.array(outs)) <= 1e-12 * r.R[t])


def test_moe_routing_special_cases():
    g = np.random.default_rng(12)
    T, H, I, E, k = 4, 256, 256, 5, 3
    x, ids, wts, w_gu, w_d, ws_gu, ws_d = _layer(g, T, H, I, E, k)
    base = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    # slot order does not matter
    perm = [2, 0, 1]
    r = oracle.moe(x, ids[:, perm], wts[:, perm], w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    assert np.all(np.abs(r.out - base.out) <= 1e-14 * base.R)
    # a skipped slot (-1) contributes nothing: equals k-1 routing of the rest
    ids2 = ids.copy(); ids2[:, 2] = -1
    r2 = oracle.moe(x, ids2, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    r2b = oracle.moe(x, ids[:, :2], wts[:, :2], w_gu, w_d, ws_gu, ws_d, H, I, E, 2)
    assert np.array_equal(r2.out, r2b.out)
    # duplicate id counts twice: (w0 + w1) * y_e
    ids3 = ids.copy(); ids3[:, 1] = ids3[:, 0]; ids3[:, 2] = -1
    r3 = oracle.moe(x, ids3, wts, w_gu, w_d, None, None, H, I, E, k)
    r4 = oracle.moe(x, ids3[:, :1], np.ones((T, 1), np.float32), w_gu, w_d, None, None, H, I, E, 1)
    wsum = wts[:, 0].astype(np.float64) + wts[:, 1].astype(np.float64)
    assert np.all(np.abs(r3.out - wsum[:, None] * r4.out) <= 1e-14 * r3.R)
    # all routing weights zero: shared expert only
    r5 = oracle.moe(x, ids, np.zeros_like(wts), w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    for t in range(T):
        ref = _textbook_swiglu(x[t], ws_gu, ws_d, H, I)
        assert np.all(np.abs(r5.out[t] - ref) <= 1e-12 * r5.R[t])
    # all tokens to one expert equals each token through that expert alone
    ids6 = np.full((T, 1), 3, np.int32)
    r6 = oracle.moe(x, ids6, np.ones((T, 1), np.float32), w_gu, w_d, None, None, H, I, E, 1)
    for t in range(T):
        ref = _textbook_swiglu(x[t], w_gu[3], w_d[3], H, I)
        assert np.all(np.abs(r6.out[t] - ref) <= 1e-12 * r6.R[t])


def test_moe_hq_in_overrides_down_input():
    g = np.random.default_rng(13)
    T, H, I, E, k = 2, 256, 256, 3, 2
    x, ids, wts, w_gu, w_d, ws_gu, ws_d = _layer(g, T, H, I, E, k)
    base = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    same = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=base.hq)
    assert np.array_equal(same.out, base.out)
    hq = base.hq.copy().reshape(-1, I // 32, 34)
    hq[0, 0, 2] = (hq[0, 0, 2].view(np.int8) + np.int8(1)).view(np.uint8)   # one code +1
    r = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=hq)
    # the change is exactly w * d_h * (column 0 of expert ids[0,0]'s down weights)
    e = ids[0, 0]
    col = _dequant(w_d[e], H, I)[:, 0]
    dh = _f16(int(oracle.q8_0_split(hq[0].reshape(1, -1))[0][0, 0]))
    assert np.all(np.abs((r.out[0] - base.out[0]) - wts[0, 0] * dh * col) <= 1e-12 * base.R[0])


def test_q8_0_candidates_cover_perturbed_inputs():
    g = np.random.default_rng(14)
    h = synth.normal_f32(g, (512,), 0.5)
    # exact input: the single candidate is Q8_0(h)
    s, lo, hi, ns = oracle.q8_0_candidates(h, np.zeros_like(h))
    d, q = oracle.q8_0_split(oracle.q8_0_quantize(h))
    assert np.all(ns == 1)
    assert np.array_equal(s[:, 0], d[0]) and np.array_equal(lo[:, 0], q[0]) and np.array_equal(hi[:, 0], q[0])
    # perturbed inputs inside the box always land in the candidate set
    dh = np.full_like(h, 2e-4)
    s, lo, hi, ns = oracle.q8_0_candidates(h, dh)
    for _ in range(50):
        hp = (h + g.uniform(-1, 1, h.shape).astype(np.float32) * dh * np.float32(0.999)).astype(np.float32)
        dp, qp = oracle.q8_0_split(oracle.q8_0_quantize(hp))
        for b in range(16):
            c = [i for i in range(ns[b]) if s[b, i] == dp[0, b]]
            assert c, "scale outside the candidate set"
            c = c[0]
            assert np.all(qp[0, b] >= lo[b, c]) and np.all(qp[0, b] <= hi[b, c])


# ------------------------------------------------------------ RMSNorm + residual
def test_rmsnorm_hand_example():
    # x = (3, 4): mean square 12.5, so xn = x / sqrt(12.5 + eps) * gamma
    x = np.array([[3.0, 4.0]], np.float32)
    g = np.array([2.0, -0.5], np.float32)
    xo, xn = oracle.rmsnorm_residual(x, None, g, eps=0.0)
    assert np.array_equal(xo, x)
    r = 12.5 ** -0.5
    assert np.allclose(xn[0], [3 * r * 2.0, 4 * r * -0.5], rtol=1e-15, atol=0)


def test_rmsnorm_constant_row_and_scale_invariance():
    g = np.random.default_rng(31)
    gamma = synth.normal_f32(g, (64,), 1.0)
    # a constant row c: xn = sign(c) * gamma (eps = 0)
    for c in (5.0, -0.25):
        _, xn = oracle.rmsnorm_residual(np.full((1, 64), c, np.float32), None, gamma, eps=0.0)
        assert np.allclose(xn[0], np.sign(c) * gamma.astype(np.float64), rtol=1e-15, atol=0)
    # a power-of-two scaling of the row leaves xn unchanged (exact in fp64)
    x = synth.normal_f32(g, (3, 64))
    _, a = oracle.rmsnorm_residual(x, None, gamma, eps=0.0)
    _, b = oracle.rmsnorm_residual(x * np.float32(8.0), None, gamma, eps=0.0)
    assert np.array_equal(a, b)
    # eps enters under the root: a zero row stays zero, a tiny row is damped
    _, z = oracle.rmsnorm_residual(np.zeros((1, 64), np.float32), None, gamma, eps=1e-6)
    assert not z.any()


def test_rmsnorm_residual_is_one_fp32_add():
    # 1 + 2^-24 rounds to 1 in binary32 (tie to even); 1 + 3*2^-24 rounds up
    x = np.array([[1.0, 1.0, -2.5, 0.0]], np.float32)
    y = np.array([[2.0 ** -24, 3 * 2.0 ** -24, 2.5, -0.0]], np.float32)
    xo, _ = oracle.rmsnorm_residual(x, y, np.ones(4, np.float32), want_norm=False)
    assert xo[0, 0] == np.float32(1.0)
    assert xo[0, 1] == np.float32(1.0 + 2.0 ** -22)
    assert xo[0, 2] == 0.0 and xo[0, 3] == 0.0


# ------------------------------------------------------------------ router top-k
def test_router_hand_example_with_tie():
    """Logits [1, 3, 2, 3], k = 3: the two 3s first (lower index first), then
    the 2; weights e^3 : e^3 : e^2 renormalized, i.e. 1 / (2 + e^-1) twice and
    e^-1 / (2 + e^-1)."""
    ids, w = oracle.router_topk(np.array([[1.0, 3.0, 2.0, 3.0]], np.float32), 3)
    assert ids.tolist() == [[1, 3, 2]]
    c = 2.0 + math.exp(-1.0)
    assert np.allclose(w[0], [1.0 / c, 1.0 / c, math.exp(-1.0) / c], rtol=0, atol=1e-15)


def test_router_matches_library_softmax_and_stable_sort():
    """Against scipy's softmax over all E and numpy's stable argsort: the
    selection is the top k of the probabilities (ties by index) and the
    weights are those probabilities renormalized."""
    from scipy.special import softmax
    g = synth.rng(61)
    for T, E, k in ((9, 256, 8), (5, 7, 7), (3, 130, 32), (4, 64, 1)):
        logits = synth.normal_f32(g, (T, E))
        logits[0, :] = np.round(logits[0, :])          # many equal logits in one row
        ids, w = oracle.router_topk(logits, k)
        p = softmax(logits.astype(np.float64), axis=1)
        order = np.argsort(-logits.astype(np.float64), axis=1, kind="stable")[:, :k]
        assert np.array_equal(ids, order)
        ref = np.take_along_axis(p, order, axis=1)
        ref /= ref.sum(axis=1, keepdims=True)
        assert np.allclose(w, ref, rtol=1e-12, atol=0)


def test_router_invariants_and_special_cases():
    g = synth.rng(62)
    logits = synth.normal_f32(g, (16, 256))
    ids, w = oracle.router_topk(logits, 8)
    assert np.allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    for t in range(16):
        assert len(set(ids[t].tolist())) == 8
        sel = logits[t, ids[t]]
        assert np.all(np.diff(sel) <= 0) and np.all(np.diff(w[t]) <= 0)
        assert sel[-1] >= np.max(np.delete(logits[t], ids[t]))
    # shift invariance (a power-of-two shift keeps the fp32 differences exact)
    ids2, w2 = oracle.router_topk(logits + np.float32(4.0), 8)
    assert np.array_equal(ids, ids2)
    assert np.allclose(w, w2, rtol=1e-6, atol=0)
    # equal logits: the first k experts, uniform weights; k = 1: weight 1
    ids3, w3 = oracle.router_topk(np.zeros((2, 10), np.float32), 4)
    assert ids3.tolist() == [[0, 1, 2, 3]] * 2 and np.all(w3 == 0.25)
    ids4, w4 = oracle.router_topk(logits, 1)
    assert np.array_equal(ids4[:, 0], np.argmax(logits, axis=1)) and np.all(w4 == 1.0)


def test_moe_shared_weight_is_linear():
    """out(s) = out(s=0) + s * (out(s=1) - out(s=0)) per token for the shared
    expert's weight s, and s = 1 is the ungated layer."""
    g = synth.rng(63)
    T, H, I, E, k = 3, 256, 256, 4, 2
    w_gu = synth.q4_0_random_blocks(g, E * 2 * I, H)
    w_d = synth.q4_0_random_blocks(g, E * H, I)
    ws_gu = synth.q4_0_random_blocks(g, 2 * I, H)
    ws_d = synth.q4_0_random_blocks(g, H, I)
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, k)
    f = lambda s: oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, shared_w=s,
                             want_intermediates=False)
    base = f(None)
    r0, r1 = f(np.zeros(T)), f(np.ones(T))
    s = np.array([0.25, 0.5, 2.0])
    rs = f(s)
    assert np.array_equal(r1.out, base.out) and np.array_equal(r1.R, base.R)
    assert np.allclose(rs.out, r0.out + s[:, None] * (r1.out - r0.out), rtol=0, atol=1e-12 * base.R.max())


def _f32_values(lo, hi):
    """Every fp32 value v with lo <= v <= hi (both fp32), in order."""
    def key(v):
        i = int(np.array([v], np.float32).view(np.int32)[0])
        return i if i >= 0 else -(i & 0x7FFFFFFF)
    k0, k1 = key(lo), key(hi)
    keys = np.arange(k0, k1 + 1, dtype=np.int64)
    bits = np.where(keys >= 0, keys, (-keys) | 0x80000000).astype(np.uint32)
    return bits.view(np.float32)


def _code_f32(v, df):
    """Q8_0 code of fp32 values v for the fp32 scale df, written from the
    format definition in numpy fp32: one multiply by 1/df, round half away
    from zero, clamp to +-127."""
    idf = np.float32(1.0) / np.float32(df)
    p = (v.astype(np.float32) * idf).astype(np.float64)
    r = np.sign(p) * np.floor(np.abs(p) + 0.5)
    return np.clip(r, -127, 127).astype(np.int64)


def test_q8_0_candidates_are_tight():
    """Tightness, not only coverage: for boxes of a few ulps placed on code
    ties (x / d at c + 1/2) and on fp16 rounding boundaries of the scale, the
    scale set and every per-element code interval equal what an independent
    enumeration of every fp32 value in the box gives (numpy fp16 conversion,
    numpy fp32 arithmetic): no listed scale or code is unreachable and none
    reachable is missing."""
    g = np.random.default_rng(15)
    nb = 24
    h = synth.normal_f32(g, (nb * 32,), 0.5)
    dh = np.zeros_like(h)
    ulp = lambda v: np.spacing(np.abs(np.float32(v))).astype(np.float32)
    d0, _ = oracle.q8_0_split(oracle.q8_0_quantize(h))
    for b in range(nb):
        blk = slice(32 * b, 32 * b + 32)
        x = h[blk]
        df = float(np.array([d0[0, b]], np.uint16).view(np.float16)[0])
        amax_i = int(np.argmax(np.abs(x)))
        # three elements on code ties c + 1/2, boxes of a few ulps
        for i in g.choice([j for j in range(32) if j != amax_i], 3, replace=False):
            c = int(g.integers(-100, 100))
            x[i] = np.float32((c + 0.5) * df)
            dh[32 * b + i] = np.float32(int(g.integers(1, 5))) * ulp(x[i])
        # three elements whose box of n ulps stops one ulp short of a tie
        # (a box even slightly too wide would reach it)
        for i in g.choice([j for j in range(32) if j != amax_i and dh[32 * b + j] == 0], 3,
                          replace=False):
            c = int(g.integers(-100, 100))
            tie = np.float32((c + 0.5) * df)
            n = int(g.integers(1, 4))
            side = 1 if g.random() < 0.5 else -1
            v = tie
            for _ in range(n + 1):
                v = np.nextafter(v, np.float32(side * np.inf))
            x[i] = v
            dh[32 * b + i] = np.float32(n) * ulp(v)
        # some other elements get a one-ulp box, the rest none
        for i in g.choice(32, 6, replace=False):
            if dh[32 * b + i] == 0 and i != amax_i:
                dh[32 * b + i] = ulp(x[i])
        if b % 2 == 0:
            # amax on an fp16 rounding boundary of amax / 127: two scales
            s = np.float16(np.float32(abs(x[amax_i])) / np.float32(127))
            s_next = np.nextafter(s, np.float16(np.inf))
            mid = (float(s) + float(s_next)) / 2.0
            x[amax_i] = np.float32(np.sign(x[amax_i]) * mid * 127.0)
            dh[32 * b + amax_i] = np.float32(3) * ulp(x[amax_i])
        elif b % 4 == 1:
            # amax two ulps past an fp16 rounding boundary, a one-ulp box:
            # one scale, unless the box is too wide
            s = np.float16(np.float32(abs(x[amax_i])) / np.float32(127))
            s_next = np.nextafter(s, np.float16(np.inf))
            mid = np.float32((float(s) + float(s_next)) / 2.0 * 127.0)
            while np.float16(mid / np.float32(127)) == s:      # first fp32 past the boundary
                mid = np.nextafter(mid, np.float32(np.inf))
            v = np.nextafter(np.nextafter(mid, np.float32(np.inf)), np.float32(np.inf))
            x[amax_i] = np.float32(np.sign(x[amax_i]) * v)
            dh[32 * b + amax_i] = ulp(v)
        h[blk] = x
    scales, qlo, qhi, ns = oracle.q8_0_candidates(h, dh)
    lo_box = (h.astype(np.float64) - dh.astype(np.float64)).astype(np.float32)
    hi_box = (h.astype(np.float64) + dh.astype(np.float64)).astype(np.float32)
    multi = 0
    for b in range(nb):
        el = range(32 * b, 32 * b + 32)
        vals = [_f32_values(lo_box[i], hi_box[i]) for i in el]
        amin = max(float(np.min(np.abs(v))) for v in vals)
        amaxv = max(float(np.max(np.abs(v))) for v in vals)
        a = _f32_values(np.float32(amin), np.float32(amaxv))
        s_enum = np.unique((a / np.float32(127)).astype(np.float32).astype(np.float16).view(np.uint16))
        assert list(s_enum) == list(scales[b, :ns[b]]), f"block {b}: scale set"
        multi += ns[b] > 1
        for c in range(ns[b]):
            df = np.array([scales[b, c]], np.uint16).view(np.float16).astype(np.float32)[0]
            for j, i in enumerate(el):
                codes = np.unique(_code_f32(vals[j], df))
                want = np.arange(int(qlo[b, c, j]), int(qhi[b, c, j]) + 1)
                assert np.array_equal(codes, want), f"block {b} scale {c} element {j}"
    assert multi >= nb // 2 - 2, "the boxes were meant to straddle scale boundaries"
    assert (qhi > qlo).sum() >= 2 * nb, "the boxes were meant to straddle code ties"
