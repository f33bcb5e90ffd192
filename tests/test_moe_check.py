"""The MoE-layer parity checker (tests/moe_check.py) on the CPU: it accepts
the oracle's own intermediates as a stand-in for a GPU result, and it rejects
each kind of planted mistake (the mistakes are planted in that stand-in)."""
import numpy as np
import pytest

import oracle
from paper_2606_24031_amd import synth
from tests import moe_check

H, I, E, K = 256, 256, 4, 2


@pytest.fixture(scope="module")
def case():
    g = synth.rng(3)
    T = 3
    w_gu = synth.q4_0_random_blocks(g, E * 2 * I, H)
    w_d = synth.q4_0_random_blocks(g, E * H, I)
    ws_gu = synth.q4_0_random_blocks(g, 2 * I, H)
    ws_d = synth.q4_0_random_blocks(g, H, I)
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, K)
    r = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, K)
    return dict(x=x, ids=ids, wts=wts, w_gu=w_gu, w_d=w_d, ws_gu=ws_gu, ws_d=ws_d,
                out=r.out.astype(np.float32), h=r.h.copy(), hq=r.hq.copy())


def _check(c, out=None, h=None, hq=None, **kw):
    return moe_check.check_layer(c["out"] if out is None else out, c["h"] if h is None else h,
                                 c["hq"] if hq is None else hq, c["x"], c["ids"], c["wts"],
                                 c["w_gu"], c["w_d"], c["ws_gu"], c["ws_d"], H, I, E, K, **kw)


def test_accepts_the_oracles_own_result(case):
    st = _check(case, max_flips=0)
    assert st["flips"] == 0 and st["pairs"] == 3 * K + 3


def test_rejects_q8_0_not_of_own_h(case):
    hq = case["hq"].copy().reshape(-1, I // 32, 34)
    hq[1, 2, 5] ^= 1                                # one code, h unchanged
    with pytest.raises(AssertionError, match="Q8_0 of the GPU's own h"):
        _check(case, hq=hq.reshape(case["hq"].shape))


def test_rejects_h_outside_its_bound(case):
    h = case["h"].copy()
    h[2, 7] = np.float32(h[2, 7] * 1.01 + 0.01)     # far outside the tolerance
    hq = case["hq"].copy()
    hq[2] = oracle.q8_0_quantize(h[2])[0]           # consistent with the planted h
    with pytest.raises(AssertionError, match="h of pair"):
        _check(case, h=h, hq=hq)


def test_counts_and_bounds_flips(case):
    # h one ulp-scale step off at a value whose code then flips: pick the
    # element closest to a rounding tie and push it across within the bound
    d, q = oracle.q8_0_split(case["hq"][0])
    df = np.array(d, np.uint16).view(np.float16).astype(np.float32)
    v = case["h"][0].reshape(-1, 32) / df[:, None]
    frac = np.abs(np.abs(v) - np.floor(np.abs(v)) - 0.5)
    b, i = np.unravel_index(np.argmin(frac), frac.shape)
    h = case["h"].copy()
    hv = h[0, 32 * b + i]
    tie = np.float32(np.sign(hv) * (np.floor(abs(float(hv) / df[b])) + 0.5) * df[b])
    # the other side of the tie, by the same distance, must stay inside the
    # bound the float tolerance allows for h
    r = oracle.moe(case["x"], case["ids"], case["wts"], case["w_gu"], case["w_d"],
                   case["ws_gu"], case["ws_d"], H, I, E, K)
    dh = moe_check.delta_h(r.gu[0], r.Rgu[0], I)[32 * b + i]
    if 2 * abs(float(hv) - float(tie)) >= dh:
        pytest.skip("no element close enough to a tie in this draw")
    h[0, 32 * b + i] = np.float32(2 * tie - hv)
    hq = case["hq"].copy()
    hq[0] = oracle.q8_0_quantize(h[0])[0]
    if np.array_equal(hq[0], case["hq"][0]):
        pytest.skip("the mirrored value quantizes alike")
    out = oracle.moe(case["x"], case["ids"], case["wts"], case["w_gu"], case["w_d"],
                     case["ws_gu"], case["ws_d"], H, I, E, K, hq_in=hq,
                     want_intermediates=False).out.astype(np.float32)
    st = _check(case, out=out, h=h, hq=hq)
    assert st["flips"] >= 1
    with pytest.raises(AssertionError, match="differ from the oracle's choice"):
        _check(case, out=out, h=h, hq=hq, max_flips=0)


def test_rejects_output_beyond_tolerance(case):
    out = case["out"].copy()
    out[1, 100] += np.float32(1e-3) * np.abs(out[1]).max()
    with pytest.raises(AssertionError, match="outputs beyond"):
        _check(case, out=out)
