"""The exact-integer layers of tests/exact_layers.py on the CPU: their
premises hold (Q8_0 of the activations and of every h block has scale 1.0
and codes equal to the values, h and the output are exact in fp32), and a
single block dot off by one changes the oracle's output, so the GPU pins
built on them see such a mistake."""
import numpy as np

import oracle
from tests import moe_check
from tests.exact_layers import ExactLayer, act_codes, design_rows

H, I = 512, 256


def test_design_rows_hits_targets():
    g = np.random.default_rng(0)
    x = act_codes(g, 2048)
    t = g.integers(-3000, 3000, size=300)
    Q = design_rows(g, x, t)
    assert Q.min() >= 0 and Q.max() <= 15
    assert np.array_equal((Q - 8) @ x, t)
    # dense rows: every code occurs, most positions are not 8
    assert len(np.unique(Q)) == 16 and (Q != 8).mean() > 0.85


def test_exact_layer_premises_and_sensitivity():
    L = ExactLayer(0, H, I, 12, 4, [(3, [0, 1, 2, 3]), (2, [4, 5, -1, 6])], shared=False)
    xq = oracle.q8_0_quantize(L.x)
    d, q = oracle.q8_0_split(xq)
    assert (d == 0x3C00).all() and np.array_equal(q.reshape(L.x.shape).astype(np.float32), L.x)
    r = oracle.moe(L.x, L.ids, L.wts, L.w_gu, L.w_d, None, None, H, I, L.E, L.k)
    pairs = moe_check.valid_pairs(L.ids, L.E, False)
    dh, qh = oracle.q8_0_split(r.hq[pairs].ravel())
    assert (dh == 0x3C00).all()
    assert np.array_equal(qh.reshape(len(pairs), I).astype(np.float32), r.h[pairs])
    g = r.gu[pairs][:, :I]
    assert g.min() >= 20 and g.max() <= 127
    assert np.array_equal(r.out.astype(np.float32).astype(np.float64), r.out)
    # one weight code +1 where the activation is +-1: that gate dot moves by
    # one and the layer output changes
    e = int(L.ids[0, 0])
    pos = int(np.nonzero(np.abs(L.x[0]) == 1)[0][0])
    w = L.w_gu.copy()
    byte = 2 + (pos % 32) % 16
    blk = w[e, 5, 18 * (pos // 32):18 * (pos // 32) + 18]
    lo = (pos % 32) < 16
    nib = (blk[byte] & 0x0F) if lo else (blk[byte] >> 4)
    step = 1 if nib < 15 else -1
    blk[byte] = (blk[byte] + step) if lo else (blk[byte] + (step << 4))
    r2 = oracle.moe(L.x, L.ids, L.wts, w, L.w_d, None, None, H, I, L.E, L.k)
    assert r2.gu[0, 5] - r.gu[0, 5] == step * L.x[0, pos]
    assert not np.array_equal(r2.out, r.out)
