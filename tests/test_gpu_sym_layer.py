"""The MoE layer in the paper's own format (moe_sym_forward: Q4_SYM weights,
Q8_F32 activations and h) against the oracle's layer in that format (GPU):
the full layer shape at one token with top-8 and top-4 of 256 and with 128
routed experts, a few tokens without a shared expert and with skipped slots,
and an exact-integer layer that must match bit for bit."""
import numpy as np
import pytest

import oracle
import paper_2606_24031_amd as w4
from paper_2606_24031_amd import synth
from tests import moe_check
from tests.exact_layers import ExactLayer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def run_sym(x, ids, wts, w, H, I, E, k):
    T = x.shape[0]
    ws = w4.moe_sym_workspace(T, H, I, E, k)
    sgu = None if w["ws_gu"] is None else dev(w["ws_gu"])
    sd = None if w["ws_d"] is None else dev(w["ws_d"])
    out = w4.moe_sym_forward(dev(x), dev(ids), dev(wts), dev(w["w_gu"]), dev(w["w_d"]), sgu, sd,
                             H, I, E, k, ws)
    torch.cuda.synchronize()
    lay = w4.moe_sym_workspace_layout(T, H, I, E, k)
    P = T * k + T
    wsn = ws.cpu().numpy()
    h = wsn[lay["h"]:lay["h"] + P * I * 4].view(np.float32).reshape(P, I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (I // 32) * 36].reshape(P, -1)
    xq = wsn[lay["xq"]:lay["xq"] + T * (H // 32) * 36].reshape(T, -1)
    assert np.array_equal(xq, oracle.q8_f32_quantize(x)), "Q8_F32(x)"
    return out.cpu().numpy(), h, hq


@pytest.fixture(scope="module")
def full_layer():
    H, I, E = 2048, 512, 256
    g = synth.rng(61)
    return dict(w_gu=synth.q4_sym_random_blocks(g, E * 2 * I, H),
                w_d=synth.q4_sym_random_blocks(g, E * H, I),
                ws_gu=synth.q4_sym_random_blocks(g, 2 * I, H),
                ws_d=synth.q4_sym_random_blocks(g, H, I))


@pytest.mark.parametrize("E,k", [(256, 8), (256, 4), (128, 8)])
def test_sym_layer_full_shape_one_token(full_layer, E, k):
    H, I = 2048, 512
    w = dict(full_layer)
    if E < 256:
        w["w_gu"] = w["w_gu"].reshape(256, -1)[:E].reshape(-1)
        w["w_d"] = w["w_d"].reshape(256, -1)[:E].reshape(-1)
    g = synth.rng(62 + E + k)
    x = synth.normal_f32(g, (1, H))
    ids, wts = synth.routing(g, 1, E, k)
    out, h, hq = run_sym(x, ids, wts, w, H, I, E, k)
    st = moe_check.check_sym_layer(out, h, hq, x, ids, wts, w["w_gu"], w["w_d"], w["ws_gu"],
                                   w["ws_d"], H, I, E, k)
    assert st["pairs"] == k + 1


def test_sym_layer_tokens_no_shared_skipped_slots():
    """Five tokens, no shared expert, a skipped slot and a repeated expert;
    I = 768 (three groups of eight blocks in the down rows)."""
    H, I, E, k, T = 1024, 768, 12, 4, 5
    g = synth.rng(63)
    w = dict(w_gu=synth.q4_sym_random_blocks(g, E * 2 * I, H),
             w_d=synth.q4_sym_random_blocks(g, E * H, I), ws_gu=None, ws_d=None)
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, k)
    ids[1, 2] = -1
    ids[3, 1] = ids[3, 0]
    out, h, hq = run_sym(x, ids, wts, w, H, I, E, k)
    moe_check.check_sym_layer(out, h, hq, x, ids, wts, w["w_gu"], w["w_d"], None, None,
                              H, I, E, k)


def test_sym_layer_exact_integer_layer():
    """Every scale 1.0, integer activations and h with block maxima 127: the
    GPU's h, Q8_F32(h) and output equal the oracle's bit for bit (a block dot
    off by one anywhere changes them)."""
    H, I, E, k = 2048, 512, 8, 4
    L = ExactLayer(64, H, I, E, k, [(3, [1, 5, -1, 7])], shared=True, lo=1)
    w_gu, w_d, ws_gu, ws_d = L.sym()
    w = dict(w_gu=w_gu, w_d=w_d, ws_gu=ws_gu, ws_d=ws_d)
    out, h, hq = run_sym(L.x, L.ids, L.wts, w, H, I, E, k)
    r = oracle.moe_sym(L.x, L.ids, L.wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    pairs = moe_check.valid_pairs(L.ids, E, True)
    assert np.array_equal(h[pairs].view(np.uint32), r.h[pairs].view(np.uint32)), "h"
    assert np.array_equal(hq[pairs], r.hq[pairs]), "Q8_F32(h)"
    assert np.array_equal(out.astype(np.float64), r.out), "layer output"
