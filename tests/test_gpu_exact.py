"""Bit-exact int32 block dots through every MoE kernel family (GPU).

On the layers of tests/exact_layers.py every block dot is an integer, every
scale 1.0 and every scaled sum exact in fp32, so the GPU's fp32 h, its Q8_0(h)
bytes and the layer output must equal the oracle's bit for bit: a block dot
off by one in any kernel -- the single-token decode kernel, the small-group
VALU kernels or the int8 MFMA tiles (64-, 32- and 16-row), gate/up or down --
changes them.
"""
import numpy as np
import pytest

import oracle
import paper_2606_24031_amd as w4
from tests import moe_check
from tests.exact_layers import ExactLayer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = "cuda"
H, I = 2048, 512


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_exact(L, ws=None):
    T, E, k = L.x.shape[0], L.E, L.k
    if ws is None:
        ws = w4.moe_workspace(T, H, I, E, k)
    sgu = None if L.ws_gu is None else dev(L.ws_gu)
    sd = None if L.ws_d is None else dev(L.ws_d)
    out = w4.moe_forward(dev(L.x), dev(L.ids), dev(L.wts), dev(L.w_gu), dev(L.w_d), sgu, sd,
                         H, I, E, k, ws)
    torch.cuda.synchronize()
    lay = w4.moe_workspace_layout(T, H, I, E, k)
    P = T * k + T
    wsn = ws.cpu().numpy()
    h = wsn[lay["h"]:lay["h"] + P * I * 4].view(np.float32).reshape(P, I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (I // 32) * 34].reshape(P, -1)
    assert not wsn[lay["sync"]:lay["sync_end"]].any(), "sync words not back to zero"
    check_exact(L, out.cpu().numpy(), h, hq)
    return ws


def check_exact(L, out, h, hq):
    E, k = L.E, L.k
    r = oracle.moe(L.x, L.ids, L.wts, L.w_gu, L.w_d, L.ws_gu, L.ws_d, H, I, E, k)
    pairs = moe_check.valid_pairs(L.ids, E, L.ws_gu is not None)
    # the premises of exactness, on the oracle's side
    d, _ = oracle.q8_0_split(r.hq[pairs].ravel())
    assert (d == 0x3C00).all(), "every h block should have scale 1.0"
    assert np.array_equal(r.out.astype(np.float32).astype(np.float64), r.out)
    assert np.array_equal(r.h[pairs], np.rint(r.h[pairs]))
    # bit for bit
    assert np.array_equal(h[pairs].view(np.uint32), r.h[pairs].view(np.uint32)), "h"
    assert np.array_equal(hq[pairs], r.hq[pairs]), "Q8_0(h)"
    assert np.array_equal(out.astype(np.float64), r.out), "layer output"


def test_exact_decode_single_token():
    """T = 1: the single-launch decode kernel (gate/up items, down slabs,
    in-workgroup combine); then the same workspace with a repeated expert and
    a skipped slot."""
    L = ExactLayer(1, H, I, 16, 8, [(1, [3, 0, 7, 12, 5, 9, 1, 14])], shared=True)
    ws = run_exact(L)
    L2 = ExactLayer(2, H, I, 16, 8, [(1, [3, 3, -1, 12, 5, 9, 1, 14])], shared=True)
    run_exact(L2, ws=ws)


def test_exact_small_group_path():
    """T <= 128: every group on the VALU kernels in chunks of 8 rows -- three
    clusters of 8 tokens on disjoint experts, and one cluster of 20 tokens
    (chunks 8, 8, 4) with the shared expert."""
    L = ExactLayer(3, H, I, 24, 8, [(8, list(range(0, 8))), (8, list(range(8, 16))),
                                    (8, list(range(16, 24)))], shared=False)
    run_exact(L)
    L2 = ExactLayer(4, H, I, 8, 8, [(20, list(range(8)))], shared=True)
    run_exact(L2)


def test_exact_mfma_path():
    """T > 128, every group on the int8 MFMA tiles: with 128 experts (88 of
    them unused) the route cuts 64-row tiles -- groups of 40 rows (one tile,
    both 32-row halves), 70 rows (a full 64-row tile and a 6-row tile on the
    16x16x32 products), 5 and 16 rows (16-row tiles) and 17 rows (a 32-row
    half); then one cluster of 150 tokens over 8 experts with the shared
    expert, so few tiles that the route cuts 32-row ones (four full tiles and
    a 22-row tile per group)."""
    L = ExactLayer(5, H, I, 128, 8, [(40, list(range(0, 8))), (70, list(range(8, 16))),
                                    (5, list(range(16, 24))), (16, list(range(24, 32))),
                                    (17, list(range(32, 40)))], shared=False)
    run_exact(L)
    L2 = ExactLayer(6, H, I, 8, 8, [(150, list(range(8)))], shared=True)
    run_exact(L2)
