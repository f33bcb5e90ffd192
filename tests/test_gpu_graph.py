"""The grouped layer with groups of every tile kind (a few rows on 16-row
tiles, larger ones on 32- and 64-row tiles): parity with the oracle,
run-to-run bit equality, and the same bits from a captured HIP graph
replayed several times with other eager calls in between (GPU)."""
import numpy as np
import pytest

import paper_2606_24031_amd as w4
from paper_2606_24031_amd import synth
from tests import moe_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

H, I, E, K = 2048, 512, 64, 4


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def test_grouped_layer_parity_determinism_and_graph_replays():
    g = synth.rng(4242)
    w_gu, w_d = synth.q4_0_random_blocks(g, E * 2 * I, H), synth.q4_0_random_blocks(g, E * H, I)
    ws_gu, ws_d = synth.q4_0_random_blocks(g, 2 * I, H), synth.q4_0_random_blocks(g, H, I)
    d_gu, d_d, d_sgu, d_sd = dev(w_gu), dev(w_d), dev(ws_gu), dev(ws_d)
    T = 136
    x = synth.normal_f32(g, (T, H))
    ids, wts = synth.routing(g, T, E, K, bias_std=1.5)
    c = np.bincount(ids.ravel(), minlength=E)
    assert ((c > 0) & (c <= 16)).any() and (c > 32).any()   # 16-row and 64-row tiles
    ws = w4.moe_workspace(T, H, I, E, K)
    xd, idd, wd = dev(x), dev(ids), dev(wts)
    out0 = w4.moe_forward(xd, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, K, ws)
    torch.cuda.synchronize()
    lay = w4.moe_workspace_layout(T, H, I, E, K)
    P = T * K + T
    wsn = ws.cpu().numpy()
    h = wsn[lay["h"]:lay["h"] + P * I * 4].view(np.float32).reshape(P, I)
    hq = wsn[lay["hq"]:lay["hq"] + P * (I // 32) * 34].reshape(P, -1)
    o0 = out0.cpu().numpy()
    moe_check.check_layer(o0, h, hq, x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, K)
    out1 = w4.moe_forward(xd, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, K, ws)
    assert np.array_equal(out1.cpu().numpy(), o0)
    out_g = torch.empty((T, H), device="cuda")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        w4.moe_forward(xd, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, K, ws, out=out_g)
    ws2 = w4.moe_workspace(T, H, I, E, K)
    x2 = dev(synth.normal_f32(g, (T, H)))
    for rep in range(3):
        out_g.fill_(0.0)
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out_g.cpu().numpy(), o0), f"replay {rep}"
        w4.moe_forward(x2, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, K, ws2)
        torch.cuda.synchronize()
