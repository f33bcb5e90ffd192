"""moe_w4a8_forward_noalloc (the entry point for callers that cannot
allocate) against moe_w4a8_forward, through the C ABI: calls in a row on the
library's shared scratch array, each smaller than the one before (a grouped
prefill-sized call, a small batch, then single-token calls that use the
hand-off region behind the grouped call's regions), every output equal byte
for byte to the workspace entry point's on a fresh workspace, and within the
oracle's tolerance."""
import numpy as np
import pytest

import paper_2606_24031_amd as w4
from paper_2606_24031_amd import synth
from tests import moe_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

H, I, E = 2048, 512, 256


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def test_noalloc_matches_workspace_entry_point():
    g = synth.rng(900)
    w_gu = synth.q4_0_random_blocks(g, E * 2 * I, H)
    w_d = synth.q4_0_random_blocks(g, E * H, I)
    s_gu = synth.q4_0_random_blocks(g, 2 * I, H)
    s_d = synth.q4_0_random_blocks(g, H, I)
    d_gu, d_d, d_sgu, d_sd = dev(w_gu), dev(w_d), dev(s_gu), dev(s_d)
    for T, k, bias in ((40, 4, 1.0), (6, 8, 0.0), (1, 8, 0.0), (1, 8, 0.0)):
        print(f"noalloc case T={T} k={k}", flush=True)
        x = synth.normal_f32(g, (T, H))
        ids, wts = synth.routing(g, T, E, k, bias_std=bias)
        if T == 6:
            ids[2, 3] = -1
        assert w4.moe_workspace_size(T, H, I, E, k) <= w4.NOALLOC_SCRATCH_BYTES
        xd, idd, wd = dev(x), dev(ids), dev(wts)
        out_na = torch.empty((T, H), dtype=torch.float32, device="cuda")
        w4.moe_forward_noalloc(xd, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, k, out=out_na)
        ws = w4.moe_workspace(T, H, I, E, k)
        out_ws = w4.moe_forward(xd, idd, wd, d_gu, d_d, d_sgu, d_sd, H, I, E, k, ws)
        torch.cuda.synchronize()
        a, b = out_na.cpu().numpy(), out_ws.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), f"T={T} k={k}"
        lay = w4.moe_workspace_layout(T, H, I, E, k)
        P = T * k + T
        wsn = ws.cpu().numpy()
        h = wsn[lay["h"]:lay["h"] + P * I * 4].view(np.float32).reshape(P, I)
        hq = wsn[lay["hq"]:lay["hq"] + P * (I // 32) * 34].reshape(P, -1)
        moe_check.check_layer(a, h, hq, x, ids, wts, w_gu, w_d, s_gu, s_d, H, I, E, k)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    g = synth.rng(901)
    T, k = 100, 8
    assert w4.moe_workspace_size(T, H, I, E, k) > w4.NOALLOC_SCRATCH_BYTES
    x = dev(synth.normal_f32(g, (T, H)))
    ids, wts = synth.routing(g, T, E, k)
    d = torch.zeros(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(w4.W4A8Error) as ei:
        w4.moe_forward_noalloc(x, dev(ids), dev(wts), d, d, None, None, H, I, E, k)
    assert ei.value.code == w4.ESCRATCH
