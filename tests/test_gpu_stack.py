"""The chained stack of pre-norm residual MoE layers (x <- x + MoE_l(RMSNorm_l(x)),
one moe_w4a8_layer call per layer) at the paper's layer shape, on the GPU.

Per sampled layer (first, middle, last) the layer is teacher-forced against
the oracle on the GPU's own inputs to that layer: x_out = x + y_prev bit-exact,
the normalized row within fp32 rounding, Q8_0 of it bit-exact, and the layer
output through the MoE check.  Then the oracle runs the whole chain on its
own and the end-to-end difference of the final residual stream is reported
(drift, not pass/fail: the paper finds W4A8 bit-stable on short runs and
diverging only on long greedy chains)."""
import numpy as np
import pytest

import oracle
import paper_2606_24031_amd as w4
from paper_2606_24031_amd import synth
from tests import moe_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

H, I, E, K = 2048, 512, 256, 8
NL = 5
SAMPLED = (0, NL // 2, NL - 1)
DRIFT = []


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


@pytest.fixture(scope="module")
def stack():
    g = synth.rng(700)
    layers = []
    for _ in range(NL):
        lay = dict(w_gu=synth.q4_0_random_blocks(g, E * 2 * I, H),
                   w_d=synth.q4_0_random_blocks(g, E * H, I),
                   ws_gu=synth.q4_0_random_blocks(g, 2 * I, H),
                   ws_d=synth.q4_0_random_blocks(g, H, I),
                   gamma=(np.float32(1.0) + synth.normal_f32(g, (H,), 0.1)).astype(np.float32))
        lay["dev"] = [dev(lay[n]) for n in ("w_gu", "w_d", "ws_gu", "ws_d", "gamma")]
        layers.append(lay)
    return layers, g


def _oracle_chain(layers, x0, routing):
    """The oracle's own stack: residual adds in fp32, the norm in fp64
    rounded to fp32 as the layer input, the layer in fp64 rounded to fp32."""
    x, y = x0, None
    for l, lay in enumerate(layers):
        ids, wts = routing[l]
        x, xn = oracle.rmsnorm_residual(x, y, lay["gamma"], eps=1e-6)
        r = oracle.moe(xn.astype(np.float32), ids, wts, lay["w_gu"], lay["w_d"], lay["ws_gu"],
                       lay["ws_d"], H, I, E, K, want_intermediates=False)
        y = r.out.astype(np.float32)
    x, _ = oracle.rmsnorm_residual(x, y, layers[0]["gamma"], eps=1e-6, want_norm=False)
    return x


@pytest.mark.parametrize("T,bias", [(1, 0.0), (40, 1.0)])
def test_stack_sampled_layers_teacher_forced(stack, T, bias):
    """T = 1: the norm and the layer in the single decode launch; T = 40: the
    norm kernel, then the grouped path (small-group and MFMA kernels)."""
    layers, g = stack
    x0 = synth.normal_f32(g, (T, H))
    routing = [synth.routing(g, T, E, K, bias_std=bias) for _ in range(NL)]
    ws = w4.moe_workspace(T, H, I, E, K)
    lay_off = w4.moe_workspace_layout(T, H, I, E, K)
    P = T * K + T
    xs = [dev(x0), torch.empty((T, H), device="cuda")]
    ys = [torch.empty((T, H), device="cuda") for _ in range(2)]
    for l, lay in enumerate(layers):
        print(f"stack T={T} layer {l}", flush=True)
        ids, wts = routing[l]
        w_gu, w_d, s_gu, s_d, gam = lay["dev"]
        x_in = xs[l % 2].cpu().numpy()
        y_in = ys[(l + 1) % 2].cpu().numpy() if l else None
        w4.moe_layer(xs[l % 2], ys[(l + 1) % 2] if l else None, gam, dev(ids), dev(wts),
                     w_gu, w_d, s_gu, s_d, H, I, E, K, ws, x_out=xs[(l + 1) % 2],
                     out=ys[l % 2])
        torch.cuda.synchronize()
        if l not in SAMPLED:
            continue
        x_out = xs[(l + 1) % 2].cpu().numpy()
        out = ys[l % 2].cpu().numpy()
        wsn = ws.cpu().numpy()
        xn = wsn[lay_off["xn"]:lay_off["xn"] + T * H * 4].view(np.float32).reshape(T, H)
        xo_ref, xn_ref = oracle.rmsnorm_residual(x_in, y_in, lay["gamma"], eps=1e-6)
        assert np.array_equal(x_out, xo_ref), f"layer {l}: x + y_prev"
        err = np.abs(xn.astype(np.float64) - xn_ref)
        assert np.all(err <= 2e-6 * np.abs(xn_ref) + 1e-7 * np.abs(lay["gamma"]).max())
        xq = wsn[lay_off["xq"]:lay_off["xq"] + T * (H // 32) * 34].reshape(T, -1)
        assert np.array_equal(xq, oracle.q8_0_quantize(xn)), f"layer {l}: Q8_0 of the norm"
        h = wsn[lay_off["h"]:lay_off["h"] + P * I * 4].view(np.float32).reshape(P, I)
        hq = wsn[lay_off["hq"]:lay_off["hq"] + P * (I // 32) * 34].reshape(P, -1)
        moe_check.check_layer(out, h, hq, xn, ids, wts, lay["w_gu"], lay["w_d"], lay["ws_gu"],
                              lay["ws_d"], H, I, E, K, max_flips=0 if T == 1 else None)
    # the final residual stream, x + the last layer's output, against the
    # oracle's own chain from the same x0 (reported, not asserted)
    xf = xs[NL % 2].cpu().numpy() + ys[(NL - 1) % 2].cpu().numpy()
    xr = _oracle_chain(layers, x0, routing)
    d = np.linalg.norm(xf.astype(np.float64) - xr, axis=1) / np.linalg.norm(xr, axis=1)
    rel = float(d.max())
    DRIFT.append((T, NL, rel))
    print(f"stack drift T={T}, {NL} layers: max over tokens of |x_gpu - x_oracle|_2 / "
          f"|x_oracle|_2 = {rel:.3g}", flush=True)
    assert np.isfinite(xf).all()
