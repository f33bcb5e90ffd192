"""The C ABI library loads, exports every entry point include/w4a8.h declares,
and rejects bad arguments on the host (these paths return before any device
call, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2606_24031_amd as w4

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "w4a8.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_0-9]+)\s*\(", src)) - {"defined"})


def test_header_declares_the_binding_exports():
    assert _declared() == sorted(w4.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = w4.lib()
    for name in _declared():
        assert hasattr(lib, name), name


def test_strerror_covers_every_code():
    for code in (w4.OK, w4.ENULL, w4.ESHAPE, w4.ERANGE, w4.EWORKSPACE, w4.EALIGN, w4.EHIP, w4.EDEVICE,
                 w4.EALIAS, w4.ESCRATCH):
        msg = w4.strerror(code)
        assert msg and msg != "unknown status code"
    assert w4.strerror(12345) == "unknown status code"


def _fake(addr):
    return ctypes.c_void_p(addr)


A = 0x10000   # an aligned fake device address (never dereferenced: validation fails first)


def test_quantize_argument_errors():
    L = w4.lib()
    for fn in (L.q8_0_quantize, L.q4_0_quantize, L.q4_sym_quantize, L.q8_f32_quantize):
        assert fn(None, _fake(A), 4, 64, None) == w4.ENULL
        assert fn(_fake(A), None, 4, 64, None) == w4.ENULL
        assert fn(_fake(A), _fake(A), 4, 48, None) == w4.ESHAPE
        assert fn(_fake(A), _fake(A), -1, 64, None) == w4.ESHAPE
        assert fn(_fake(A), _fake(A), 4, 0, None) == w4.ESHAPE
        assert fn(_fake(A + 4), _fake(A), 4, 64, None) == w4.EALIGN
        assert fn(_fake(A), _fake(A), 0, 64, None) == w4.OK       # empty: no-op
        assert fn(_fake(A), _fake(A), 1 << 40, 64, None) == w4.ERANGE


def test_gemv_argument_errors():
    L = w4.lib()
    y = _fake(A)
    assert L.q4q8_gemv(None, _fake(A), y, 8, 256, None) == w4.ENULL
    assert L.q4q8_gemv(_fake(A), _fake(A), y, 8, 128, None) == w4.ESHAPE   # K % 256
    assert L.q4q8_gemv(_fake(A), _fake(A), y, 0, 256, None) == w4.ESHAPE
    assert L.q4q8_gemv(_fake(A), _fake(A + 2), y, 8, 256, None) == w4.EALIGN
    G = L.q4sym_q8f32_gemv
    assert G(None, _fake(A), y, 8, 256, None) == w4.ENULL
    assert G(_fake(A), _fake(A), None, 8, 256, None) == w4.ENULL
    assert G(_fake(A), _fake(A), y, 8, 128, None) == w4.ESHAPE            # K % 256
    assert G(_fake(A), _fake(A), y, 0, 256, None) == w4.ESHAPE
    assert G(_fake(A), _fake(A), y, 8, 32768 + 256, None) == w4.ERANGE    # staged whole in LDS
    assert G(_fake(A + 4), _fake(A), y, 8, 256, None) == w4.EALIGN


def test_gemm_argument_errors():
    L = w4.lib()
    S = L.q4q8_gemm_workspace_size
    assert S(33, 2048) >= 33 * 2048 + 33 * 64 * 4
    assert S(4, 2000) == 0 and S(-1, 256) == 0 and S(1 << 31, 256) == 0   # K % 256, M range
    ws, n = _fake(A + 0x100000), S(33, 2048)
    G = L.q4q8_gemm
    y = _fake(A + 0x200000)
    assert G(None, _fake(A), y, 33, 64, 2048, ws, n, None) == w4.ENULL
    assert G(_fake(A), _fake(A + 0x10), None, 33, 64, 2048, ws, n, None) == w4.ENULL
    assert G(_fake(A), _fake(A + 0x10), y, 33, 64, 2048, None, n, None) == w4.ENULL
    assert G(_fake(A), _fake(A + 0x10), y, 33, 64, 2000, ws, n, None) == w4.ESHAPE   # K % 256
    assert G(_fake(A), _fake(A + 0x10), y, -1, 64, 2048, ws, n, None) == w4.ESHAPE
    assert G(_fake(A), _fake(A + 0x10), y, 33, 0, 2048, ws, n, None) == w4.ESHAPE
    assert G(_fake(A), _fake(A + 0x10), y, 1 << 31, 64, 256, ws, n, None) == w4.ERANGE
    assert G(_fake(A), _fake(A + 0x10), y, 1 << 21, 1 << 20, 256, ws, n, None) == w4.ERANGE
    assert G(_fake(A), _fake(A + 0x10), y, 33, 64, 2048, ws, n - 1, None) == w4.EWORKSPACE
    assert G(_fake(A), _fake(A + 0x12), y, 33, 64, 2048, ws, n, None) == w4.EALIGN
    assert G(_fake(A), _fake(A + 0x10), y, 33, 64, 2048, _fake(A + 0x100008), n,
             None) == w4.EALIGN
    assert G(_fake(A), _fake(A + 0x10), y, 0, 64, 2048, None, 0, None) == w4.OK   # empty


def test_moe_sym_argument_errors():
    L = w4.lib()
    S = L.moe_sym_workspace_size
    assert S(1, 2048, 512, 256, 8) > 0
    assert S(1, 2000, 512, 256, 8) == 0 and S(1, 2048, 500, 256, 8) == 0      # H, I % 256
    assert S(1, 2048, 512, 256, 0) == 0 and S(-1, 2048, 512, 256, 8) == 0
    assert S(1, 32768, 512, 256, 8) == 0                                        # H > 16384
    n = S(2, 2048, 512, 256, 8)
    offs = (ctypes.c_size_t * 3)()
    assert L.moe_sym_workspace_layout(2, 2048, 512, 256, 8, offs) == w4.OK
    assert offs[0] < offs[1] < offs[2] < n
    assert L.moe_sym_workspace_layout(2, 2048, 512, 256, 8, None) == w4.ENULL
    F = L.moe_sym_forward
    p = [_fake(A + 0x1000 * i) for i in range(10)]
    args = lambda **kw: [kw.get(k, v) for k, v in zip(
        ("x", "ids", "w", "gu", "d", "sgu", "sd", "out"), p[:8])]
    ok = args()
    assert F(*args(x=None), 2, 2048, 512, 256, 8, p[8], n, None) == w4.ENULL
    assert F(*args(sgu=None), 2, 2048, 512, 256, 8, p[8], n, None) == w4.ENULL   # one of the pair
    assert F(*ok, 2, 2048, 512, 256, 8, None, n, None) == w4.ENULL
    assert F(*ok, 2, 2000, 512, 256, 8, p[8], n, None) == w4.ESHAPE
    assert F(*ok, 2, 2048, 512, 256, 65, p[8], n, None) == w4.ERANGE
    assert F(*ok, 2, 2048, 512, 256, 8, p[8], n - 1, None) == w4.EWORKSPACE
    assert F(*args(out=_fake(A + 0x7004)), 2, 2048, 512, 256, 8, p[8], n, None) == w4.EALIGN
    assert F(*ok, 0, 2048, 512, 256, 8, p[8], n, None) == w4.OK                  # empty


def test_gdn_argument_errors():
    L = w4.lib()
    S = L.gdn_workspace_size
    assert S(947, 32, 128, 128) > 0 and S(0, 32, 128, 128) > 0
    assert S(8, 2, 96, 128) == 0 and S(8, 2, 128, 36) == 0 and S(8, 0, 128, 128) == 0
    assert S(8, 2, 128, 8192) == 0 and S(-1, 2, 128, 128) == 0
    n = S(40, 2, 128, 64)
    p = [_fake(A + 0x10000 * i) for i in range(9)]
    F = L.gdn_chunked_scan
    ok = lambda **kw: [kw.get(name, p[i]) for i, name in enumerate(
        ("q", "k", "v", "g", "beta", "s0", "out", "s_out"))]
    assert F(*ok(q=None), 40, 2, 128, 64, p[8], n, None) == w4.ENULL
    assert F(*ok(beta=None), 40, 2, 128, 64, p[8], n, None) == w4.ENULL
    assert F(*ok(), 40, 2, 128, 64, None, n, None) == w4.ENULL
    assert F(*ok(), 40, 2, 96, 64, p[8], n, None) == w4.ESHAPE
    assert F(*ok(), 40, 2, 128, 64, p[8], n - 1, None) == w4.EWORKSPACE
    assert F(*ok(v=_fake(A + 0x20008)), 40, 2, 128, 64, p[8], n, None) == w4.EALIGN
    assert F(*ok(g=_fake(A + 0x30002)), 40, 2, 128, 64, p[8], n, None) == w4.EALIGN
    assert F(None, None, None, None, None, None, None, None, 0, 2, 128, 64, None, 0,
             None) == w4.OK                                               # empty, no state out


def test_moe_workspace_size_and_layout():
    assert w4.moe_workspace_size(1, 2048, 512, 256, 8) > 0
    assert w4.moe_workspace_size(1, 2000, 512, 256, 8) == 0          # H % 256
    assert w4.moe_workspace_size(1, 2048, 512, 256, 0) == 0          # k < 1
    assert w4.moe_workspace_size(1, 2048, 512, 5000, 8) == 0         # E > 4096
    small = w4.moe_workspace_size(1, 2048, 512, 256, 8)
    big = w4.moe_workspace_size(947, 2048, 512, 256, 8)
    assert big > small
    lay = w4.moe_workspace_layout(947, 2048, 512, 256, 8)
    assert all(v % 256 == 0 for v in lay.values())
    assert lay["hq"] - lay["h"] >= (947 * 9) * 512 * 4
    with pytest.raises(w4.W4A8Error):
        w4.moe_workspace_layout(3, 100, 512, 256, 8)


def test_moe_argument_errors():
    L = w4.lib()
    f = L.moe_w4a8_forward
    T, H, I, E, k = 2, 256, 256, 4, 2
    ws = w4.moe_workspace_size(T, H, I, E, k)
    p = _fake(A)
    names = ("x", "ids", "w", "wgu", "wd", "sgu", "sd", "out")
    args = lambda **kw: [kw.get(n, _fake(A + 0x1000 * i)) for i, n in enumerate(names)]
    assert f(*args(x=None), T, H, I, E, k, p, ws, None) == w4.ENULL
    assert f(*args(sgu=None), T, H, I, E, k, p, ws, None) == w4.ENULL      # one shared ptr alone
    assert f(*args(), T, 255, I, E, k, p, ws, None) == w4.ESHAPE
    assert f(*args(), T, H, 128, E, k, p, ws, None) == w4.ESHAPE
    assert f(*args(), -1, H, I, E, k, p, ws, None) == w4.ESHAPE
    assert f(*args(), T, H, I, E, 0, p, ws, None) == w4.ERANGE
    assert f(*args(), T, H, I, E, 33, p, ws, None) == w4.ERANGE
    assert f(*args(), T, H, I, 0, k, p, ws, None) == w4.ERANGE
    assert f(*args(x=_fake(A + 8)), T, H, I, E, k, p, ws, None) == w4.EALIGN
    assert f(*args(), T, H, I, E, k, p, ws - 1, None) == w4.EWORKSPACE
    assert f(*args(out=_fake(A)), T, H, I, E, k, p, ws, None) == w4.EALIAS   # out == hidden
    assert f(*args(), 0, H, I, E, k, p, ws, None) == w4.OK                 # empty: no-op


def test_moe_noalloc_argument_errors():
    """The no-allocation entry point validates like moe_w4a8_forward, and
    sizes whose workspace exceeds its fixed scratch give W4A8_ESCRATCH (all
    before any device call)."""
    f = w4.lib().moe_w4a8_forward_noalloc
    names = ("x", "ids", "w", "wgu", "wd", "sgu", "sd", "out")
    args = lambda **kw: [kw.get(n, _fake(A + 0x1000 * i)) for i, n in enumerate(names)]
    H, I, E, k = 2048, 512, 256, 8
    assert w4.moe_workspace_size(66, H, I, E, k) <= w4.NOALLOC_SCRATCH_BYTES
    assert w4.moe_workspace_size(67, H, I, E, k) > w4.NOALLOC_SCRATCH_BYTES
    assert f(*args(), 67, H, I, E, k, None) == w4.ESCRATCH
    assert f(*args(), 947, H, I, E, k, None) == w4.ESCRATCH
    assert f(*args(x=None), 1, H, I, E, k, None) == w4.ENULL
    assert f(*args(sd=None), 1, H, I, E, k, None) == w4.ENULL
    assert f(*args(), 1, 2000, I, E, k, None) == w4.ESHAPE
    assert f(*args(), 1, H, I, E, 0, None) == w4.ERANGE
    assert f(*args(ids=_fake(A + 4)), 1, H, I, E, k, None) == w4.EALIGN
    assert f(*args(out=_fake(A)), 1, H, I, E, k, None) == w4.EALIAS
    assert f(*args(), 0, H, I, E, k, None) == w4.OK                      # empty: no-op


def test_decode_wait_bound_set_and_restore():
    prev = w4.decode_wait_bound(-1)        # query
    assert prev >= 0
    assert w4.decode_wait_bound(7) == prev
    assert w4.decode_wait_bound(-5) == 7   # negative leaves it
    assert w4.decode_wait_bound(prev) == 7
    assert w4.decode_wait_bound(-1) == prev


def test_rmsnorm_argument_errors():
    L = w4.lib()
    f = L.rmsnorm_residual
    p = _fake(A)
    assert f(None, None, p, p, p, 2, 256, 1e-6, None) == w4.ENULL
    assert f(p, None, None, p, p, 2, 256, 1e-6, None) == w4.ENULL      # norm without gamma
    assert f(p, None, p, p, p, 2, 258, 1e-6, None) == w4.ESHAPE        # H % 4
    assert f(p, None, p, p, p, -1, 256, 1e-6, None) == w4.ESHAPE
    assert f(p, None, p, p, p, 2, 256, -1.0, None) == w4.ESHAPE       # eps < 0
    assert f(p, _fake(A + 4), p, p, p, 2, 256, 1e-6, None) == w4.EALIGN
    assert f(p, None, p, p, p, 0, 256, 1e-6, None) == w4.OK            # empty: no-op
    assert f(p, None, p, p, p, 1 << 31, 256, 1e-6, None) == w4.ERANGE


def test_moe_layer_argument_errors():
    L = w4.lib()
    f = L.moe_w4a8_layer
    T, H, I, E, k = 2, 256, 256, 4, 2
    need = L.moe_w4a8_workspace_size(T, H, I, E, k)
    x, yp, g, xo, ids, tw, wgu, wd, out, ws = (_fake(A + 4096 * i) for i in range(10))

    def call(x=x, yp=yp, g=g, eps=1e-6, xo=xo, out=out, T=T, ws_bytes=need):
        return f(x, yp, g, eps, xo, ids, tw, wgu, wd, None, None, out, T, H, I, E, k, ws,
                 ws_bytes, None)
    assert call(g=None) == w4.ENULL
    assert call(xo=None) == w4.ENULL
    assert call(x=None) == w4.ENULL
    assert call(eps=-1.0) == w4.ESHAPE
    assert call(yp=_fake(A + 2)) == w4.EALIGN
    assert call(g=_fake(A + 8)) == w4.EALIGN
    assert call(xo=x) == w4.EALIAS
    assert call(xo=yp) == w4.EALIAS
    assert call(out=xo) == w4.EALIAS
    assert call(out=yp) == w4.EALIAS
    assert call(ws_bytes=need - 1) == w4.EWORKSPACE
    assert call(T=0) == w4.OK                                         # empty: no-op


def test_router_argument_errors():
    f = w4.lib().moe_router_topk
    p = _fake(A)
    assert f(None, p, p, 4, 256, 8, None) == w4.ENULL
    assert f(p, p, None, 4, 256, 8, None) == w4.ENULL
    assert f(p, p, p, -1, 256, 8, None) == w4.ESHAPE
    assert f(p, p, p, 4, 0, 1, None) == w4.ERANGE          # E < 1
    assert f(p, p, p, 4, 4097, 8, None) == w4.ERANGE       # E > 4096
    assert f(p, p, p, 4, 256, 0, None) == w4.ERANGE        # k < 1
    assert f(p, p, p, 4, 256, 33, None) == w4.ERANGE       # k > 32
    assert f(p, p, p, 4, 6, 7, None) == w4.ERANGE          # k > E
    assert f(p, p, p, 1 << 31, 256, 8, None) == w4.ERANGE
    assert f(p, _fake(A + 2), p, 4, 256, 8, None) == w4.EALIGN
    assert f(p, p, p, 0, 256, 8, None) == w4.OK            # empty: no-op


def test_layer_routed_argument_errors():
    f = w4.lib().moe_w4a8_layer_routed
    H, I, E, k, T = 256, 256, 4, 2, 3
    need = w4.moe_workspace_size(T, H, I, E, k)
    x, yp, g, xo, lg, gt, wgu, wd, sgu, sd, out, ids, tw, ws = (_fake(A + 4096 * i)
                                                                for i in range(14))
    def call(**kw):
        a = dict(x=x, yp=yp, g=g, eps=1e-6, xo=xo, lg=lg, gt=gt, wgu=wgu, wd=wd, sgu=sgu, sd=sd,
                 out=out, ids=ids, tw=tw, T=T, E=E, k=k, ws=ws, n=need)
        a.update(kw)
        return f(a["x"], a["yp"], a["g"], a["eps"], a["xo"], a["lg"], a["gt"], a["wgu"], a["wd"],
                 a["sgu"], a["sd"], a["out"], a["ids"], a["tw"], a["T"], H, I, a["E"], a["k"],
                 a["ws"], a["n"], None)
    assert call(lg=None) == w4.ENULL
    assert call(sgu=None, sd=None) == w4.ENULL          # a gate for a missing shared expert
    assert call(ids=None) == w4.ENULL
    assert call(lg=_fake(A + 2)) == w4.EALIGN
    assert call(gt=_fake(A + 1)) == w4.EALIGN
    assert call(k=5, n=w4.moe_workspace_size(T, H, I, E, 5)) == w4.ERANGE   # k > E
    assert call(xo=x) == w4.EALIAS
    assert call(n=need - 1) == w4.EWORKSPACE
    assert call(T=0) == w4.OK
