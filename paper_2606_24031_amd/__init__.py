"""W4A8 (Q4_0 weight x Q8_0 activation) MoE hot path for AMD MI355X (gfx950).

A thin ctypes binding over ``libw4a8.so``: every function marshals torch
tensors (device memory and the current HIP stream) into the C ABI declared in
``include/w4a8.h`` and raises on a non-zero status.  All arithmetic runs in the
HIP kernels; there is no CPU or PyTorch fallback -- if the library is missing
or the device is not gfx950 the calls raise.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libw4a8.so")

OK, ENULL, ESHAPE, ERANGE, EWORKSPACE, EALIGN, EHIP, EDEVICE, EALIAS, ESCRATCH = \
    0, -1, -2, -3, -4, -5, -6, -7, -8, -9
NOALLOC_SCRATCH_BYTES = 8 << 20
Q4_0_BLOCK_BYTES = 18
Q8_0_BLOCK_BYTES = 34
Q4_SYM_BLOCK_BYTES = 20
Q8_F32_BLOCK_BYTES = 36
WS_XQ, WS_H, WS_HQ, WS_PERM, WS_COUNT, WS_SYNC, WS_SYNC_END, WS_XN = 0, 1, 2, 3, 4, 5, 6, 7
WS_NFIELDS = 8

EXPORTS = ("w4a8_strerror", "q8_0_quantize", "q4_0_quantize", "q4q8_gemv",
           "moe_w4a8_workspace_size", "moe_w4a8_workspace_init",
           "moe_w4a8_workspace_layout", "moe_w4a8_forward", "moe_w4a8_layer",
           "rmsnorm_residual", "moe_router_topk", "moe_w4a8_layer_routed",
           "q4_sym_quantize", "q8_f32_quantize", "q4sym_q8f32_gemv",
           "w4a8_decode_wait_bound", "moe_w4a8_forward_noalloc", "q4q8_gemm_workspace_size",
           "q4q8_gemm", "moe_sym_workspace_size", "moe_sym_workspace_layout", "moe_sym_forward",
           "gdn_workspace_size", "gdn_chunked_scan")

_lib = None


class W4A8Error(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {strerror(code)} ({code})")


def lib() -> ctypes.CDLL:
    """Load libw4a8.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2606_24031_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    L.w4a8_strerror.argtypes = [ctypes.c_int]
    L.w4a8_strerror.restype = ctypes.c_char_p
    for name in ("q8_0_quantize", "q4_0_quantize", "q4_sym_quantize", "q8_f32_quantize"):
        getattr(L, name).argtypes = [P, P, I64, I64, P]
        getattr(L, name).restype = ctypes.c_int
    L.q4q8_gemv.argtypes = [P, P, P, I64, I64, P]
    L.q4q8_gemv.restype = ctypes.c_int
    L.q4sym_q8f32_gemv.argtypes = [P, P, P, I64, I64, P]
    L.q4sym_q8f32_gemv.restype = ctypes.c_int
    L.moe_w4a8_workspace_size.argtypes = [I64, I64, I64, I64, I64]
    L.moe_w4a8_workspace_size.restype = SZ
    L.moe_w4a8_workspace_init.argtypes = [P, SZ, P]
    L.moe_w4a8_workspace_init.restype = ctypes.c_int
    L.moe_w4a8_workspace_layout.argtypes = [I64, I64, I64, I64, I64, P]
    L.moe_w4a8_workspace_layout.restype = ctypes.c_int
    L.moe_w4a8_forward.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, P, SZ, P]
    L.moe_w4a8_forward.restype = ctypes.c_int
    L.moe_w4a8_layer.argtypes = [P, P, P, ctypes.c_float, P, P, P, P, P, P, P, P,
                                 I64, I64, I64, I64, I64, P, SZ, P]
    L.moe_w4a8_layer.restype = ctypes.c_int
    L.rmsnorm_residual.argtypes = [P, P, P, P, P, I64, I64, ctypes.c_float, P]
    L.rmsnorm_residual.restype = ctypes.c_int
    L.moe_router_topk.argtypes = [P, P, P, I64, I64, I64, P]
    L.moe_router_topk.restype = ctypes.c_int
    L.moe_w4a8_layer_routed.argtypes = [P, P, P, ctypes.c_float, P, P, P, P, P, P, P, P, P, P,
                                        I64, I64, I64, I64, I64, P, SZ, P]
    L.moe_w4a8_layer_routed.restype = ctypes.c_int
    L.w4a8_decode_wait_bound.argtypes = [I64]
    L.w4a8_decode_wait_bound.restype = ctypes.c_int
    L.moe_w4a8_forward_noalloc.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, P]
    L.moe_w4a8_forward_noalloc.restype = ctypes.c_int
    L.q4q8_gemm_workspace_size.argtypes = [I64, I64]
    L.q4q8_gemm_workspace_size.restype = SZ
    L.q4q8_gemm.argtypes = [P, P, P, I64, I64, I64, P, SZ, P]
    L.q4q8_gemm.restype = ctypes.c_int
    L.moe_sym_workspace_size.argtypes = [I64, I64, I64, I64, I64]
    L.moe_sym_workspace_size.restype = SZ
    L.moe_sym_workspace_layout.argtypes = [I64, I64, I64, I64, I64, P]
    L.moe_sym_workspace_layout.restype = ctypes.c_int
    L.moe_sym_forward.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, P, SZ, P]
    L.moe_sym_forward.restype = ctypes.c_int
    L.gdn_workspace_size.argtypes = [I64, I64, I64, I64]
    L.gdn_workspace_size.restype = SZ
    L.gdn_chunked_scan.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, P, SZ, P]
    L.gdn_chunked_scan.restype = ctypes.c_int
    _lib = L
    return L


def strerror(code: int) -> str:
    return lib().w4a8_strerror(code).decode()


def _check(rc: int, where: str):
    if rc != OK:
        raise W4A8Error(rc, where)


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _u8(t):
    import torch
    assert t.dtype == torch.uint8 and t.is_contiguous()
    return t


# ------------------------------------------------------------------ entry points
def q8_0_quantize(x, out=None, stream=None):
    """Q8_0 of fp32 rows x [rows, K] -> uint8 [rows, K/32*34] on x's device."""
    import torch
    assert x.dtype == torch.float32 and x.is_contiguous()
    rows, K = (1, x.numel()) if x.dim() == 1 else (x.numel() // x.shape[-1], x.shape[-1])
    if out is None:
        out = torch.empty((rows, K // 32 * Q8_0_BLOCK_BYTES), dtype=torch.uint8, device=x.device)
    _check(lib().q8_0_quantize(_p(x), _p(_u8(out)), rows, K, _stream(stream)), "q8_0_quantize")
    return out


def q4_0_quantize(w, out=None, stream=None):
    """Q4_0 of fp32 rows w [rows, K] -> uint8 [rows, K/32*18] on w's device."""
    import torch
    assert w.dtype == torch.float32 and w.is_contiguous()
    rows, K = (1, w.numel()) if w.dim() == 1 else (w.numel() // w.shape[-1], w.shape[-1])
    if out is None:
        out = torch.empty((rows, K // 32 * Q4_0_BLOCK_BYTES), dtype=torch.uint8, device=w.device)
    _check(lib().q4_0_quantize(_p(w), _p(_u8(out)), rows, K, _stream(stream)), "q4_0_quantize")
    return out


def q4q8_gemv(w, xq, N, K, y=None, stream=None):
    """y[N] = W4A8(w [N, K/32 Q4_0 blocks], xq [K/32 Q8_0 blocks]) in fp32."""
    import torch
    if y is None:
        y = torch.empty(N, dtype=torch.float32, device=w.device)
    _check(lib().q4q8_gemv(_p(_u8(w)), _p(_u8(xq)), _p(y), N, K, _stream(stream)), "q4q8_gemv")
    return y


def gemm_workspace(M, K, device="cuda"):
    """A workspace for q4q8_gemm with M activation rows of length K."""
    import torch
    n = int(lib().q4q8_gemm_workspace_size(M, K))
    if n == 0:
        raise W4A8Error(ESHAPE, "q4q8_gemm_workspace_size")
    return torch.empty(n, dtype=torch.uint8, device=device)


def q4q8_gemm(w, xq, M, N, K, y=None, workspace=None, stream=None):
    """y[M, N] = W4A8(xq [M, K/32 Q8_0 blocks], w [N, K/32 Q4_0 blocks]) in fp32."""
    import torch
    if y is None:
        y = torch.empty((M, N), dtype=torch.float32, device=w.device)
    if workspace is None and M > 1:
        workspace = gemm_workspace(M, K, device=w.device)
    nbytes = 0 if workspace is None else workspace.numel()
    _check(lib().q4q8_gemm(_p(_u8(w)), _p(_u8(xq)), _p(y), M, N, K, _p(workspace), nbytes,
                           _stream(stream)), "q4q8_gemm")
    return y


def moe_sym_workspace(T, H, I, E, k, device="cuda"):
    """A workspace for moe_sym_forward."""
    import torch
    n = int(lib().moe_sym_workspace_size(T, H, I, E, k))
    if n == 0:
        raise W4A8Error(ESHAPE, "moe_sym_workspace_size")
    return torch.empty(n, dtype=torch.uint8, device=device)


def moe_sym_workspace_layout(T, H, I, E, k) -> dict:
    offs = (ctypes.c_size_t * 3)()
    _check(lib().moe_sym_workspace_layout(T, H, I, E, k, offs), "moe_sym_workspace_layout")
    return {"xq": offs[0], "h": offs[1], "hq": offs[2]}


def moe_sym_forward(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
                    H, I, E, k, workspace, out=None, stream=None):
    """The MoE layer in the paper's own format (Q4_SYM weights, Q8_F32
    activations); returns out [T, H] fp32."""
    import torch
    T = hidden.shape[0]
    assert hidden.dtype == torch.float32 and hidden.is_contiguous()
    assert topk_ids.dtype == torch.int32 and topk_ids.is_contiguous()
    assert topk_w.dtype == torch.float32 and topk_w.is_contiguous()
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    rc = lib().moe_sym_forward(_p(hidden), _p(topk_ids), _p(topk_w), _p(_u8(w_gate_up)),
                               _p(_u8(w_down)), _p(ws_gate_up), _p(ws_down), _p(out),
                               T, H, I, E, k, _p(workspace), workspace.numel(), _stream(stream))
    _check(rc, "moe_sym_forward")
    return out


def gdn_scan(q, k, v, g, beta, s0=None, out=None, s_out=None, workspace=None, stream=None):
    """The gated-delta-net recurrence as a chunked scan (gdn_chunked_scan):
    q, k [T, NH, DK], v [T, NH, DV], g and beta [T, NH], s0 [NH, DK, DV] or
    None; returns (out [T, NH, DV], s_out [NH, DK, DV]), fp32."""
    import torch
    T, NH, DK = k.shape
    DV = v.shape[2]
    for t in (q, k, v, g, beta, s0):
        assert t is None or (t.dtype == torch.float32 and t.is_contiguous())
    if out is None:
        out = torch.empty((T, NH, DV), dtype=torch.float32, device=k.device)
    if s_out is None:
        s_out = torch.empty((NH, DK, DV), dtype=torch.float32, device=k.device)
    if workspace is None:
        n = int(lib().gdn_workspace_size(T, NH, DK, DV))
        if n == 0:
            raise W4A8Error(ESHAPE, "gdn_workspace_size")
        workspace = torch.empty(n, dtype=torch.uint8, device=k.device)
    _check(lib().gdn_chunked_scan(_p(q), _p(k), _p(v), _p(g), _p(beta), _p(s0), _p(out),
                                  _p(s_out), T, NH, DK, DV, _p(workspace), workspace.numel(),
                                  _stream(stream)), "gdn_chunked_scan")
    return out, s_out


def q4_sym_quantize(w, out=None, stream=None):
    """The paper's symmetric 4-bit weights ({-7..7}, fp32 scale per 32) of fp32
    rows w [rows, K] -> uint8 [rows, K/32*20] on w's device."""
    import torch
    assert w.dtype == torch.float32 and w.is_contiguous()
    rows, K = (1, w.numel()) if w.dim() == 1 else (w.numel() // w.shape[-1], w.shape[-1])
    if out is None:
        out = torch.empty((rows, K // 32 * Q4_SYM_BLOCK_BYTES), dtype=torch.uint8, device=w.device)
    _check(lib().q4_sym_quantize(_p(w), _p(_u8(out)), rows, K, _stream(stream)), "q4_sym_quantize")
    return out


def q8_f32_quantize(x, out=None, stream=None):
    """8-bit activations with an fp32 scale per 32 of fp32 rows x [rows, K] ->
    uint8 [rows, K/32*36] on x's device."""
    import torch
    assert x.dtype == torch.float32 and x.is_contiguous()
    rows, K = (1, x.numel()) if x.dim() == 1 else (x.numel() // x.shape[-1], x.shape[-1])
    if out is None:
        out = torch.empty((rows, K // 32 * Q8_F32_BLOCK_BYTES), dtype=torch.uint8, device=x.device)
    _check(lib().q8_f32_quantize(_p(x), _p(_u8(out)), rows, K, _stream(stream)), "q8_f32_quantize")
    return out


def q4sym_q8f32_gemv(w, xq, N, K, y=None, stream=None):
    """y[N] = product of w [N, K/32 Q4_SYM blocks] and xq [K/32 Q8_F32 blocks]."""
    import torch
    if y is None:
        y = torch.empty(N, dtype=torch.float32, device=w.device)
    _check(lib().q4sym_q8f32_gemv(_p(_u8(w)), _p(_u8(xq)), _p(y), N, K, _stream(stream)),
           "q4sym_q8f32_gemv")
    return y


def router_topk(logits, k, ids=None, weights=None, stream=None):
    """Top-k of fp32 logits [T, E] (descending, equal logits by increasing
    index) and the softmax weights renormalized over the selection; returns
    (ids int32 [T, k], weights fp32 [T, k])."""
    import torch
    assert logits.dtype == torch.float32 and logits.is_contiguous() and logits.dim() == 2
    T, E = logits.shape
    if ids is None:
        ids = torch.empty((T, k), dtype=torch.int32, device=logits.device)
    if weights is None:
        weights = torch.empty((T, k), dtype=torch.float32, device=logits.device)
    _check(lib().moe_router_topk(_p(logits), _p(ids), _p(weights), T, E, k, _stream(stream)),
           "moe_router_topk")
    return ids, weights


def moe_workspace_size(T, H, I, E, k) -> int:
    return int(lib().moe_w4a8_workspace_size(T, H, I, E, k))


def moe_workspace(T, H, I, E, k, device="cuda", stream=None):
    """Allocate and zero-fill a workspace for these sizes."""
    import torch
    n = moe_workspace_size(T, H, I, E, k)
    if n == 0:
        raise W4A8Error(ESHAPE, "moe_workspace_size")
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    _check(lib().moe_w4a8_workspace_init(_p(ws), n, _stream(stream)), "moe_w4a8_workspace_init")
    return ws


def moe_workspace_layout(T, H, I, E, k) -> dict:
    offs = (ctypes.c_size_t * WS_NFIELDS)()
    _check(lib().moe_w4a8_workspace_layout(T, H, I, E, k, offs), "moe_w4a8_workspace_layout")
    return {"xq": offs[WS_XQ], "h": offs[WS_H], "hq": offs[WS_HQ], "perm": offs[WS_PERM],
            "count": offs[WS_COUNT], "sync": offs[WS_SYNC], "sync_end": offs[WS_SYNC_END],
            "xn": offs[WS_XN]}


def moe_forward(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
                H, I, E, k, workspace, out=None, stream=None):
    """One routed + shared W4A8 MoE layer; returns out [T, H] fp32."""
    import torch
    T = hidden.shape[0]
    assert hidden.dtype == torch.float32 and hidden.is_contiguous()
    assert topk_ids.dtype == torch.int32 and topk_ids.is_contiguous()
    assert topk_w.dtype == torch.float32 and topk_w.is_contiguous()
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    rc = lib().moe_w4a8_forward(_p(hidden), _p(topk_ids), _p(topk_w), _p(_u8(w_gate_up)),
                                _p(_u8(w_down)), _p(ws_gate_up), _p(ws_down), _p(out),
                                T, H, I, E, k, _p(workspace), workspace.numel(),
                                _stream(stream))
    _check(rc, "moe_w4a8_forward")
    return out


def rmsnorm_residual(x, y, gamma, eps=1e-6, x_out=None, xn=None, want_norm=True, stream=None):
    """x_out = x + y (y may be None) and xn = RMSNorm(x_out) * gamma per row of
    [T, H] fp32; returns (x_out, xn).  x_out may be x itself (in place)."""
    import torch
    T, H = x.shape
    for t in (x, y, gamma):
        assert t is None or (t.dtype == torch.float32 and t.is_contiguous())
    if x_out is None:
        x_out = torch.empty_like(x)
    if want_norm and xn is None:
        xn = torch.empty_like(x)
    rc = lib().rmsnorm_residual(_p(x), _p(y), _p(gamma if want_norm else None), _p(x_out),
                                _p(xn if want_norm else None), T, H, float(eps), _stream(stream))
    _check(rc, "rmsnorm_residual")
    return x_out, (xn if want_norm else None)


def moe_layer(x, y_prev, gamma, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
              H, I, E, k, workspace, eps=1e-6, x_out=None, out=None, stream=None):
    """One pre-norm residual MoE step: x_out = x + y_prev, out = MoE(RMSNorm(x_out)
    * gamma); returns (x_out, out)."""
    import torch
    T = x.shape[0]
    for t in (x, y_prev, gamma, topk_w):
        assert t is None or (t.dtype == torch.float32 and t.is_contiguous())
    assert topk_ids.dtype == torch.int32 and topk_ids.is_contiguous()
    if x_out is None:
        x_out = torch.empty_like(x)
    if out is None:
        out = torch.empty_like(x)
    rc = lib().moe_w4a8_layer(_p(x), _p(y_prev), _p(gamma), float(eps), _p(x_out), _p(topk_ids),
                              _p(topk_w), _p(_u8(w_gate_up)), _p(_u8(w_down)), _p(ws_gate_up),
                              _p(ws_down), _p(out), T, H, I, E, k, _p(workspace),
                              workspace.numel(), _stream(stream))
    _check(rc, "moe_w4a8_layer")
    return x_out, out


def moe_layer_routed(x, y_prev, gamma, router_logits, w_gate_up, w_down, ws_gate_up, ws_down,
                     H, I, E, k, workspace, shared_gate=None, eps=1e-6, x_out=None, out=None,
                     topk_ids=None, topk_w=None, stream=None):
    """moe_layer with the router in front: top-k of router_logits [T, E] and
    the renormalized softmax weights, an optional sigmoid gate [T] on the
    shared expert; returns (x_out, out, topk_ids, topk_w)."""
    import torch
    T = x.shape[0]
    for t in (x, y_prev, gamma, router_logits, shared_gate):
        assert t is None or (t.dtype == torch.float32 and t.is_contiguous())
    if x_out is None:
        x_out = torch.empty_like(x)
    if out is None:
        out = torch.empty_like(x)
    if topk_ids is None:
        topk_ids = torch.empty((T, k), dtype=torch.int32, device=x.device)
    if topk_w is None:
        topk_w = torch.empty((T, k), dtype=torch.float32, device=x.device)
    rc = lib().moe_w4a8_layer_routed(_p(x), _p(y_prev), _p(gamma), float(eps), _p(x_out),
                                     _p(router_logits), _p(shared_gate), _p(_u8(w_gate_up)),
                                     _p(_u8(w_down)), _p(ws_gate_up), _p(ws_down), _p(out),
                                     _p(topk_ids), _p(topk_w), T, H, I, E, k, _p(workspace),
                                     workspace.numel(), _stream(stream))
    _check(rc, "moe_w4a8_layer_routed")
    return x_out, out, topk_ids, topk_w


def decode_wait_bound(rounds: int = -1) -> int:
    """Set the single-token kernel's bound on poll rounds (rounds >= 0);
    returns the previous bound."""
    return int(lib().w4a8_decode_wait_bound(int(rounds)))


def moe_forward_noalloc(hidden, topk_ids, topk_w, w_gate_up, w_down, ws_gate_up, ws_down,
                        H, I, E, k, out=None, stream=None):
    """moe_forward without a workspace argument: the library's fixed per-GPU
    scratch array serves as the workspace (moe_w4a8_forward_noalloc).  With
    `out` given, nothing is allocated."""
    import torch
    T = hidden.shape[0]
    assert hidden.dtype == torch.float32 and hidden.is_contiguous()
    assert topk_ids.dtype == torch.int32 and topk_ids.is_contiguous()
    assert topk_w.dtype == torch.float32 and topk_w.is_contiguous()
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    rc = lib().moe_w4a8_forward_noalloc(_p(hidden), _p(topk_ids), _p(topk_w), _p(_u8(w_gate_up)),
                                        _p(_u8(w_down)), _p(ws_gate_up), _p(ws_down), _p(out),
                                        T, H, I, E, k, _stream(stream))
    _check(rc, "moe_w4a8_forward_noalloc")
    return out
