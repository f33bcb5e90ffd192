"""CPU oracle for the W4A8 MoE hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library
(``paper_2606_24031_amd``) never imports it and shares no code with it.

This module is a thin ctypes/numpy wrapper around ``oracle.c`` (plain C,
scalar, fp64 accumulation, no FMA contraction).  Every function cites the
passage of the paper it follows in ``oracle.c``; the readings the paper leaves
open are listed in the design notes and in the header of ``oracle.c``.

Pair numbering used by :func:`moe`: routed slot ``j`` of token ``t`` is pair
``t*k + j``; the shared expert of token ``t`` is pair ``T*k + t``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

QK = 32
Q4_BYTES = 18
Q8_BYTES = 34
Q4S_BYTES = 20      # the paper's symmetric 4-bit block: fp32 scale + 16 bytes
Q8F_BYTES = 36      # 8-bit activations with an fp32 scale: fp32 scale + 32 codes


def build() -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, no FMA contraction)."""
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", _LIB_PATH + ".tmp",
           _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.orc_f32_to_f16.argtypes = [ctypes.c_float]
    lib.orc_f32_to_f16.restype = ctypes.c_uint16
    lib.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_f16_to_f32.restype = ctypes.c_float
    lib.orc_q8_0_quantize.argtypes = [P, P, I64, I64]
    lib.orc_q4_0_quantize.argtypes = [P, P, I64, I64]
    lib.orc_blockdot.argtypes = [P, P]
    lib.orc_blockdot.restype = ctypes.c_int32
    lib.orc_gemv.argtypes = [P, P, I64, I64, P, P]
    lib.orc_q4_sym_quantize.argtypes = [P, P, I64, I64]
    lib.orc_q8_f32_quantize.argtypes = [P, P, I64, I64]
    lib.orc_blockdot_sym.argtypes = [P, P]
    lib.orc_blockdot_sym.restype = ctypes.c_int32
    lib.orc_gemv_sym.argtypes = [P, P, I64, I64, P, P]
    lib.orc_gemv_dequant.argtypes = [P, P, I64, I64, P]
    lib.orc_moe.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, P,
                            P, P, P, P, P, P, P]
    lib.orc_moe.restype = ctypes.c_int
    lib.orc_moe_sym.argtypes = lib.orc_moe.argtypes
    lib.orc_moe_sym.restype = ctypes.c_int
    lib.orc_q8_0_candidates.argtypes = [P, P, I64, P, P, P, P]
    lib.orc_q8_0_candidates.restype = ctypes.c_int
    lib.orc_threads.restype = ctypes.c_int
    lib.orc_set_threads.argtypes = [ctypes.c_int]
    lib.orc_rmsnorm_residual.argtypes = [P, P, P, P, P, I64, I64, ctypes.c_double]
    lib.orc_router_topk.argtypes = [P, P, P, I64, I64, I64, P]
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use (OMP_NUM_THREADS)."""
    return int(_load().orc_threads())


def set_threads(n: int) -> None:
    """Use n OpenMP threads from now on (timing only; results do not depend
    on it)."""
    _load().orc_set_threads(int(n))


# ---------------------------------------------------------------- fp16
def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    """IEEE binary32 -> binary16 bits, round-to-nearest-even (elementwise)."""
    lib = _load()
    x = np.asarray(x, dtype=np.float32).ravel()
    return np.array([lib.orc_f32_to_f16(float(v)) for v in x], dtype=np.uint16)


def f16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    lib = _load()
    h = np.asarray(h, dtype=np.uint16).ravel()
    return np.array([lib.orc_f16_to_f32(int(v)) for v in h], dtype=np.float32)


# ---------------------------------------------------------------- formats
def q8_0_quantize(x: np.ndarray) -> np.ndarray:
    """Q8_0 of fp32 rows [rows, K] -> uint8 [rows, K/32*34]."""
    x = _c(x, np.float32)
    if x.ndim == 1:
        x = x[None, :]
    rows, K = x.shape
    assert K % QK == 0
    out = np.empty((rows, K // QK * Q8_BYTES), dtype=np.uint8)
    _load().orc_q8_0_quantize(_ptr(x), _ptr(out), rows, K)
    return out


def q4_0_quantize(w: np.ndarray) -> np.ndarray:
    """Q4_0 of fp32 rows [rows, K] -> uint8 [rows, K/32*18]."""
    w = _c(w, np.float32)
    if w.ndim == 1:
        w = w[None, :]
    rows, K = w.shape
    assert K % QK == 0
    out = np.empty((rows, K // QK * Q4_BYTES), dtype=np.uint8)
    _load().orc_q4_0_quantize(_ptr(w), _ptr(out), rows, K)
    return out


def blockdot(wblock: np.ndarray, ablock: np.ndarray) -> int:
    wb = _c(wblock, np.uint8)
    ab = _c(ablock, np.uint8)
    assert wb.size == Q4_BYTES and ab.size == Q8_BYTES
    return int(_load().orc_blockdot(_ptr(wb), _ptr(ab)))


def gemv(w: np.ndarray, xq: np.ndarray, N: int, K: int):
    """W4A8 product: returns (y fp64 [N], R fp64 [N]) with R = sum |term|."""
    w = _c(w, np.uint8)
    xq = _c(xq, np.uint8)
    assert w.size == N * (K // QK) * Q4_BYTES and xq.size == (K // QK) * Q8_BYTES
    y = np.empty(N, dtype=np.float64)
    R = np.empty(N, dtype=np.float64)
    _load().orc_gemv(_ptr(w), _ptr(xq), N, K, _ptr(y), _ptr(R))
    return y, R


def gemv_dequant(w: np.ndarray, xq: np.ndarray, N: int, K: int) -> np.ndarray:
    """fp64 dequantize-then-dot cross-check of :func:`gemv`."""
    w = _c(w, np.uint8)
    xq = _c(xq, np.uint8)
    y = np.empty(N, dtype=np.float64)
    _load().orc_gemv_dequant(_ptr(w), _ptr(xq), N, K, _ptr(y))
    return y


class MoeResult:
    """Outputs of :func:`moe`: out/R [T,H] fp64, gu [P,2I] fp32, Rgu [P,2I]
    fp64, h [P,I] fp32, hq [P, I/32*34] uint8 (P = T*k + T pairs; rows of
    skipped slots are zero)."""

    def __init__(self, out, R, gu, Rgu, h, hq):
        self.out, self.R, self.gu, self.Rgu, self.h, self.hq = out, R, gu, Rgu, h, hq


def moe(hidden, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=None,
        want_intermediates=True, shared_w=None) -> MoeResult:
    """Routed + shared W4A8 MoE layer, one token at a time (see orc_moe).

    hidden [T,H] fp32; ids [T,k] int32 (-1 = skipped slot); wts [T,k] fp32;
    w_gu [E, 2I, H/32*18] and w_d [E, H, I/32*18] uint8 (any shape with that
    many bytes); ws_gu/ws_d the shared expert (None = no shared expert).
    hq_in: optional [P, I/32*34] codes for h to use in the down projection.
    shared_w: optional [T] fp64 weights of the shared expert's output (its
    gate); None = 1.
    """
    hidden = _c(hidden, np.float32).reshape(-1, H)
    T = hidden.shape[0]
    ids = _c(ids, np.int32).reshape(T, k)
    wts = _c(wts, np.float32).reshape(T, k)
    w_gu = _c(w_gu, np.uint8).ravel()
    w_d = _c(w_d, np.uint8).ravel()
    assert w_gu.size == E * 2 * I * (H // QK) * Q4_BYTES
    assert w_d.size == E * H * (I // QK) * Q4_BYTES
    if ws_gu is not None:
        ws_gu = _c(ws_gu, np.uint8).ravel()
        ws_d = _c(ws_d, np.uint8).ravel()
    P = T * k + T
    out = np.zeros((T, H), dtype=np.float64)
    R = np.zeros((T, H), dtype=np.float64)
    gu = Rgu = h = hq = None
    if want_intermediates:
        gu = np.zeros((P, 2 * I), dtype=np.float32)
        Rgu = np.zeros((P, 2 * I), dtype=np.float64)
        h = np.zeros((P, I), dtype=np.float32)
        hq = np.zeros((P, I // QK * Q8_BYTES), dtype=np.uint8)
    if hq_in is not None:
        hq_in = _c(hq_in, np.uint8).reshape(P, I // QK * Q8_BYTES)
    if shared_w is not None:
        shared_w = _c(shared_w, np.float64).reshape(T)
    rc = _load().orc_moe(_ptr(hidden), _ptr(ids), _ptr(wts), _ptr(w_gu), _ptr(w_d),
                         _ptr(ws_gu), _ptr(ws_d), T, H, I, E, k, _ptr(hq_in),
                         _ptr(out), _ptr(R), _ptr(gu), _ptr(Rgu), _ptr(h), _ptr(hq),
                         _ptr(shared_w))
    if rc != 0:
        raise ValueError(f"orc_moe failed ({rc})")
    return MoeResult(out, R, gu, Rgu, h, hq)


def moe_sym(hidden, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=None,
            want_intermediates=True, shared_w=None) -> MoeResult:
    """The MoE layer of :func:`moe` in the paper's own format (Q4_SYM weights,
    Q8_F32 activations and h; see orc_moe_sym): w_gu [E, 2I, H/32*20], w_d
    [E, H, I/32*20]; hq and hq_in hold [P, I/32*36] Q8_F32 blocks."""
    hidden = _c(hidden, np.float32).reshape(-1, H)
    T = hidden.shape[0]
    ids = _c(ids, np.int32).reshape(T, k)
    wts = _c(wts, np.float32).reshape(T, k)
    w_gu = _c(w_gu, np.uint8).ravel()
    w_d = _c(w_d, np.uint8).ravel()
    assert w_gu.size == E * 2 * I * (H // QK) * Q4S_BYTES
    assert w_d.size == E * H * (I // QK) * Q4S_BYTES
    if ws_gu is not None:
        ws_gu = _c(ws_gu, np.uint8).ravel()
        ws_d = _c(ws_d, np.uint8).ravel()
    P = T * k + T
    out = np.zeros((T, H), dtype=np.float64)
    R = np.zeros((T, H), dtype=np.float64)
    gu = Rgu = h = hq = None
    if want_intermediates:
        gu = np.zeros((P, 2 * I), dtype=np.float32)
        Rgu = np.zeros((P, 2 * I), dtype=np.float64)
        h = np.zeros((P, I), dtype=np.float32)
        hq = np.zeros((P, I // QK * Q8F_BYTES), dtype=np.uint8)
    if hq_in is not None:
        hq_in = _c(hq_in, np.uint8).reshape(P, I // QK * Q8F_BYTES)
    if shared_w is not None:
        shared_w = _c(shared_w, np.float64).reshape(T)
    rc = _load().orc_moe_sym(_ptr(hidden), _ptr(ids), _ptr(wts), _ptr(w_gu), _ptr(w_d),
                             _ptr(ws_gu), _ptr(ws_d), T, H, I, E, k, _ptr(hq_in),
                             _ptr(out), _ptr(R), _ptr(gu), _ptr(Rgu), _ptr(h), _ptr(hq),
                             _ptr(shared_w))
    if rc != 0:
        raise ValueError(f"orc_moe_sym failed ({rc})")
    return MoeResult(out, R, gu, Rgu, h, hq)


def rmsnorm_residual(x, y, gamma, eps: float = 1e-6, want_norm: bool = True):
    """x_out = x + y (fp32, y may be None) and xn = RMSNorm(x_out) * gamma in
    fp64, per row of [T, H] (see orc_rmsnorm_residual)."""
    x = _c(x, np.float32)
    T, H = x.shape
    y = None if y is None else _c(y, np.float32).reshape(T, H)
    gamma = _c(gamma, np.float32).reshape(H)
    x_out = np.zeros((T, H), dtype=np.float32)
    xn = np.zeros((T, H), dtype=np.float64) if want_norm else None
    _load().orc_rmsnorm_residual(_ptr(x), _ptr(y), _ptr(gamma), _ptr(x_out), _ptr(xn), T, H,
                                 float(eps))
    return x_out, xn


def router_topk(logits: np.ndarray, k: int):
    """Router top-k of fp32 logits [T, E] (see orc_router_topk): ids int32
    [T, k] in descending logit order (equal logits by increasing index) and
    the renormalized softmax weights fp64 [T, k]."""
    logits = _c(logits, np.float32)
    T, E = logits.shape
    ids = np.zeros((T, k), dtype=np.int32)
    w = np.zeros((T, k), dtype=np.float64)
    taken = np.zeros(E, dtype=np.uint8)
    _load().orc_router_topk(_ptr(logits), _ptr(ids), _ptr(w), T, E, k, _ptr(taken))
    return ids, w


def q8_0_candidates(h: np.ndarray, dh: np.ndarray):
    """Valid Q8_0 results for h known to +-dh (see orc_q8_0_candidates).

    Returns (scales [nb,4] uint16, qlo [nb,4,32] int8, qhi [nb,4,32] int8,
    nscales [nb] int32) for a 1-D h of length K; only the first nscales[b]
    entries of block b are meaningful."""
    h = _c(h, np.float32).ravel()
    dh = _c(dh, np.float32).ravel()
    K = h.size
    nb = K // QK
    scales = np.zeros((nb, 4), dtype=np.uint16)
    qlo = np.zeros((nb, 4, QK), dtype=np.int8)
    qhi = np.zeros((nb, 4, QK), dtype=np.int8)
    ns = np.zeros(nb, dtype=np.int32)
    rc = _load().orc_q8_0_candidates(_ptr(h), _ptr(dh), K, _ptr(scales), _ptr(qlo),
                                     _ptr(qhi), _ptr(ns))
    if rc != 0:
        raise ValueError("uncertainty box admits more than 4 Q8_0 scales")
    return scales, qlo, qhi, ns


# ---------------------------------------------------------------- helpers on the byte formats
def q8_0_split(xq: np.ndarray):
    """34-byte blocks -> (fp16 scale bits [..., nb], codes int8 [..., nb, 32])."""
    b = np.asarray(xq, dtype=np.uint8)
    b = b.reshape(b.shape[:-1] + (-1, Q8_BYTES))
    d = b[..., 0].astype(np.uint16) | (b[..., 1].astype(np.uint16) << 8)
    q = b[..., 2:].view(np.int8)
    return d, q


def q4_0_split(wq: np.ndarray):
    """18-byte blocks -> (fp16 scale bits [..., nb], codes uint8 0..15 [..., nb, 32])."""
    b = np.asarray(wq, dtype=np.uint8)
    b = b.reshape(b.shape[:-1] + (-1, Q4_BYTES))
    d = b[..., 0].astype(np.uint16) | (b[..., 1].astype(np.uint16) << 8)
    nib = b[..., 2:]
    q = np.concatenate([nib & 0x0F, nib >> 4], axis=-1)
    return d, q


# ------------------------------------------- the paper's own block format
def q4_sym_quantize(w: np.ndarray) -> np.ndarray:
    """Symmetric 4-bit weights in {-7..7} with an fp32 scale per 32 (Sec. 2.3),
    fp32 rows [rows, K] -> uint8 [rows, K/32*20]."""
    w = _c(w, np.float32)
    if w.ndim == 1:
        w = w[None, :]
    rows, K = w.shape
    assert K % QK == 0
    out = np.empty((rows, K // QK * Q4S_BYTES), dtype=np.uint8)
    _load().orc_q4_sym_quantize(_ptr(w), _ptr(out), rows, K)
    return out


def q8_f32_quantize(x: np.ndarray) -> np.ndarray:
    """8-bit activations with an fp32 scale per 32 (Sec. 3.3), fp32 rows
    [rows, K] -> uint8 [rows, K/32*36]."""
    x = _c(x, np.float32)
    if x.ndim == 1:
        x = x[None, :]
    rows, K = x.shape
    assert K % QK == 0
    out = np.empty((rows, K // QK * Q8F_BYTES), dtype=np.uint8)
    _load().orc_q8_f32_quantize(_ptr(x), _ptr(out), rows, K)
    return out


def blockdot_sym(wblock: np.ndarray, ablock: np.ndarray) -> int:
    wb = _c(wblock, np.uint8)
    ab = _c(ablock, np.uint8)
    assert wb.size == Q4S_BYTES and ab.size == Q8F_BYTES
    return int(_load().orc_blockdot_sym(_ptr(wb), _ptr(ab)))


def gemv_sym(w: np.ndarray, xq: np.ndarray, N: int, K: int):
    """Product in the paper's format: returns (y fp64 [N], R fp64 [N])."""
    w = _c(w, np.uint8)
    xq = _c(xq, np.uint8)
    assert w.size == N * (K // QK) * Q4S_BYTES and xq.size == (K // QK) * Q8F_BYTES
    y = np.empty(N, dtype=np.float64)
    R = np.empty(N, dtype=np.float64)
    _load().orc_gemv_sym(_ptr(w), _ptr(xq), N, K, _ptr(y), _ptr(R))
    return y, R
