"""Parity check of one MoE layer against the oracle (used by the GPU tests and
the smoke check).

Q8_0(h) is an integer decision taken on an fp32 value whose last bits depend
on summation order, so near a rounding boundary more than one result is
correct.  The check therefore:
  1. bounds the GPU's fp32 h against the oracle's h by dh, the change the
     float tolerance (1e-5 of sum |terms|) of gate and up can cause in
     SiLU(gate) * up;
  2. requires every GPU Q8_0(h) block to be one of the results the oracle
     accepts for an input known to +-dh (q8_0_candidates), and counts the
     blocks that differ from the oracle's own choice ("flips");
  3. evaluates the oracle's down projection and combine on that accepted
     Q8_0(h) and requires |out - ref| <= 1e-5 * sum |terms| elementwise.
"""
from __future__ import annotations

import numpy as np

import oracle

EPS = 1e-5


def delta_h(gu: np.ndarray, Rgu: np.ndarray, I: int, eps: float = EPS) -> np.ndarray:
    g = gu[..., :I].astype(np.float64)
    u = gu[..., I:].astype(np.float64)
    dg = eps * Rgu[..., :I]
    du = eps * Rgu[..., I:]
    with np.errstate(over="ignore"):
        s = g / (1.0 + np.exp(-g))
    h = s * u
    # |silu'| <= 1.0998; fp32 rounding of silu, expf and the product: 2^-20 |h|
    dh = 1.1 * dg * (np.abs(u) + du) + (np.abs(s) + 1.1 * dg) * du + 2.0**-20 * np.abs(h) + 1e-30
    return dh.astype(np.float32)


def valid_pairs(ids: np.ndarray, E: int, shared: bool):
    T, k = ids.shape
    routed = [t * k + j for t in range(T) for j in range(k) if 0 <= ids[t, j] < E]
    return routed + ([T * k + t for t in range(T)] if shared else [])


def check_layer(out_gpu, h_gpu, hq_gpu, x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k,
                shared_w=None):
    """All GPU arrays in the oracle's pair numbering for these T tokens:
    out_gpu [T,H] fp32, h_gpu [P,I] fp32, hq_gpu [P, I/32*34] uint8.
    shared_w: the shared expert's per-token weight (fp64 [T]), None = 1."""
    T = x.shape[0]
    shared = ws_gu is not None
    r = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, shared_w=shared_w)
    pairs = valid_pairs(ids, E, shared)
    nb = I // 32
    sel = r.hq.copy()
    flips = 0
    worst_h = 0.0
    for p in pairs:
        dh = delta_h(r.gu[p], r.Rgu[p], I)
        err = np.abs(h_gpu[p].astype(np.float64) - r.h[p].astype(np.float64))
        assert np.all(err <= dh), f"h of pair {p}: max err/bound {np.max(err / dh):.3g}"
        worst_h = max(worst_h, float(np.max(err / dh)))
        scales, qlo, qhi, ns = oracle.q8_0_candidates(r.h[p], dh)
        d_g, q_g = oracle.q8_0_split(hq_gpu[p].reshape(1, -1))
        d_r, q_r = oracle.q8_0_split(r.hq[p].reshape(1, -1))
        for b in range(nb):
            c = [i for i in range(ns[b]) if scales[b, i] == d_g[0, b]]
            assert c, f"pair {p} block {b}: scale {d_g[0, b]:#06x} not a valid result"
            c = c[0]
            assert np.all(q_g[0, b] >= qlo[b, c]) and np.all(q_g[0, b] <= qhi[b, c]), \
                f"pair {p} block {b}: codes outside the valid set"
            if d_g[0, b] != d_r[0, b] or not np.array_equal(q_g[0, b], q_r[0, b]):
                flips += 1
        sel[p] = hq_gpu[p]
    r2 = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=sel,
                    want_intermediates=False, shared_w=shared_w)
    err = np.abs(out_gpu.astype(np.float64) - r2.out)
    bound = EPS * r2.R
    bad = err > bound
    assert not bad.any(), (f"{bad.sum()} outputs beyond 1e-5 * sum|terms|; "
                           f"worst ratio {np.max(err / np.maximum(bound, 1e-300)):.3g}")
    rel = float(np.max(err / np.maximum(r2.R, 1e-300)))
    return {"pairs": len(pairs), "flips": flips, "max_rel_err": rel, "h_err_over_bound": worst_h}


def gather_tokens(tokens, T, k, out_gpu, h_gpu, hq_gpu):
    """Re-number a subset of the GPU's tokens into the oracle's numbering for
    those tokens alone."""
    tokens = np.asarray(tokens)
    Ts = len(tokens)
    rows = [t * k + j for t in tokens for j in range(k)] + [T * k + t for t in tokens]
    return out_gpu[tokens], h_gpu[rows], hq_gpu[rows], Ts
