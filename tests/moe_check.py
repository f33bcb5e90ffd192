"""Parity check of one MoE layer against the oracle (used by the GPU tests and
the smoke check).

Q8_0(h) is an integer decision taken on an fp32 value whose last bits depend
on summation order, so near a rounding boundary more than one result is
correct.  The check therefore, for every valid token-expert pair:
  1. requires the GPU's Q8_0(h) to be bit-exactly Q8_0 of the GPU's own fp32 h
     (both are in the workspace): the quantizer itself has one right answer;
  2. bounds the GPU's fp32 h against the oracle's h by dh, the change the
     float tolerance (1e-5 of sum |terms|) of gate and up can cause in
     SiLU(gate) * up;
  3. requires every GPU Q8_0(h) block to be one of the results the oracle
     accepts for an input known to +-dh (q8_0_candidates), and counts the
     blocks that differ from the oracle's own choice ("flips"), optionally
     bounding their number;
  4. evaluates the oracle's down projection and combine on the GPU's Q8_0(h)
     (teacher forcing) and requires |out - ref| <= 1e-5 * sum |terms|
     elementwise.
"""
from __future__ import annotations

import os

import numpy as np

import oracle

EPS = 1e-5
STATS = []      # (test, result of check_layer) of every check, for the run's summary


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
                shared_w=None, max_flips=None):
    """All GPU arrays in the oracle's pair numbering for these T tokens:
    out_gpu [T,H] fp32, h_gpu [P,I] fp32, hq_gpu [P, I/32*34] uint8.
    shared_w: the shared expert's per-token weight (fp64 [T]), None = 1.
    max_flips: largest number of Q8_0(h) blocks allowed to differ from the
    oracle's own choice (None: counted, not bounded)."""
    shared = ws_gu is not None
    r = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, shared_w=shared_w)
    pairs = np.asarray(valid_pairs(ids, E, shared), dtype=np.int64)
    nb = I // 32
    np_ = len(pairs)
    hg = np.ascontiguousarray(h_gpu[pairs], dtype=np.float32)
    qg = np.ascontiguousarray(hq_gpu[pairs], dtype=np.uint8)

    # 1. the GPU's Q8_0(h) is Q8_0 of its own h, byte for byte
    q_own = oracle.q8_0_quantize(hg) if np_ else qg
    if not np.array_equal(qg, q_own):
        bad = np.nonzero((qg != q_own).reshape(np_, nb, 34).any(axis=2))
        raise AssertionError(f"Q8_0(h) differs from Q8_0 of the GPU's own h at "
                             f"{len(bad[0])} blocks, first (pair {pairs[bad[0][0]]}, "
                             f"block {bad[1][0]})")

    # 2. h within dh of the oracle's h
    dh = delta_h(r.gu[pairs], r.Rgu[pairs], I)
    hr = r.h[pairs]
    err = np.abs(hg.astype(np.float64) - hr.astype(np.float64))
    ratio = err / dh
    if np_ and not np.all(err <= dh):
        i, j = np.unravel_index(np.argmax(ratio), ratio.shape)
        raise AssertionError(f"h of pair {pairs[i]} column {j}: err/bound {ratio[i, j]:.3g}")
    worst_h = float(ratio.max()) if np_ else 0.0

    # 3. every block one of the valid results for h known to +-dh
    flips = 0
    if np_:
        scales, qlo, qhi, ns = oracle.q8_0_candidates(hr.ravel(), dh.ravel())
        d_g, q_g = oracle.q8_0_split(qg.ravel())
        d_r, q_r = oracle.q8_0_split(r.hq[pairs].ravel())
        member = (scales == d_g[:, None]) & (np.arange(scales.shape[1])[None, :] < ns[:, None])
        okscale = member.any(axis=1)
        if not okscale.all():
            b = int(np.nonzero(~okscale)[0][0])
            raise AssertionError(f"pair {pairs[b // nb]} block {b % nb}: scale "
                                 f"{d_g[b]:#06x} not a valid result")
        c = np.argmax(member, axis=1)
        lo = qlo[np.arange(np_ * nb), c]
        hi = qhi[np.arange(np_ * nb), c]
        inside = ((q_g >= lo) & (q_g <= hi)).all(axis=1)
        if not inside.all():
            b = int(np.nonzero(~inside)[0][0])
            raise AssertionError(f"pair {pairs[b // nb]} block {b % nb}: codes outside the "
                                 f"valid set")
        flips = int(((d_g != d_r) | (q_g != q_r).any(axis=1)).sum())
    if max_flips is not None:
        assert flips <= max_flips, f"{flips} Q8_0(h) blocks differ from the oracle's choice"

    # 4. teacher-forced down projection and combine
    sel = r.hq.copy()
    sel[pairs] = qg
    r2 = oracle.moe(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=sel,
                    want_intermediates=False, shared_w=shared_w)
    err = np.abs(out_gpu.astype(np.float64) - r2.out)
    bound = EPS * r2.R
    bad = err > bound
    assert not bad.any(), (f"{bad.sum()} outputs beyond 1e-5 * sum|terms|; "
                           f"worst ratio {np.max(err / np.maximum(bound, 1e-300)):.3g}")
    rel = float(np.max(err / np.maximum(r2.R, 1e-300)))
    st = {"pairs": np_, "flips": flips, "blocks": np_ * nb, "max_rel_err": rel,
          "h_err_over_bound": worst_h}
    STATS.append((os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], st))
    return st


def gather_tokens(tokens, T, k, out_gpu, h_gpu, hq_gpu):
    """Re-number a subset of the GPU's tokens into the oracle's numbering for
    those tokens alone."""
    tokens = np.asarray(tokens)
    Ts = len(tokens)
    rows = [t * k + j for t in tokens for j in range(k)] + [T * k + t for t in tokens]
    return out_gpu[tokens], h_gpu[rows], hq_gpu[rows], Ts


def check_sym_layer(out_gpu, h_gpu, hq_gpu, x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k,
                    max_flips=None):
    """The same check for the layer in the paper's own format (Q8_F32 h,
    hq_gpu [P, I/32*36]): Q8_F32(h) of the GPU's own h byte for byte, h
    within dh of the oracle's h (so the codes are those of an h the float
    tolerance allows), flips against the oracle's own codes counted, and the
    output teacher-forced on the GPU's codes within 1e-5 * sum |terms|."""
    shared = ws_gu is not None
    r = oracle.moe_sym(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k)
    pairs = np.asarray(valid_pairs(ids, E, shared), dtype=np.int64)
    nb = I // 32
    np_ = len(pairs)
    hg = np.ascontiguousarray(h_gpu[pairs], dtype=np.float32)
    qg = np.ascontiguousarray(hq_gpu[pairs], dtype=np.uint8)
    q_own = oracle.q8_f32_quantize(hg) if np_ else qg
    if not np.array_equal(qg, q_own):
        bad = np.nonzero((qg != q_own).reshape(np_, nb, 36).any(axis=2))
        raise AssertionError(f"Q8_F32(h) differs from Q8_F32 of the GPU's own h at "
                             f"{len(bad[0])} blocks, first (pair {pairs[bad[0][0]]}, "
                             f"block {bad[1][0]})")
    dh = delta_h(r.gu[pairs], r.Rgu[pairs], I)
    err = np.abs(hg.astype(np.float64) - r.h[pairs].astype(np.float64))
    ratio = err / dh
    if np_ and not np.all(err <= dh):
        i, j = np.unravel_index(np.argmax(ratio), ratio.shape)
        raise AssertionError(f"h of pair {pairs[i]} column {j}: err/bound {ratio[i, j]:.3g}")
    # a flip: a block whose codes differ from the oracle's (the fp32 scale
    # follows h's last bits and is bounded through h)
    flips = int((qg.reshape(np_, nb, 36)[..., 4:] !=
                 r.hq[pairs].reshape(np_, nb, 36)[..., 4:]).any(axis=2).sum())
    if max_flips is not None:
        assert flips <= max_flips, f"{flips} Q8_F32(h) blocks differ from the oracle's choice"
    sel = r.hq.copy()
    sel[pairs] = qg
    r2 = oracle.moe_sym(x, ids, wts, w_gu, w_d, ws_gu, ws_d, H, I, E, k, hq_in=sel,
                        want_intermediates=False)
    err = np.abs(out_gpu.astype(np.float64) - r2.out)
    bad = err > EPS * r2.R
    assert not bad.any(), (f"{bad.sum()} outputs beyond 1e-5 * sum|terms|; worst ratio "
                           f"{np.max(err / np.maximum(EPS * r2.R, 1e-300)):.3g}")
    rel = float(np.max(err / np.maximum(r2.R, 1e-300)))
    st = {"pairs": np_, "flips": flips, "blocks": np_ * nb, "max_rel_err": rel,
          "h_err_over_bound": float(ratio.max()) if np_ else 0.0}
    STATS.append((os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], st))
    return st
