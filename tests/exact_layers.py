"""MoE layers on which every W4A8 value is an exact integer (test inputs for
the bit-exact block-dot pins).

Construction:
  * Q4_0 weights with every scale 1.0, so a weight is its code q - 8;
  * activations whose 32-blocks are integers with largest magnitude 127, so
    Q8_0 gives scale 1.0 and codes equal to the values (checked);
  * gate/up rows built against the activations of the tokens they serve so
    that every gate sum g lies in [20, 127] and g * u in [-127, 127], with one
    column of every 32-column h block at g * u = +-127: then SiLU(g) rounds to
    g in fp32 on both sides (e^-20 < 2^-28), h = g * u exactly, and Q8_0 of
    every h block has scale 1.0 and codes h;
  * down rows of random codes (scale 1.0), routing weights 0.5, 1 or 2.
Every block dot is then an integer, every scaled sum an exact fp32 value (all
partial sums are multiples of 1/2 far below 2^23), so the GPU's h, Q8_0(h)
and output must equal the oracle's bit for bit, whatever the summation order;
a block dot off by one anywhere changes them.

Tokens come in clusters that share one activation vector and a disjoint set
of experts (the gate/up rows of an expert can only be built against one
vector); the shared expert needs a single cluster.  The rows themselves are
dense: every code 0..15 at every position, steered to their targets by
greedy changes of single codes.
"""
from __future__ import annotations

import numpy as np

QK = 32


def act_codes(g: np.random.Generator, K: int) -> np.ndarray:
    """Integers in [-127, 127]: per 32-block one +-127 and two +-1 at random
    positions, the rest uniform in [-126, 126]."""
    x = g.integers(-126, 127, size=K).astype(np.int64)
    for b in range(K // QK):
        pos = g.choice(QK, 3, replace=False)
        x[QK * b + pos[0]] = 127 if g.random() < 0.5 else -127
        x[QK * b + pos[1:]] = np.where(g.random(2) < 0.5, 1, -1)
    return x


def design_rows(g: np.random.Generator, x: np.ndarray, targets: np.ndarray,
                lo: int = 0) -> np.ndarray:
    """Codes Q [R, K] in lo..15 with (Q - 8) @ x == targets: random codes, then
    repeatedly the single-code change that brings each row's residual
    closest to zero, over the positions of +-127, +-1 and 64 others."""
    R, K = len(targets), len(x)
    Q = g.integers(lo, 16, size=(R, K)).astype(np.int64)
    big = np.nonzero(np.abs(x) == 127)[0]
    unit = np.nonzero(np.abs(x) == 1)[0]
    other = g.choice(np.nonzero(np.abs(x) > 1)[0], 64, replace=False)
    C = np.unique(np.concatenate([big, unit, other]))
    xc = x[C].astype(np.float64)
    res = targets.astype(np.int64) - (Q - 8) @ x
    for _ in range(400):
        live = np.nonzero(res)[0]
        if live.size == 0:
            return Q
        QC = Q[np.ix_(live, C)]
        D = np.rint(res[live, None] / xc[None, :])
        D = np.clip(D, lo - QC, 15 - QC).astype(np.int64)
        after = np.abs(res[live, None] - D * x[C][None, :])
        j = np.argmin(after, axis=1)
        d = D[np.arange(live.size), j]
        Q[live, C[j]] += d
        res[live] -= d * x[C[j]]
    raise RuntimeError("row design did not converge")


def gateup_targets(g: np.random.Generator, I: int):
    """Gate sums g in [20, 127] and up sums u with |g u| <= 127; per 32-column
    block one column at g * u = +-127 (127 is prime: g = 127, u = +-1)."""
    gt = g.integers(20, 128, size=I)
    lim = 127 // gt
    ut = np.array([g.integers(-l, l + 1) for l in lim])
    for b in range(I // QK):
        c = QK * b + int(g.integers(QK))
        gt[c] = 127
        ut[c] = 1 if g.random() < 0.5 else -1
    return gt.astype(np.int64), ut.astype(np.int64)


def pack_q4_0(Q: np.ndarray) -> np.ndarray:
    """Codes [R, K] -> Q4_0 rows [R, K/32*18] with every scale 1.0."""
    R, K = Q.shape
    q = Q.reshape(R, K // QK, QK).astype(np.uint8)
    blk = np.empty((R, K // QK, 18), np.uint8)
    blk[..., 0:2] = np.array([0x3C00], np.uint16).view(np.uint8)
    blk[..., 2:] = q[..., :16] | (q[..., 16:] << 4)
    return blk.reshape(R, K // QK * 18)


def q4_0_to_sym(w: np.ndarray) -> np.ndarray:
    """Q4_0 rows with every scale 1.0 and no nibble 0 -> the same weights as
    symmetric 4-bit blocks (fp32 scale 1.0, the same 16 payload bytes); the
    all-zero blocks of unused experts become zero blocks (scale 0, codes 0)."""
    b = np.ascontiguousarray(w, dtype=np.uint8).reshape(-1, 18)
    zero = ~b.any(axis=1)
    used = b[~zero]
    assert (used[:, 0:2].copy().view(np.uint16) == 0x3C00).all()
    assert ((used[:, 2:] & 0x0F) != 0).all() and ((used[:, 2:] >> 4) != 0).all()
    out = np.empty((b.shape[0], 20), np.uint8)
    out[:, 0:4] = np.array([1.0], np.float32).view(np.uint8)
    out[:, 4:] = b[:, 2:]
    out[zero, 0:4] = 0
    out[zero, 4:] = 0x88
    return out.reshape(w.shape[:-1] + (w.shape[-1] // 18 * 20,))


class ExactLayer:
    """clusters: list of (n_tokens, experts) with disjoint expert lists, each
    expert list of length k (skipped slots: -1).  shared: a shared expert
    (only with one cluster).  lo: smallest stored code (1 keeps every weight
    in -7..7, so q4_0_to_sym gives the same layer in the symmetric format)."""

    def __init__(self, seed, H, I, E, k, clusters, shared, lo=0):
        g = np.random.default_rng(seed)
        self.lo = lo
        assert not shared or len(clusters) == 1
        self.H, self.I, self.E, self.k = H, I, E, k
        self.w_gu = np.zeros((E, 2 * I, H // QK * 18), np.uint8)
        self.w_d = np.zeros((E, H, I // QK * 18), np.uint8)
        xs, ids = [], []
        xvec = {}
        for n, experts in clusters:
            assert len(experts) == k
            x = act_codes(g, H)
            for e in experts:
                if e >= 0 and e not in xvec:
                    xvec[e] = x
                    self.w_gu[e] = self._gateup(g, x)
                    self.w_d[e] = pack_q4_0(g.integers(lo, 16, size=(H, I)))
            xs.append(np.repeat(x[None, :], n, axis=0))
            ids.append(np.repeat(np.asarray(experts, np.int32)[None, :], n, axis=0))
        for e, x in xvec.items():
            assert all(xe is x for ee, xe in xvec.items() if ee == e)
        self.x = np.concatenate(xs).astype(np.float32)
        self.ids = np.concatenate(ids).astype(np.int32)
        T = self.x.shape[0]
        self.wts = g.choice(np.array([0.5, 1.0, 2.0], np.float32), size=(T, k))
        self.ws_gu = self.ws_d = None
        if shared:
            self.ws_gu = self._gateup(g, xs[0][0])
            self.ws_d = pack_q4_0(g.integers(self.lo, 16, size=(H, I)))

    def _gateup(self, g, x):
        gt, ut = gateup_targets(g, self.I)
        return np.concatenate([pack_q4_0(design_rows(g, x, gt, self.lo)),
                               pack_q4_0(design_rows(g, x, ut, self.lo))])

    def sym(self):
        """(w_gu, w_d, ws_gu, ws_d) in the symmetric format (needs lo >= 1)."""
        c = (lambda w: None if w is None else q4_0_to_sym(w))
        return c(self.w_gu), c(self.w_d), c(self.ws_gu), c(self.ws_d)
