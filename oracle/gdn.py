"""CPU oracle of the gated-delta-net (GDN) recurrence -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the product library never does.

The model's GDN layers carry, per value head, a state S in R^{dk x dv} that is
updated token by token (Sec. 2.2 "The model"; 32 value heads with
dk = dv = 128).  The paper names the layer a gated extension of the delta
rule and does not write the update out; the reading taken here is the gated
delta rule of the work it cites, for each head and token t:

    S_t = alpha_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T
    o_t = S_t^T q_t

with alpha_t = exp(g_t) in (0, 1] (the decay gate, given in log form g_t <= 0)
and beta_t in [0, 1] (the delta-rule step).  The projections that produce q,
k, v, g and beta from the hidden state, their short convolutions, the L2
normalization of q and k, and the output norm and gate belong to the model's
layer and are inputs here.

Plain numpy in fp64, the recurrence exactly as written (one token at a time,
all heads at once).
"""
from __future__ import annotations

import numpy as np


def gdn_recurrent(q, k, v, g, beta, s0=None):
    """The GDN recurrence.

    q, k: [T, NH, DK]; v: [T, NH, DV]; g, beta: [T, NH]; s0: [NH, DK, DV] or
    None (zero state).  Returns (o [T, NH, DV], s_final [NH, DK, DV],
    smax [NH, DV]) in fp64, where smax[h, c] is the largest 2-norm over time
    of column c of head h's state (a magnitude for tolerances)."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    g = np.asarray(g, np.float64)
    beta = np.asarray(beta, np.float64)
    T, NH, DK = k.shape
    DV = v.shape[2]
    S = np.zeros((NH, DK, DV)) if s0 is None else np.array(s0, np.float64, copy=True)
    o = np.zeros((T, NH, DV))
    smax = np.sqrt((S * S).sum(axis=1))
    for t in range(T):
        a = np.exp(g[t])[:, None, None]
        b = beta[t][:, None, None]
        kt = k[t][:, :, None]                              # [NH, DK, 1]
        kS = np.einsum("hd,hdv->hv", k[t], S)[:, None, :]  # k_t^T S, [NH, 1, DV]
        S = a * (S - b * kt * kS) + b * kt * v[t][:, None, :]
        o[t] = np.einsum("hdv,hd->hv", S, q[t])
        smax = np.maximum(smax, np.sqrt((S * S).sum(axis=1)))
    return o, S, smax
