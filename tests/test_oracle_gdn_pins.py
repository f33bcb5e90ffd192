"""Pins for the oracle of the gated-delta-net recurrence (oracle/gdn.py):
two steps worked by hand (tests/golden/gdn_two_steps.txt), closed forms (no
write: pure decay of the initial state; unit steps on orthonormal keys: exact
key-value memory with overwrite), linearity in the values and the initial
state, state hand-over between two runs, and an independently written
chunkwise form of the same recurrence (WY representation of the products of
(I - beta k k^T), solved per chunk), which must agree to fp64 rounding.  CPU
only."""
import os

import numpy as np
import pytest

from oracle.gdn import gdn_recurrent
from paper_2606_24031_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "gdn_two_steps.txt")


def _golden():
    d = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, vals = [c.strip() for c in line.split("|")]
        d[name] = np.array([float(x) for x in vals.split()])
    return d


def test_two_steps_by_hand():
    d = _golden()
    T = 2
    q = d["q"].reshape(T, 1, 2)
    k = d["k"].reshape(T, 1, 2)
    v = d["v"].reshape(T, 1, 2)
    g = np.log(d["alpha"]).reshape(T, 1)
    beta = d["beta"].reshape(T, 1)
    o, s, _ = gdn_recurrent(q, k, v, g, beta, d["s0"].reshape(1, 2, 2))
    assert np.allclose(o.ravel(), d["o"], rtol=0, atol=1e-14)
    assert np.allclose(s.ravel(), d["s_final"], rtol=0, atol=1e-14)


def test_no_write_is_pure_decay():
    """beta = 0: the state only decays, S_t = exp(sum_{l<=t} g_l) S0."""
    g_ = synth.rng(1)
    q, k, v, gate, _, s0 = synth.gdn_inputs(g_, 9, 3, 8, 5)
    beta = np.zeros((9, 3), np.float32)
    o, s, _ = gdn_recurrent(q, k, v, gate, beta, s0)
    cum = np.cumsum(gate.astype(np.float64), axis=0)
    ref = np.exp(cum)[:, :, None] * np.einsum("hdv,thd->thv", s0.astype(np.float64), q)
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-15)
    assert np.allclose(s, np.exp(cum[-1])[:, None, None] * s0, rtol=1e-12, atol=1e-15)


def test_unit_steps_on_orthonormal_keys_are_a_memory():
    """alpha = 1, beta = 1, keys e_{pi(t)}: each step replaces row pi(t) of
    the state by v_t (the delta rule's exact overwrite), so reading with
    q = k_t returns v_t, and a key written twice keeps the later value."""
    DK, DV, NH = 6, 4, 2
    keys = [3, 1, 4, 1, 5, 3, 0]
    T = len(keys)
    g_ = synth.rng(2)
    v = synth.normal_f32(g_, (T, NH, DV)).astype(np.float64)
    k = np.zeros((T, NH, DK))
    for t, key in enumerate(keys):
        k[t, :, key] = 1.0
    o, s, _ = gdn_recurrent(k, k, v, np.zeros((T, NH)), np.ones((T, NH)))
    assert np.array_equal(o, v)
    last = {key: t for t, key in enumerate(keys)}
    for key in range(DK):
        want = v[last[key]] if key in last else np.zeros((NH, DV))
        assert np.array_equal(s[:, key, :], want)


def test_linear_in_values_and_initial_state():
    g_ = synth.rng(3)
    q, k, v1, gate, beta, s1 = synth.gdn_inputs(g_, 11, 2, 8, 6)
    v2 = synth.normal_f32(g_, v1.shape)
    s2 = synth.normal_f32(g_, s1.shape, 0.1)
    oa, sa, _ = gdn_recurrent(q, k, v1, gate, beta, s1)
    ob, sb, _ = gdn_recurrent(q, k, v2, gate, beta, s2)
    oc, sc, _ = gdn_recurrent(q, k, v1.astype(np.float64) + v2, gate, beta,
                              s1.astype(np.float64) + s2)
    assert np.allclose(oc, oa + ob, rtol=1e-12, atol=1e-12)
    assert np.allclose(sc, sa + sb, rtol=1e-12, atol=1e-12)


def test_state_handover_between_runs():
    g_ = synth.rng(4)
    q, k, v, gate, beta, s0 = synth.gdn_inputs(g_, 20, 3, 8, 4)
    o, s, _ = gdn_recurrent(q, k, v, gate, beta, s0)
    o1, s1, _ = gdn_recurrent(q[:7], k[:7], v[:7], gate[:7], beta[:7], s0)
    o2, s2, _ = gdn_recurrent(q[7:], k[7:], v[7:], gate[7:], beta[7:], s1)
    assert np.array_equal(np.concatenate([o1, o2]), o) and np.array_equal(s2, s)


def _chunkwise(q, k, v, g, beta, s0, C):
    """The same recurrence chunk by chunk, written from its closed form: with
    G_i = sum of g over the chunk up to token i, u_i = beta_i (v_i - alpha_i
    S_{i-1}^T k_i) gives S_i = e^{G_i} S0 + sum_{j<=i} e^{G_i-G_j} k_j u_j^T,
    so the u solve the unit lower-triangular system (I + A) U = diag(beta)
    (V - diag(e^G) K S0), A_ij = beta_i e^{G_i-G_j} k_i.k_j (j < i), and
    O = diag(e^G) Q S0 + (e^{G_i-G_j} q_i.k_j)_{j<=i} U."""
    q, k, v, g, beta = (np.asarray(a, np.float64) for a in (q, k, v, g, beta))
    T, NH, DK = k.shape
    S = np.array(s0, np.float64, copy=True)
    o = np.zeros((T, NH, v.shape[2]))
    for t0 in range(0, T, C):
        sl = slice(t0, min(T, t0 + C))
        for h in range(NH):
            K, Q, V = k[sl, h], q[sl, h], v[sl, h]
            G = np.cumsum(g[sl, h])
            b = beta[sl, h]
            n = len(G)
            D = np.exp(G[:, None] - G[None, :])
            A = np.tril(b[:, None] * D * (K @ K.T), -1)
            rhs = b[:, None] * (V - np.exp(G)[:, None] * (K @ S[h]))
            U = np.linalg.solve(np.eye(n) + A, rhs)
            P = np.tril(D * (Q @ K.T))
            o[sl, h] = np.exp(G)[:, None] * (Q @ S[h]) + P @ U
            S[h] = np.exp(G[-1]) * S[h] + K.T @ (np.exp(G[-1] - G)[:, None] * U)
    return o, S


@pytest.mark.parametrize("T,C", [(13, 4), (64, 32), (5, 8)])
def test_matches_an_independent_chunkwise_form(T, C):
    g_ = synth.rng(5 + T)
    q, k, v, gate, beta, s0 = synth.gdn_inputs(g_, T, 3, 16, 8)
    o, s, _ = gdn_recurrent(q, k, v, gate, beta, s0)
    oc, sc = _chunkwise(q, k, v, gate, beta, s0, C)
    assert np.allclose(oc, o, rtol=1e-11, atol=1e-12)
    assert np.allclose(sc, s, rtol=1e-11, atol=1e-12)
