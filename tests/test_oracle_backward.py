"""Pins of the oracle's backward pass (App. D, "Mesa layer backward pass").

The oracle computes the gradients by walking the state adjoints backwards in
time.  These tests tie it to things other than itself: central finite
differences of the exact (Cholesky) forward, the converged-CG special case, and
a brute-force evaluation of the paper's sums over t >= s with the states
materialised token by token.
"""
import numpy as np
import pytest

import oracle


def _inputs(B, H, T, dk, dv, seed, gamma_lo=0.5):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(B, H, T, dk))
    k = rng.normal(size=(B, H, T, dk)) / np.sqrt(dk)
    v = rng.normal(size=(B, H, T, dv))
    g = rng.uniform(gamma_lo, 0.97, size=(B, H, T))
    b = rng.uniform(0.2, 0.9, size=(B, H, T))
    lam = rng.uniform(0.25, 1.0, size=(H, dk))
    e = rng.normal(size=(B, H, T, dv))
    return dict(q=q, k=k, v=v, gamma=g, beta=b, lam=lam), e


def _loss(x, e):
    out = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 0, solver="cholesky")["out"]
    return float((out * e).sum())


def _rel(a, b):
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(b), 1e-300))


def test_backward_matches_finite_differences():
    """Every gradient of L = sum_t e_t . o_t against central differences of the
    exact forward.  T = 70 crosses the oracle's 64-token checkpoint block; a zero
    forget gate sits inside; B = H = 2 makes dLambda a sum over the batch; d_k != d_v
    catches transposed operands."""
    x, e = _inputs(2, 2, 70, 5, 3, seed=1)
    x["gamma"][1, 0, 30] = 0.0
    g = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], e, 0, solver="cholesky")
    h = 1e-6
    rng = np.random.default_rng(2)
    for name, key in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("gamma", "dgamma"), ("beta", "dbeta"), ("lam", "dlam")):
        a = x[name]
        flat = list(np.ndindex(a.shape))
        idx = [flat[i] for i in rng.choice(len(flat), size=min(len(flat), 160), replace=False)]
        fd, an = [], []
        for ix in idx:
            xp = dict(x); xp[name] = a.copy(); xp[name][ix] += h
            xm = dict(x); xm[name] = a.copy(); xm[name][ix] -= h
            fd.append((_loss(xp, e) - _loss(xm, e)) / (2 * h))
            an.append(g[key][ix])
        err = _rel(an, fd)
        assert err < 1e-7, (name, err)


def test_backward_converged_cg_equals_exact():
    """CG with n_cg = d_k loop iterations is exact in exact arithmetic, so both solves
    of the backward and every gradient must agree with the Cholesky route."""
    x, e = _inputs(1, 2, 40, 8, 6, seed=3)
    a = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], e, 8, solver="cg")
    b = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], e, 0, solver="cholesky")
    for key in ("dq", "dk", "dv", "dgamma", "dbeta", "dlam"):
        assert _rel(a[key], b[key]) < 1e-9, key


def _paper_sums(x, e, estar_value_term):
    """The paper's gradient sums over t >= s, evaluated by brute force for one
    (batch, head) with the input gate written in: states are built token by token,
    zeta_{t,s} = prod_{s<u<=t} gamma_u.  estar_value_term selects the literal form
    of the value term of dL/dk_s (q*_t e*_t^T v_s) instead of q*_t e_t^T v_s."""
    q, k, v, g, b = (x[n][0, 0] for n in ("q", "k", "v", "gamma", "beta"))
    lam = x["lam"][0]
    ee = e[0, 0]
    T, dk = q.shape
    dv = v.shape[1]
    Hs, Gs = [np.zeros((dk, dk))], [np.zeros((dv, dk))]
    for t in range(T):
        Hs.append(g[t] * Hs[-1] + b[t] * np.outer(k[t], k[t]))
        Gs.append(g[t] * Gs[-1] + b[t] * np.outer(v[t], k[t]))
    A = [Hs[t + 1] + np.diag(lam) for t in range(T)]
    qs = np.stack([np.linalg.solve(A[t], q[t]) for t in range(T)])
    es = np.stack([np.linalg.solve(A[t], Gs[t + 1].T @ ee[t]) for t in range(T)])
    zeta = np.ones((T, T))
    for t in range(T):
        for s in range(t):
            zeta[t, s] = np.prod(g[s + 1:t + 1])
    dv_ = np.zeros((T, dv)); dk_ = np.zeros((T, dk)); dg = np.zeros(T); db = np.zeros(T)
    for s in range(T):
        for t in range(s, T):
            z = zeta[t, s]
            vt = es[t] if estar_value_term else ee[t]
            dv_[s] += z * b[s] * ee[t] * (qs[t] @ k[s])
            dk_[s] += z * b[s] * (qs[t] * (vt @ v[s]) - es[t] * (qs[t] @ k[s]) - qs[t] * (es[t] @ k[s]))
            db[s] += z * ((ee[t] @ v[s]) * (k[s] @ qs[t]) - (k[s] @ es[t]) * (qs[t] @ k[s]))
            dg[s] += z * (qs[t] @ Gs[s].T @ ee[t] - es[t] @ Hs[s] @ qs[t])
    return dict(dq=es, dk=dk_, dv=dv_, dgamma=dg, dbeta=db, dlam=-(qs * es).sum(0))


def test_backward_equals_paper_sums():
    """The adjoint walk equals the paper's sums over t >= s (input gate included)."""
    x, e = _inputs(1, 1, 23, 6, 4, seed=5)
    got = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], e, 0, solver="cholesky")
    ref = _paper_sums(x, e, estar_value_term=False)
    for key in ("dq", "dk", "dv", "dgamma", "dbeta"):
        assert _rel(got[key][0, 0], ref[key]) < 1e-10, key
    assert _rel(got["dlam"][0], ref["dlam"]) < 1e-10


def test_value_term_of_dk_reads_e_not_estar():
    """The paper prints q*_t e*_t^T v_s as the first term of dL/dk_s; differentiating
    e_t^T G_t q*_t gives q*_t e_t^T v_s.  The literal form is defined only when
    d_k = d_v (e*_t has d_k entries, v_s has d_v), so it is evaluated there: it
    disagrees with finite differences, the reading adopted by the oracle agrees."""
    x, e = _inputs(1, 1, 12, 4, 4, seed=7)
    literal = _paper_sums(x, e, estar_value_term=True)["dk"]
    adopted = _paper_sums(x, e, estar_value_term=False)["dk"]
    h = 1e-6
    fd = np.zeros_like(adopted)
    for ix in np.ndindex(fd.shape):
        xp = dict(x); xp["k"] = x["k"].copy(); xp["k"][(0, 0) + ix] += h
        xm = dict(x); xm["k"] = x["k"].copy(); xm["k"][(0, 0) + ix] -= h
        fd[ix] = (_loss(xp, e) - _loss(xm, e)) / (2 * h)
    assert _rel(adopted, fd) < 1e-7
    assert _rel(literal, fd) > 1e-2


def test_backward_degenerate_cases():
    """dout = 0 gives zero gradients; with every beta = 0 the states stay zero, so
    o = 0 whatever q: dq = dv = dgamma = 0, dk = 0, and only dbeta is non-zero."""
    x, e = _inputs(1, 2, 20, 4, 4, seed=9)
    z = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], np.zeros_like(e), 0, solver="cholesky")
    for key in ("dq", "dk", "dv", "dgamma", "dbeta", "dlam"):
        assert np.all(z[key] == 0.0), key
    x["beta"][...] = 0.0
    g = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], e, 0, solver="cholesky")
    for key in ("dq", "dk", "dv", "dgamma", "dlam"):
        assert np.all(g[key] == 0.0), key
    assert np.abs(g["dbeta"]).max() > 0.0
