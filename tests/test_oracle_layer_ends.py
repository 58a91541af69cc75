"""Pins of the oracle's front and back end of the Mesa layer (oracle/layer_ends.py)
against what the paper and the mathematics fix: hand-worked values
(tests/golden/layer_ends_worked.json, App. E and App. G.5), an independent library
convolution, impulse responses, identities of SiLU and softplus, the unit norm of keys
and queries, the limits of the gate cap, the floor of Lambda and the invariances of the
RMSNorm."""
import json
import os

import numpy as np
import pytest

from oracle import layer_ends as E

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "layer_ends_worked.json")))


def test_golden_conv():
    g = GOLD["conv"]
    x = np.array(g["x"])[:, None]
    w = np.array(g["w"])[None, :]
    assert np.array_equal(E.short_conv(x, w)[:, 0], np.array(g["y"]))  # dyadic: exact


def test_golden_silu_l2_gates_lambda_rms():
    g = GOLD["silu"]
    np.testing.assert_allclose(E.silu(g["x"]), g["y"], rtol=1e-15, atol=1e-300)
    np.testing.assert_allclose(E.l2_normalize(np.array(GOLD["l2"]["x"]), 0.0), GOLD["l2"]["y"], rtol=1e-15)
    g = GOLD["gates"]
    gamma, beta = E.gates(np.array(g["a_gamma"]), np.array(g["a_beta"]), 0.9975)
    np.testing.assert_allclose(beta, g["beta"], rtol=1e-15)
    np.testing.assert_allclose(gamma, g["gamma"], rtol=1e-14)
    np.testing.assert_allclose(E.regulariser(np.array(GOLD["lambda"]["theta"])), GOLD["lambda"]["lam"], rtol=1e-15)
    g = GOLD["rmsnorm"]
    o = np.array(g["o"])[None, None, None, :]
    y = E.output_norm(o, np.array(g["w"])[None, :], eps=0.0)
    np.testing.assert_allclose(y[0, 0, 0], g["y"], rtol=1e-15)


def test_conv_matches_library_convolution_per_channel():
    """numpy's full convolution of each channel with its filter, cut to the first T
    samples, is the causal window-4 convolution with zeros before the start."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 37, 5))
    w = rng.standard_normal((5, 4))
    y = E.short_conv(x, w)
    for b in range(2):
        for c in range(5):
            np.testing.assert_allclose(y[b, :, c], np.convolve(x[b, :, c], w[c])[:37], rtol=1e-13, atol=1e-14)


def test_conv_impulse_response_is_causal_and_ordered():
    """An impulse at t0 produces w_1 .. w_4 at t0 .. t0+3 and nothing before it: a
    filter applied acausally or in reversed tap order fails."""
    T, t0 = 12, 5
    w = np.array([[1.0, 10.0, 100.0, 1000.0]])
    x = np.zeros((T, 1))
    x[t0, 0] = 1.0
    y = E.short_conv(x, w)[:, 0]
    want = np.zeros(T)
    want[t0:t0 + 4] = w[0]
    assert np.array_equal(y, want)
    # tokens shorter than the window: only the taps that reach a token enter
    assert np.array_equal(E.short_conv(np.ones((2, 1)), w)[:, 0], [1.0, 11.0])


def test_silu_and_softplus_identities():
    x = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(E.silu(x) - E.silu(-x), x, rtol=1e-14, atol=1e-13)
    np.testing.assert_allclose(E.softplus(x) - E.softplus(-x), x, rtol=1e-14, atol=1e-13)
    assert E.silu(0.0) == 0.0 and abs(E.silu(40.0) - 40.0) < 1e-15
    h = 1e-6
    assert abs((E.silu(h) - E.silu(-h)) / (2 * h) - 0.5) < 1e-9   # SiLU'(0) = sigma(0) = 1/2
    assert np.all(E.regulariser(np.linspace(-50, 50, 101)) >= 0.25)


def test_gate_cap_limits():
    """With beta = 1 the forget gate tends to b_gamma as its logit grows (App. G.5's cap);
    with beta -> 0 it is the plain sigmoid; gates stay in [0, 1]."""
    g, b = E.gates(np.array([40.0]), np.array([40.0]), 0.9975)
    assert abs(g[0] - 0.9975) < 1e-12 and abs(b[0] - 1.0) < 1e-15
    g, b = E.gates(np.array([1.3]), np.array([-40.0]), 0.9975)
    assert abs(g[0] - E.sigmoid(1.3)) < 1e-15
    g, b = E.gates(np.array([0.7]), np.array([0.4]), 1.0)   # b_gamma = 1: no cap
    assert abs(g[0] - E.sigmoid(0.7)) < 1e-15
    rng = np.random.default_rng(2)
    g, b = E.gates(rng.normal(0, 5, 1000), rng.normal(0, 5, 1000), 0.9975)
    assert np.all((g >= 0) & (g <= 1) & (b >= 0) & (b <= 1)) and np.all(g <= 1 - (1 - 0.9975) * b * b)


def _frontend_inputs(B=2, T=9, H=3, dk=4, dv=5, seed=3):
    rng = np.random.default_rng(seed)
    return dict(qp=rng.standard_normal((B, T, H, dk)), kp=rng.standard_normal((B, T, H, dk)),
                vp=rng.standard_normal((B, T, H, dv)), conv_q=rng.standard_normal((H * dk, 4)),
                conv_k=rng.standard_normal((H * dk, 4)), conv_v=rng.standard_normal((H * dv, 4)),
                a_gamma=rng.standard_normal((B, T, H)), a_beta=rng.standard_normal((B, T, H)),
                theta=rng.standard_normal((H, dk)))


def test_frontend_brute_force_per_element():
    """Every output of the fused front end against a per-element evaluation of the
    definitions (explicit tap loop, scalar SiLU and norm), with eps 0."""
    a = _frontend_inputs()
    out = E.frontend(**a, gamma_cap=0.99, l2_eps=0.0)
    B, T, H, dk = a["qp"].shape
    dv = a["vp"].shape[-1]
    for name, src, w, d, norm in (("q", "qp", "conv_q", dk, True), ("k", "kp", "conv_k", dk, True),
                                  ("v", "vp", "conv_v", dv, False)):
        for b in range(B):
            for h in range(H):
                for t in range(T):
                    z = np.zeros(d)
                    for c in range(d):
                        s = 0.0
                        for i in range(4):
                            if t - i >= 0:
                                s += a[w][h * d + c, i] * a[src][b, t - i, h, c]
                        z[c] = s / (1.0 + np.exp(-s))
                    if norm:
                        z = z / np.sqrt(np.sum(z * z))
                    np.testing.assert_allclose(out[name][b, h, t], z, rtol=1e-12, atol=1e-14)
    for b in range(B):
        for h in range(H):
            for t in range(T):
                beta = 1.0 / (1.0 + np.exp(-a["a_beta"][b, t, h]))
                gamma = 1.0 / (1.0 + np.exp(-a["a_gamma"][b, t, h])) * (1.0 - 0.01 * beta * beta)
                assert abs(out["beta"][b, h, t] - beta) < 1e-15 and abs(out["gamma"][b, h, t] - gamma) < 1e-15


def test_frontend_unit_norm_direction_and_value_passthrough():
    a = _frontend_inputs(seed=4)
    out = E.frontend(**a, l2_eps=1e-12)
    np.testing.assert_allclose(np.linalg.norm(out["q"], axis=-1), 1.0, rtol=1e-10)
    np.testing.assert_allclose(np.linalg.norm(out["k"], axis=-1), 1.0, rtol=1e-10)
    # scaling a projection by c > 0 changes the convolution by c, SiLU not linearly:
    # the normalised direction of keys changes, but a zero projection stays zero
    z = dict(a)
    z["kp"] = np.zeros_like(a["kp"])
    assert np.all(E.frontend(**z)["k"] == 0.0)
    # without a value filter the values pass through, only transposed
    a["conv_v"] = None
    out = E.frontend(**a)
    assert np.array_equal(out["v"], a["vp"].transpose(0, 2, 1, 3))


def test_output_norm_invariances():
    rng = np.random.default_rng(5)
    o = rng.standard_normal((2, 3, 7, 8))
    w = rng.standard_normal((3, 8))
    y = E.output_norm(o, w, eps=0.0)
    assert y.shape == (2, 7, 3, 8)
    np.testing.assert_allclose(np.mean((y / w[None, None]) ** 2, axis=-1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(E.output_norm(3.5 * o, w, eps=0.0), y, rtol=1e-12)
    # head h of token t is o[b, h, t] normalised with weight row h
    np.testing.assert_allclose(y[1, 4, 2], o[1, 2, 4] / np.sqrt(np.mean(o[1, 2, 4] ** 2)) * w[2], rtol=1e-13)
