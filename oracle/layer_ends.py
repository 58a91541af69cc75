"""fp64 CPU oracle of the Mesa layer's front and back end (MesaNet, arXiv 2506.05233).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module; the product path never
imports, links or calls it, and it shares no code with that path.

What it computes, written from App. E ("A Full Description of the Mesa Layer")
and App. G.5 ("Notes on precision used in the CG-solver"), per head h:

  front end, from the projections q_t = W_q e_t, k_t = W_k e_t, v_t = W_v e_t and
  the gate projections a_t^gamma = e_t W_gamma + b_gamma, a_t^beta = e_t W_beta + b_beta:
    short convolution in time, window 4:  x_t <- sum_{i=0..3} w_{i+1} x_{t-i}
        (one filter per feature channel; x_s = 0 before the first token)
    SiLU(x) = x sigma(x), then keys and queries (not values) normalised to unit L2 norm
    input gate beta_t = sigma(a_t^beta)
    forget gate gamma_t = sigma(a_t^gamma) s_t,  s_t = 1 - (1 - b_gamma) beta_t^2
        (the cap of App. G.5: with beta_t = 1 the gate stays below b_gamma = 0.9975)
    regulariser Lambda = 0.25 + softplus(theta)   (App. G.5's lower bound 0.25)
  back end: the head's output through its RMSNorm before the output projection,
    y_t = o_t / sqrt(mean(o_t^2) + eps) * w_h.

Readings where the paper is silent:
  - the convolution is depthwise (one 4-tap filter per channel of every head) and
    causal with zeros before the sequence start; the paper's w_{i+1} multiplies x_{t-i};
  - the values take the convolution and SiLU only when a filter for them is given
    (App. E convolves "them" after all three projections, App. G.2 convolves keys and
    queries), and are never normalised;
  - the L2 normalisation divides by sqrt(|x|^2 + eps_l2) (eps_l2 small, so a zero
    vector stays zero); the RMSNorm divides by sqrt(mean(o^2) + eps_rms) and scales by
    a learnable weight per head and feature;
  - the input gate enters the cap as beta_t^2 exactly as printed.

Layouts: projections [B, T, H, d] (the heads of a token side by side, as a projection
produces them); the layer's inputs q, k [B, H, T, d_k], v [B, H, T, d_v], gamma, beta
[B, H, T], Lambda [H, d_k]; the back end's output [B, T, H, d_v].
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def sigmoid(x):
    """sigma(x) = 1 / (1 + exp(-x))."""
    return 1.0 / (1.0 + np.exp(-_f64(x)))


def silu(x):
    """SiLU(x) = x sigma(x) (App. E)."""
    x = _f64(x)
    return x * sigmoid(x)


def softplus(x):
    """log(1 + exp(x)), evaluated as max(x, 0) + log(1 + exp(-|x|))."""
    x = _f64(x)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def short_conv(x, w):
    """Causal convolution of window 4 along time (App. E): y_t = sum_{i=0..3} w[c, i] x_{t-i}
    for every channel c, with x_s = 0 for s < 0.  x [..., T, C], w [C, 4]."""
    x, w = _f64(x), _f64(w)
    T = x.shape[-2]
    y = np.zeros_like(x)
    for i in range(4):
        if i < T:
            y[..., i:, :] += w[:, i] * x[..., :T - i, :]
    return y


def l2_normalize(x, eps):
    """x / sqrt(|x|^2 + eps) over the last axis."""
    x = _f64(x)
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def gates(a_gamma, a_beta, gamma_cap):
    """Input and forget gates of App. E with the cap of App. G.5:
    beta = sigma(a_beta), gamma = sigma(a_gamma) (1 - (1 - gamma_cap) beta^2)."""
    beta = sigmoid(a_beta)
    gamma = sigmoid(a_gamma) * (1.0 - (1.0 - float(gamma_cap)) * beta * beta)
    return gamma, beta


def regulariser(theta):
    """Lambda = 0.25 + softplus(theta) (App. G.5)."""
    return 0.25 + softplus(theta)


def frontend(qp, kp, vp, conv_q, conv_k, conv_v, a_gamma, a_beta, theta, gamma_cap=0.9975,
             l2_eps=1e-6):
    """The layer's inputs from the projections.

    qp, kp [B, T, H, d_k], vp [B, T, H, d_v]; conv_q, conv_k [H*d_k, 4], conv_v
    [H*d_v, 4] or None; a_gamma, a_beta [B, T, H]; theta [H, d_k].
    Returns a dict: q, k [B, H, T, d_k], v [B, H, T, d_v], gamma, beta [B, H, T],
    lam [H, d_k].
    """
    qp, kp, vp = _f64(qp), _f64(kp), _f64(vp)
    B, T, H, dk = qp.shape
    dv = vp.shape[-1]

    def conv_silu(x, w, d):
        y = short_conv(x.reshape(B, T, H * d), w)
        return silu(y).reshape(B, T, H, d)

    q = l2_normalize(conv_silu(qp, conv_q, dk), l2_eps)
    k = l2_normalize(conv_silu(kp, conv_k, dk), l2_eps)
    v = conv_silu(vp, conv_v, dv) if conv_v is not None else vp
    gamma, beta = gates(a_gamma, a_beta, gamma_cap)
    return {
        "q": np.ascontiguousarray(q.transpose(0, 2, 1, 3)),
        "k": np.ascontiguousarray(k.transpose(0, 2, 1, 3)),
        "v": np.ascontiguousarray(v.transpose(0, 2, 1, 3)),
        "gamma": np.ascontiguousarray(gamma.transpose(0, 2, 1)),
        "beta": np.ascontiguousarray(beta.transpose(0, 2, 1)),
        "lam": regulariser(theta),
    }


def output_norm(o, weight, eps=1e-6):
    """Per-head RMSNorm of the layer's output (App. E): o [B, H, T, d_v], weight [H, d_v]
    -> y [B, T, H, d_v] = o / sqrt(mean(o^2) + eps) * weight[h]."""
    o, weight = _f64(o), _f64(weight)
    y = o / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps) * weight[None, :, None, :]
    return np.ascontiguousarray(y.transpose(0, 2, 1, 3))
