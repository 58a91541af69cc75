"""Seeded synthetic inputs for the Mesa layer, shaped like MesaNet's workloads.

This module draws random numbers and nothing else: it holds none of the
layer's arithmetic, so both the HIP path and the fp64 oracle can consume its
output without sharing any of the method.  Distributions follow the layer's
front end (App. E): queries and keys are L2-normalised, forget and input gates
are sigmoids of Gaussian logits, and the regulariser Lambda is a positive
diagonal with the 0.25 lower bound of App. G.5 (here U[0.25, 1] per head and
dimension).  Key size 128 matches the 1B model (App. G.4), train length 2048 and
10-30 CG steps match Secs. 3-5 and App. G.7.  No dataset is used.

Draw order per workload: q, k, v, gamma logits, beta logits, lambda.  Values
are produced in fp64, rounded to fp32, and, for bf16 workloads, q/k/v are then
rounded to bf16 (round to nearest even) and returned as the fp32 numbers that
the bf16 values denote exactly.  Gates and lambda stay fp32.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class ForwardWorkload:
    name: str
    batch: int
    heads: int
    seq_len: int
    d_k: int
    d_v: int
    chunk: int
    n_cg: int
    dtype: str          # "f32" or "bf16": the dtype of q, k, v at the boundary
    gamma_mu: float     # mean of the forget-gate logits
    seed: int


@dataclass(frozen=True)
class DecodeWorkload:
    name: str
    seqs: int
    heads: int
    d_k: int
    d_v: int
    n_cg: int
    steps: int
    prefill: int        # gated updates that fill the state before the first step
    dtype: str
    gamma_mu: float
    seed: int
    step_seed: int = field(default=0)


# The five workloads: three sizes of sequence forward, a long-context forward,
# and a batched recurrent decode.
TINY_F32 = ForwardWorkload("tiny_f32_B1_H2_T256_d64", 1, 2, 256, 64, 64, 64, 10, "f32", 3.0, 0)
SMALL_F32 = ForwardWorkload("small_f32_B4_H8_T2048_d64", 4, 8, 2048, 64, 64, 64, 15, "f32", 3.0, 1)
LAYER_1B_BF16 = ForwardWorkload("layer1b_bf16_B8_H16_T2048_d128", 8, 16, 2048, 128, 128, 64, 15,
                                "bf16", 4.0, 2)
LONG_BF16 = ForwardWorkload("longctx_bf16_B1_H16_T16384_d128", 1, 16, 16384, 128, 128, 64, 20,
                            "bf16", 5.0, 3)
DECODE_BF16 = DecodeWorkload("decode_bf16_N256_H16_d128", 256, 16, 128, 128, 15, 1024, 4096,
                             "bf16", 4.0, 4, 1004)

FORWARD_WORKLOADS = (TINY_F32, SMALL_F32, LAYER_1B_BF16, LONG_BF16)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 array -> fp32 array of the nearest bf16 values (ties to even)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _unit_rows(rng, shape):
    x = rng.standard_normal(shape)
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _finish(x, dtype):
    x = np.asarray(x, dtype=np.float32)
    return round_to_bf16(x) if dtype == "bf16" else x


def forward_inputs(batch, heads, seq_len, d_k, d_v, dtype="f32", gamma_mu=3.0, seed=0):
    """Inputs of one forward call: dict of fp32 numpy arrays
    q, k [B,H,T,d_k], v [B,H,T,d_v], gamma, beta [B,H,T], lam [H,d_k]."""
    rng = np.random.default_rng(seed)
    q = _unit_rows(rng, (batch, heads, seq_len, d_k))
    k = _unit_rows(rng, (batch, heads, seq_len, d_k))
    v = rng.standard_normal((batch, heads, seq_len, d_v))
    gamma = _sigmoid(rng.normal(gamma_mu, 1.0, (batch, heads, seq_len)))
    beta = _sigmoid(rng.standard_normal((batch, heads, seq_len)))
    lam = rng.uniform(0.25, 1.0, (heads, d_k))
    return {
        "q": _finish(q, dtype), "k": _finish(k, dtype), "v": _finish(v, dtype),
        "gamma": gamma.astype(np.float32), "beta": beta.astype(np.float32),
        "lam": lam.astype(np.float32),
    }


def workload_inputs(w: ForwardWorkload, seed=None):
    return forward_inputs(w.batch, w.heads, w.seq_len, w.d_k, w.d_v, w.dtype, w.gamma_mu,
                          w.seed if seed is None else seed)


def decode_prefill_tokens(w: DecodeWorkload, seq_lo: int, seq_hi: int):
    """Prefill tokens (k, v, gamma, beta) for sequences [seq_lo, seq_hi) of a
    decode workload, [n, H, prefill, d] each.  Each sequence has its own
    generator (seeded from the workload seed and the sequence index), so any
    slice can be drawn alone and all slices agree."""
    ks, vs, gs, bs = [], [], [], []
    for s in range(seq_lo, seq_hi):
        rng = np.random.default_rng([w.seed, s])
        ks.append(_unit_rows(rng, (w.heads, w.prefill, w.d_k)))
        vs.append(rng.standard_normal((w.heads, w.prefill, w.d_v)))
        gs.append(_sigmoid(rng.normal(w.gamma_mu, 1.0, (w.heads, w.prefill))))
        bs.append(_sigmoid(rng.standard_normal((w.heads, w.prefill))))
    return {
        "k": _finish(np.stack(ks), w.dtype), "v": _finish(np.stack(vs), w.dtype),
        "gamma": np.stack(gs).astype(np.float32), "beta": np.stack(bs).astype(np.float32),
    }


def decode_lambda(w: DecodeWorkload):
    rng = np.random.default_rng([w.seed, 1 << 20])
    return rng.uniform(0.25, 1.0, (w.heads, w.d_k)).astype(np.float32)


def decode_step_inputs(w: DecodeWorkload, step: int, seqs=None):
    """Per-step token of every sequence: q, k [N,H,d_k], v [N,H,d_v], gamma, beta [N,H].
    Seeded by (step seed, step), so step i can be drawn without the others."""
    n = w.seqs if seqs is None else seqs
    rng = np.random.default_rng([w.step_seed, step])
    q = _unit_rows(rng, (n, w.heads, w.d_k))
    k = _unit_rows(rng, (n, w.heads, w.d_k))
    v = rng.standard_normal((n, w.heads, w.d_v))
    gamma = _sigmoid(rng.normal(w.gamma_mu, 1.0, (n, w.heads)))
    beta = _sigmoid(rng.standard_normal((n, w.heads)))
    return {
        "q": _finish(q, w.dtype), "k": _finish(k, w.dtype), "v": _finish(v, w.dtype),
        "gamma": gamma.astype(np.float32), "beta": beta.astype(np.float32),
    }


def repeated_key_inputs(batch, heads, seq_len, d_k, d_v, pool=1, dtype="bf16", gamma_mu=5.0,
                        seed=7):
    """Ill-conditioned stress input: keys drawn from a pool of `pool` unit
    vectors per head, gates near one.  Repeated tokens with gamma close to one
    are the case App. G.5 singles out as hard for the solver."""
    rng = np.random.default_rng(seed)
    q = _unit_rows(rng, (batch, heads, seq_len, d_k))
    pool_keys = _unit_rows(rng, (batch, heads, pool, d_k))
    idx = rng.integers(0, pool, (batch, heads, seq_len))
    k = np.take_along_axis(pool_keys, idx[..., None].repeat(d_k, -1), axis=2)
    v = rng.standard_normal((batch, heads, seq_len, d_v))
    gamma = _sigmoid(rng.normal(gamma_mu, 1.0, (batch, heads, seq_len)))
    beta = _sigmoid(rng.standard_normal((batch, heads, seq_len)))
    lam = rng.uniform(0.25, 1.0, (heads, d_k))
    return {
        "q": _finish(q, dtype), "k": _finish(k, dtype), "v": _finish(v, dtype),
        "gamma": gamma.astype(np.float32), "beta": beta.astype(np.float32),
        "lam": lam.astype(np.float32),
    }
