"""fp64 CPU oracle of the Mesa layer (MesaNet, arXiv 2506.05233).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product path
(``paper_2506_05233_amd``, ``libmesa``) never imports, links or calls it, and
it shares no code with that path.

The arithmetic lives in ``mesa_oracle.c`` (plain C, fp64, the sequential
recurrence of Sec. 2 / App. D with Alg. 1 conjugate gradients or an exact
Cholesky solve).  This module compiles it with gcc on first use, wraps it with
ctypes, and adds one more route to the states: the unrolled sums of App. D,
H_t = sum_i zeta_{t,i} beta_i k_i k_i^T and G_t = sum_i zeta_{t,i} beta_i v_i k_i^T,
with a numpy matmul as the summation step.

Every array argument is a numpy array; it is converted to contiguous float64.
Inputs that the GPU receives in bf16 or fp32 widen exactly to fp64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mesa_oracle.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD_DIR, "libmesa_oracle.so")

SOLVE_CG = 0
SOLVE_CHOLESKY = 1
INIT_JACOBI = 0
INIT_QUERY = 1

_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile mesa_oracle.c into oracle/_build/libmesa_oracle.so with gcc."""
    os.makedirs(_BUILD_DIR, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB_PATH)
            P = ctypes.POINTER(ctypes.c_double)
            i64, ci = ctypes.c_int64, ctypes.c_int
            I32 = ctypes.POINTER(ctypes.c_int32)
            dbl = ctypes.c_double
            lib.oracle_forward.argtypes = [P, P, P, P, P, P, i64, i64, i64, i64, i64, ci, ci, ci,
                                           dbl, P, P, P, P, I32, ci]
            lib.oracle_forward.restype = ci
            lib.oracle_decode_step.argtypes = [P, P, P, P, P, P, P, P, i64, i64, i64, i64, ci, ci,
                                               ci, dbl, P, P, I32, ci]
            lib.oracle_decode_step.restype = ci
            lib.oracle_backward.argtypes = [P, P, P, P, P, P, P, i64, i64, i64, i64, i64, ci, ci,
                                            ci, P, P, P, P, P, P, P, P, ci]
            lib.oracle_backward.restype = ci
            lib.oracle_cg.argtypes = [P, P, i64, ci, ci, dbl, P, P]
            lib.oracle_cg.restype = ci
            lib.oracle_cholesky_solve.argtypes = [P, P, i64, P, P]
            lib.oracle_cholesky_solve.restype = ci
            _lib = lib
    return _lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _iptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _eps(eps):
    eps = float(eps)
    if not eps >= 0.0 or eps == float("inf"):
        raise ValueError("eps must be finite and >= 0")
    return eps


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def forward(q, k, v, gamma, beta, lam, n_cg, solver="cg", init="jacobi", want_qstar=False,
            want_states=False, threads=None, eps=0.0, want_steps=False):
    """Sequential Mesa forward over [B, H, T, d] inputs.

    solver: "cg" (Alg. 1, at most n_cg loop iterations, relative tolerance eps;
            eps = 0 is the fixed-step solve) or "cholesky" (exact; n_cg ignored).
    init:   "jacobi" (x0 = q / diag(H_t + Lambda), the paper's choice) or
            "query" (x0 = q; only to check the GLA remark with n_cg = 0).
    Returns a dict with "out" [B,H,T,dv] and, if asked, "qstar" [B,H,T,dk],
    "H" [B,H,dk,dk], "G" [B,H,dv,dk] (final states), "steps" [B,H,T] int32
    (CG iterations per token).
    """
    lib = _load()
    q, k, v, gamma, beta, lam = map(_f64, (q, k, v, gamma, beta, lam))
    B, Hh, T, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == (B, Hh, T, dk) and v.shape == (B, Hh, T, dv)
    assert gamma.shape == (B, Hh, T) and beta.shape == (B, Hh, T) and lam.shape == (Hh, dk)
    out = np.zeros((B, Hh, T, dv))
    qstar = np.zeros((B, Hh, T, dk)) if want_qstar else None
    fH = np.zeros((B, Hh, dk, dk)) if want_states else None
    fG = np.zeros((B, Hh, dv, dk)) if want_states else None
    steps = np.zeros((B, Hh, T), dtype=np.int32) if want_steps else None
    s = {"cg": SOLVE_CG, "cholesky": SOLVE_CHOLESKY}[solver]
    i = {"jacobi": INIT_JACOBI, "query": INIT_QUERY}[init]
    rc = lib.oracle_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam),
                            B, Hh, T, dk, dv, int(n_cg), s, i, _eps(eps), _ptr(out), _ptr(qstar),
                            _ptr(fH), _ptr(fG), _iptr(steps), int(threads or default_threads()))
    if rc != 0:
        raise FloatingPointError("oracle: a system H_t + Lambda was not positive definite")
    res = {"out": out}
    if want_qstar:
        res["qstar"] = qstar
    if want_states:
        res["H"] = fH
        res["G"] = fG
    if want_steps:
        res["steps"] = steps
    return res


def decode_step(state_H, state_G, q, k, v, gamma, beta, lam, n_cg, solver="cg", init="jacobi",
                want_qstar=False, threads=None, eps=0.0, steps_out=None):
    """One recurrent step on [N, H, ...] states.  Returns (out, H_new, G_new[, qstar]).
    eps: CG relative tolerance (0: fixed steps); steps_out: optional int32 [N, H]
    array that receives the CG iterations of every (sequence, head)."""
    lib = _load()
    H = _f64(state_H).copy()
    G = _f64(state_G).copy()
    q, k, v, gamma, beta, lam = map(_f64, (q, k, v, gamma, beta, lam))
    N, Hh, dk = q.shape
    dv = v.shape[-1]
    assert H.shape == (N, Hh, dk, dk) and G.shape == (N, Hh, dv, dk)
    out = np.zeros((N, Hh, dv))
    qstar = np.zeros((N, Hh, dk)) if want_qstar else None
    s = {"cg": SOLVE_CG, "cholesky": SOLVE_CHOLESKY}[solver]
    i = {"jacobi": INIT_JACOBI, "query": INIT_QUERY}[init]
    if steps_out is not None:
        assert steps_out.shape == (N, Hh) and steps_out.dtype == np.int32 and steps_out.flags.c_contiguous
    rc = lib.oracle_decode_step(_ptr(H), _ptr(G), _ptr(q), _ptr(k), _ptr(v), _ptr(gamma),
                                _ptr(beta), _ptr(lam), N, Hh, dk, dv, int(n_cg), s, i, _eps(eps),
                                _ptr(out), _ptr(qstar), _iptr(steps_out),
                                int(threads or default_threads()))
    if rc != 0:
        raise FloatingPointError("oracle: a system H_t + Lambda was not positive definite")
    if want_qstar:
        return out, H, G, qstar
    return out, H, G


def backward(q, k, v, gamma, beta, lam, dout, n_cg, solver="cg", init="jacobi", want_solves=False,
             threads=None):
    """Gradients of the Mesa layer (App. D backward pass) given dout = dL/do [B,H,T,dv].

    q*_t and e*_t = (H_t + Lambda)^{-1} G_t^T e_t come from the same solver
    ("cg": Alg. 1 with n_cg loop iterations, tolerance zero; "cholesky": exact).
    Returns a dict with "dq", "dk" [B,H,T,dk], "dv" [B,H,T,dv], "dgamma",
    "dbeta" [B,H,T], "dlam" [H,dk] (summed over batch and time) and, with
    want_solves, "qstar" and "estar" [B,H,T,dk].
    """
    lib = _load()
    q, k, v, gamma, beta, lam, dout = map(_f64, (q, k, v, gamma, beta, lam, dout))
    B, Hh, T, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == (B, Hh, T, dk) and v.shape == (B, Hh, T, dv) and dout.shape == (B, Hh, T, dv)
    assert gamma.shape == (B, Hh, T) and beta.shape == (B, Hh, T) and lam.shape == (Hh, dk)
    res = {"dq": np.zeros((B, Hh, T, dk)), "dk": np.zeros((B, Hh, T, dk)), "dv": np.zeros((B, Hh, T, dv)),
           "dgamma": np.zeros((B, Hh, T)), "dbeta": np.zeros((B, Hh, T))}
    dlam_part = np.zeros((B, Hh, dk))
    qstar = np.zeros((B, Hh, T, dk)) if want_solves else None
    estar = np.zeros((B, Hh, T, dk)) if want_solves else None
    s = {"cg": SOLVE_CG, "cholesky": SOLVE_CHOLESKY}[solver]
    i = {"jacobi": INIT_JACOBI, "query": INIT_QUERY}[init]
    rc = lib.oracle_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam), _ptr(dout),
                             B, Hh, T, dk, dv, int(n_cg), s, i, _ptr(res["dq"]), _ptr(res["dk"]),
                             _ptr(res["dv"]), _ptr(res["dgamma"]), _ptr(res["dbeta"]), _ptr(dlam_part),
                             _ptr(qstar), _ptr(estar), int(threads or default_threads()))
    if rc != 0:
        raise FloatingPointError("oracle: a system H_t + Lambda was not positive definite")
    res["dlam"] = dlam_part.sum(axis=0)
    if want_solves:
        res["qstar"] = qstar
        res["estar"] = estar
    return res


def cg_solve(A, b, n_cg, init="jacobi", eps=0.0, return_steps=False):
    """Alg. 1 on one SPD system (at most n_cg iterations, relative tolerance eps);
    returns x, or (x, iterations) with return_steps."""
    lib = _load()
    A = _f64(A)
    b = _f64(b)
    n = b.shape[0]
    x = np.zeros(n)
    work = np.zeros(3 * n)
    it = lib.oracle_cg(_ptr(A), _ptr(b), n, int(n_cg), {"jacobi": INIT_JACOBI, "query": INIT_QUERY}[init],
                       _eps(eps), _ptr(x), _ptr(work))
    return (x, it) if return_steps else x


def cholesky_solve(A, b):
    lib = _load()
    A = _f64(A)
    b = _f64(b)
    n = b.shape[0]
    x = np.zeros(n)
    work = np.zeros(n * n)
    if lib.oracle_cholesky_solve(_ptr(A), _ptr(b), n, _ptr(x), _ptr(work)) != 0:
        raise FloatingPointError("oracle: matrix is not positive definite")
    return x


def unrolled_states(k, v, gamma, beta):
    """Final states after T tokens from the unrolled sums of App. D:
    H_T = sum_i zeta_{T,i} beta_i k_i k_i^T,  G_T = sum_i zeta_{T,i} beta_i v_i k_i^T,
    with zeta_{T,i} = prod_{s=i+1..T} gamma_s (zeta_{T,T} = 1).

    k [..., T, dk], v [..., T, dv], gamma/beta [..., T] -> (H [..., dk, dk], G [..., dv, dk]).
    The weights come from a reversed cumulative product; the sums are one matmul.
    """
    k, v, gamma, beta = map(_f64, (k, v, gamma, beta))
    T = gamma.shape[-1]
    # suffix products: zeta_{T,i} = prod_{s>i} gamma_s
    shifted = np.concatenate([gamma[..., 1:], np.ones(gamma.shape[:-1] + (1,))], axis=-1)
    zeta = np.flip(np.cumprod(np.flip(shifted, -1), axis=-1), -1)
    w = zeta * beta
    assert w.shape[-1] == T
    kw = k * w[..., None]
    H = np.matmul(np.swapaxes(kw, -1, -2), k)
    G = np.matmul(np.swapaxes(v * w[..., None], -1, -2), k)
    return H, G
