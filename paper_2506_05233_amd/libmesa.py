"""Thin ctypes binding of libmesa (include/libmesa.h).

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity, then their data pointers and torch's current HIP stream go to the C
ABI.  Every step of the layer runs in libmesa's HIP kernels; there is no
fallback.  Loading fails loudly when the built library is missing.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libmesa.so")

MESA_DTYPE_F32 = 0
MESA_DTYPE_BF16 = 1
MESA_PREC_AUTO = 0
MESA_PREC_F32 = 1
MESA_PREC_BF16 = 2
MESA_PREC_BF16X3 = 3
MESA_OK = 0
MESA_ERR_NULL = 1
MESA_ERR_SHAPE = 2
MESA_ERR_UNSUPPORTED = 3
MESA_ERR_ARG = 4
MESA_ERR_WORKSPACE = 5
MESA_ERR_HIP = 6
MESA_ERR_NONFINITE = 7
MESA_MAX_NCG = 1024
MESA_NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTED = ("mesa_forward", "mesa_forward_ex", "mesa_forward_states", "mesa_forward_solve",
            "mesa_forward_tol", "mesa_forward_workspace_bytes", "mesa_decode_step",
            "mesa_decode_step_tol", "mesa_decode_step_packed", "mesa_pack_state", "mesa_unpack_state",
            "mesa_backward", "mesa_backward_workspace_bytes", "mesa_forward_noalloc",
            "mesa_frontend", "mesa_output_norm",
            "mesa_status_string", "mesa_version")

_lib = None


class MesaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (where, status_string(status), status))


def load():
    """Load libmesa.so (built by paper_2506_05233_amd/build.py); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libmesa is not built: %s is missing (run __graft_entry__.build())" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, fp, i64, ci, sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
    lib.mesa_forward_workspace_bytes.argtypes = [i64, i64, i64, i64, i64, ci]
    lib.mesa_forward_workspace_bytes.restype = sz
    lib.mesa_forward.argtypes = [vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, fp, vp, sz, vp]
    lib.mesa_forward.restype = ci
    lib.mesa_forward_ex.argtypes = [vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, ci,
                                    fp, fp, fp, fp, vp, sz, vp]
    lib.mesa_forward_ex.restype = ci
    lib.mesa_forward_states.argtypes = [vp, vp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, fp, fp, vp, sz, vp]
    lib.mesa_forward_states.restype = ci
    lib.mesa_forward_solve.argtypes = [vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, ci,
                                       fp, fp, vp, sz, vp]
    lib.mesa_forward_solve.restype = ci
    lib.mesa_decode_step.argtypes = [fp, fp, vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, ci, ci, fp, vp]
    lib.mesa_decode_step.restype = ci
    cf = ctypes.c_float
    lib.mesa_forward_tol.argtypes = [vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, cf, ci, ci,
                                     fp, fp, vp, vp, sz, vp]
    lib.mesa_forward_tol.restype = ci
    lib.mesa_decode_step_tol.argtypes = [fp, fp, vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, ci, ci, cf,
                                         fp, vp, vp]
    lib.mesa_decode_step_tol.restype = ci
    lib.mesa_decode_step_packed.argtypes = [fp, fp, vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, ci, ci, cf,
                                            fp, vp, vp]
    lib.mesa_decode_step_packed.restype = ci
    lib.mesa_pack_state.argtypes = [fp, fp, i64, i64, i64, vp]
    lib.mesa_pack_state.restype = ci
    lib.mesa_unpack_state.argtypes = [fp, fp, i64, i64, i64, vp]
    lib.mesa_unpack_state.restype = ci
    lib.mesa_backward_workspace_bytes.argtypes = [i64, i64, i64, i64, i64]
    lib.mesa_backward_workspace_bytes.restype = sz
    lib.mesa_backward.argtypes = [vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, fp, fp,
                                  fp, fp, fp, fp, fp, fp, vp, sz, vp]
    lib.mesa_backward.restype = ci
    lib.mesa_forward_noalloc.argtypes = [vp, vp, vp, fp, fp, fp, i64, i64, i64, i64, i64, ci, ci, ci, fp, vp]
    lib.mesa_forward_noalloc.restype = ci
    lib.mesa_frontend.argtypes = [vp, vp, vp, fp, fp, fp, fp, fp, fp, cf, cf, i64, i64, i64, i64, i64, ci,
                                   vp, vp, vp, fp, fp, fp, vp]
    lib.mesa_frontend.restype = ci
    lib.mesa_output_norm.argtypes = [fp, fp, cf, i64, i64, i64, i64, ci, vp, vp]
    lib.mesa_output_norm.restype = ci
    lib.mesa_status_string.argtypes = [ci]
    lib.mesa_status_string.restype = ctypes.c_char_p
    lib.mesa_version.argtypes = []
    lib.mesa_version.restype = ci
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().mesa_status_string(int(status)).decode()


def version() -> int:
    return load().mesa_version()


def forward_workspace_bytes(batch, heads, seq_len, d_k, d_v, chunk) -> int:
    return load().mesa_forward_workspace_bytes(batch, heads, seq_len, d_k, d_v, chunk)


def bf16_path_available(d_k, d_v, chunk, seq_len=2048) -> bool:
    """Whether MESA_PREC_BF16 (the matrix-core path) supports this shape: a
    zero-batch solve call validates the arguments and launches nothing."""
    st = load().mesa_forward_solve(None, None, None, None, None, None, 0, 1, seq_len, d_k, d_v,
                                   MESA_DTYPE_BF16, 1, chunk, MESA_PREC_BF16, None, None, None, 0,
                                   None)
    return st == MESA_OK


# ---------------------------------------------------------------- torch glue
def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return MESA_DTYPE_F32
    if t.dtype == torch.bfloat16:
        return MESA_DTYPE_BF16
    raise TypeError("q, k, v must be float32 or bfloat16, got %s" % t.dtype)


def _check(t, name, shape, dtype=None, device=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def forward(q, k, v, gamma, beta, lam, n_cg, chunk=64, precision=MESA_PREC_AUTO, want_qstar=False,
            want_states=False, out=None, workspace=None, eps=None, want_steps=False):
    """Mesa forward over q, k [B,H,T,d_k], v [B,H,T,d_v] (fp32 or bf16, same dtype),
    gamma, beta [B,H,T] fp32, lam [H,d_k] fp32.  Returns out [B,H,T,d_v] fp32, or a
    dict with "out" and, if asked, "qstar" [B,H,T,d_k], "H" [B,H,d_k,d_k], "G" [B,H,d_v,d_k],
    "steps" [B,H,T] int32 (CG iterations per token).
    eps: CG relative tolerance (Alg. 1's |r_k| <= eps |r_0|; n_cg is then the limit),
    through mesa_forward_tol; None or 0 with want_steps False is the fixed-step solve.
    Runs on torch's current stream of q's device."""
    torch = _torch()
    lib = load()
    B, H, T, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    _check(q, "q", (B, H, T, dk), device=dev)
    _check(k, "k", (B, H, T, dk), q.dtype, dev)
    _check(v, "v", (B, H, T, dv), q.dtype, dev)
    _check(gamma, "gamma", (B, H, T), torch.float32, dev)
    _check(beta, "beta", (B, H, T), torch.float32, dev)
    _check(lam, "lam", (H, dk), torch.float32, dev)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
    _check(out, "out", (B, H, T, dv), torch.float32, dev)
    need = lib.mesa_forward_workspace_bytes(B, H, T, dk, dv, chunk)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    qstar = torch.empty((B, H, T, dk), dtype=torch.float32, device=dev) if want_qstar else None
    if eps is not None or want_steps:
        if want_states:
            raise ValueError("mesa_forward_tol returns no final states")
        steps = torch.empty((B, H, T), dtype=torch.int32, device=dev) if want_steps else None
        st = lib.mesa_forward_tol(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam), B, H,
                                  T, dk, dv, code, int(n_cg), float(eps or 0.0), int(chunk),
                                  int(precision), _ptr(out), _ptr(qstar), _ptr(steps), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(dev))
        if st != MESA_OK:
            raise MesaError(st, "mesa_forward_tol")
        res = {"out": out}
        if want_qstar:
            res["qstar"] = qstar
        if want_steps:
            res["steps"] = steps
        return res if (want_qstar or want_steps) else out
    fH = torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev) if want_states else None
    fG = torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev) if want_states else None
    st = lib.mesa_forward_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam), B, H, T,
                             dk, dv, code, int(n_cg), int(chunk), int(precision), _ptr(out),
                             _ptr(qstar), _ptr(fH), _ptr(fG), _ptr(workspace),
                             workspace.numel() * workspace.element_size(), _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_forward_ex")
    if not (want_qstar or want_states):
        return out
    res = {"out": out}
    if want_qstar:
        res["qstar"] = qstar
    if want_states:
        res["H"] = fH
        res["G"] = fG
    return res


def frontend(qp, kp, vp, conv_q, conv_k, conv_v, a_gamma, a_beta, theta, gamma_cap=0.9975, l2_eps=1e-6):
    """mesa_frontend: the layer's inputs from the projections (App. E, App. G.5).
    qp, kp [B,T,H,d_k], vp [B,T,H,d_v] (fp32 or bf16, one dtype); conv_q, conv_k
    [H*d_k,4], conv_v [H*d_v,4] or None; a_gamma, a_beta [B,T,H]; theta [H,d_k] (fp32).
    Returns a dict: q, k [B,H,T,d_k], v [B,H,T,d_v] (the projections' dtype), gamma,
    beta [B,H,T], lam [H,d_k] (fp32)."""
    torch = _torch()
    lib = load()
    B, T, H, dk = qp.shape
    dv = vp.shape[-1]
    dev = qp.device
    f32 = torch.float32
    _check(qp, "qp", (B, T, H, dk), device=dev)
    _check(kp, "kp", (B, T, H, dk), qp.dtype, dev)
    _check(vp, "vp", (B, T, H, dv), qp.dtype, dev)
    _check(conv_q, "conv_q", (H * dk, 4), f32, dev)
    _check(conv_k, "conv_k", (H * dk, 4), f32, dev)
    if conv_v is not None:
        _check(conv_v, "conv_v", (H * dv, 4), f32, dev)
    _check(a_gamma, "a_gamma", (B, T, H), f32, dev)
    _check(a_beta, "a_beta", (B, T, H), f32, dev)
    _check(theta, "theta", (H, dk), f32, dev)
    res = {"q": torch.empty((B, H, T, dk), dtype=qp.dtype, device=dev),
           "k": torch.empty((B, H, T, dk), dtype=qp.dtype, device=dev),
           "v": torch.empty((B, H, T, dv), dtype=qp.dtype, device=dev),
           "gamma": torch.empty((B, H, T), dtype=f32, device=dev),
           "beta": torch.empty((B, H, T), dtype=f32, device=dev),
           "lam": torch.empty((H, dk), dtype=f32, device=dev)}
    st = lib.mesa_frontend(_ptr(qp), _ptr(kp), _ptr(vp), _ptr(conv_q), _ptr(conv_k), _ptr(conv_v), _ptr(a_gamma),
                           _ptr(a_beta), _ptr(theta), float(gamma_cap), float(l2_eps), B, H, T, dk, dv,
                           _dtype_code(qp), _ptr(res["q"]), _ptr(res["k"]), _ptr(res["v"]), _ptr(res["gamma"]),
                           _ptr(res["beta"]), _ptr(res["lam"]), _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_frontend")
    return res


def output_norm(o, weight, eps=1e-6, out_dtype=None):
    """mesa_output_norm: per-head RMSNorm of the layer output o [B,H,T,d_v] fp32 with
    weight [H,d_v], into [B,T,H,d_v] of out_dtype (torch.bfloat16 by default)."""
    torch = _torch()
    lib = load()
    B, H, T, dv = o.shape
    dev = o.device
    _check(o, "o", (B, H, T, dv), torch.float32, dev)
    _check(weight, "weight", (H, dv), torch.float32, dev)
    out_dtype = torch.bfloat16 if out_dtype is None else out_dtype
    y = torch.empty((B, T, H, dv), dtype=out_dtype, device=dev)
    st = lib.mesa_output_norm(_ptr(o), _ptr(weight), float(eps), B, H, T, dv, _dtype_code(y), _ptr(y),
                              _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_output_norm")
    return y


def forward_noalloc(q, k, v, gamma, beta, lam, n_cg, chunk=64, out=None):
    """mesa_forward_noalloc: the forward with the chunk states in the library's own
    fixed device buffer (no workspace; MesaError with MESA_ERR_WORKSPACE when the
    shape needs more than MESA_NOALLOC_SCRATCH_BYTES).  Same inputs as forward();
    returns out [B,H,T,d_v] fp32 (allocated here unless given)."""
    torch = _torch()
    lib = load()
    B, H, T, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    _check(q, "q", (B, H, T, dk), device=dev)
    _check(k, "k", (B, H, T, dk), q.dtype, dev)
    _check(v, "v", (B, H, T, dv), q.dtype, dev)
    _check(gamma, "gamma", (B, H, T), torch.float32, dev)
    _check(beta, "beta", (B, H, T), torch.float32, dev)
    _check(lam, "lam", (H, dk), torch.float32, dev)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
    _check(out, "out", (B, H, T, dv), torch.float32, dev)
    st = lib.mesa_forward_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam), B, H, T,
                                  dk, dv, _dtype_code(q), int(n_cg), int(chunk), _ptr(out), _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_forward_noalloc")
    return out


class ForwardPlan:
    """Pre-checked arguments of one forward shape, for repeated calls of the two
    launches (mesa_forward_states, then mesa_forward_solve) on torch's current
    stream.  Holds the output and workspace tensors; used by the benchmark to
    time each launch with events on the launch stream."""

    def __init__(self, q, k, v, gamma, beta, lam, n_cg, chunk=64, precision=MESA_PREC_AUTO):
        torch = _torch()
        self.lib = load()
        B, H, T, dk = q.shape
        dv = v.shape[-1]
        dev = q.device
        _check(q, "q", (B, H, T, dk), device=dev)
        _check(k, "k", (B, H, T, dk), q.dtype, dev)
        _check(v, "v", (B, H, T, dv), q.dtype, dev)
        _check(gamma, "gamma", (B, H, T), torch.float32, dev)
        _check(beta, "beta", (B, H, T), torch.float32, dev)
        _check(lam, "lam", (H, dk), torch.float32, dev)
        self.tensors = (q, k, v, gamma, beta, lam)
        self.dims = (B, H, T, dk, dv)
        self.code = _dtype_code(q)
        self.n_cg, self.chunk, self.precision = int(n_cg), int(chunk), int(precision)
        self.device = dev
        self.out = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
        self.ws_bytes = self.lib.mesa_forward_workspace_bytes(B, H, T, dk, dv, chunk)
        self.workspace = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)

    def states(self):
        q, k, v, gamma, beta, lam = self.tensors
        B, H, T, dk, dv = self.dims
        st = self.lib.mesa_forward_states(_ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), B, H, T, dk, dv,
                                          self.code, self.chunk, self.precision, None, None,
                                          _ptr(self.workspace), self.ws_bytes, _stream(self.device))
        if st != MESA_OK:
            raise MesaError(st, "mesa_forward_states")

    def solve(self):
        q, k, v, gamma, beta, lam = self.tensors
        B, H, T, dk, dv = self.dims
        st = self.lib.mesa_forward_solve(_ptr(q), _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam),
                                         B, H, T, dk, dv, self.code, self.n_cg, self.chunk,
                                         self.precision, _ptr(self.out), None, _ptr(self.workspace),
                                         self.ws_bytes, _stream(self.device))
        if st != MESA_OK:
            raise MesaError(st, "mesa_forward_solve")
        return self.out

    def __call__(self):
        self.states()
        return self.solve()


def backward_workspace_bytes(batch, heads, seq_len, d_k, d_v) -> int:
    return load().mesa_backward_workspace_bytes(batch, heads, seq_len, d_k, d_v)


def backward(k, v, gamma, beta, lam, qstar, dout, n_cg, precision=MESA_PREC_AUTO, workspace=None):
    """Gradients of the layer given dout = dL/do [B,H,T,d_v] fp32 and the forward's
    q* [B,H,T,d_k] fp32 (mesa_backward).  k, v [B,H,T,d] fp32 or bf16; gamma, beta
    [B,H,T]; lam [H,d_k].  precision selects the solve for e* (MESA_PREC_F32, or
    MESA_PREC_BF16 on the matrix cores; AUTO: BF16 for bf16 inputs).  Returns a dict
    of fp32 tensors: "dq", "dk" [B,H,T,d_k], "dv" [B,H,T,d_v], "dgamma", "dbeta"
    [B,H,T], "dlam" [H,d_k].
    Runs on torch's current stream of k's device."""
    torch = _torch()
    lib = load()
    B, H, T, dk = k.shape
    dv = v.shape[-1]
    dev = k.device
    _check(k, "k", (B, H, T, dk), device=dev)
    _check(v, "v", (B, H, T, dv), k.dtype, dev)
    _check(gamma, "gamma", (B, H, T), torch.float32, dev)
    _check(beta, "beta", (B, H, T), torch.float32, dev)
    _check(lam, "lam", (H, dk), torch.float32, dev)
    _check(qstar, "qstar", (B, H, T, dk), torch.float32, dev)
    _check(dout, "dout", (B, H, T, dv), torch.float32, dev)
    need = lib.mesa_backward_workspace_bytes(B, H, T, dk, dv)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    res = {"dq": torch.empty((B, H, T, dk), **f32), "dk": torch.empty((B, H, T, dk), **f32),
           "dv": torch.empty((B, H, T, dv), **f32), "dgamma": torch.empty((B, H, T), **f32),
           "dbeta": torch.empty((B, H, T), **f32), "dlam": torch.empty((H, dk), **f32)}
    st = lib.mesa_backward(_ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), _ptr(lam), B, H, T, dk, dv,
                           _dtype_code(k), int(n_cg), int(precision), _ptr(qstar), _ptr(dout), _ptr(res["dq"]),
                           _ptr(res["dk"]), _ptr(res["dv"]), _ptr(res["dgamma"]), _ptr(res["dbeta"]),
                           _ptr(res["dlam"]), _ptr(workspace), workspace.numel() * workspace.element_size(),
                           _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_backward")
    return res


def prefill_states(k, v, gamma, beta, chunk=64, workspace=None):
    """States after the last token only (mesa_forward_ex with out = NULL):
    returns (H [B,H,d_k,d_k], G [B,H,d_v,d_k]) fp32, the input of decode_step.
    workspace: optional device tensor of at least mesa_forward_workspace_bytes,
    scratch that lets the scan of few long sequences run in segments."""
    torch = _torch()
    lib = load()
    B, H, T, dk = k.shape
    dv = v.shape[-1]
    dev = k.device
    _check(k, "k", (B, H, T, dk), device=dev)
    _check(v, "v", (B, H, T, dv), k.dtype, dev)
    _check(gamma, "gamma", (B, H, T), torch.float32, dev)
    _check(beta, "beta", (B, H, T), torch.float32, dev)
    code = _dtype_code(k)
    fH = torch.empty((B, H, dk, dk), dtype=torch.float32, device=dev)
    fG = torch.empty((B, H, dv, dk), dtype=torch.float32, device=dev)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _check(workspace, "workspace", tuple(workspace.shape), device=dev)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    st = lib.mesa_forward_ex(None, _ptr(k), _ptr(v), _ptr(gamma), _ptr(beta), None, B, H, T, dk, dv,
                             code, 0, int(chunk), MESA_PREC_AUTO, None, None, _ptr(fH), _ptr(fG),
                             ws_ptr, ws_bytes, _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_forward_ex(states only)")
    return fH, fG


def pack_state(state_H):
    """Full symmetric decode state H [N,H,d_k,d_k] -> packed cyclic diagonals
    [N,H,d_k/2+1,d_k] (mesa_pack_state)."""
    torch = _torch()
    lib = load()
    N, H, dk, _ = state_H.shape
    _check(state_H, "state_H", (N, H, dk, dk), torch.float32, state_H.device)
    hp = torch.empty((N, H, dk // 2 + 1, dk), dtype=torch.float32, device=state_H.device)
    st = lib.mesa_pack_state(_ptr(state_H), _ptr(hp), N, H, dk, _stream(state_H.device))
    if st != MESA_OK:
        raise MesaError(st, "mesa_pack_state")
    return hp


def unpack_state(state_HP):
    """Packed [N,H,d_k/2+1,d_k] -> full symmetric H [N,H,d_k,d_k] (mesa_unpack_state)."""
    torch = _torch()
    lib = load()
    N, H, _, dk = state_HP.shape
    _check(state_HP, "state_HP", (N, H, dk // 2 + 1, dk), torch.float32, state_HP.device)
    h = torch.empty((N, H, dk, dk), dtype=torch.float32, device=state_HP.device)
    st = lib.mesa_unpack_state(_ptr(state_HP), _ptr(h), N, H, dk, _stream(state_HP.device))
    if st != MESA_OK:
        raise MesaError(st, "mesa_unpack_state")
    return h


def decode_step(state_H, state_G, q, k, v, gamma, beta, lam, n_cg, out=None, eps=None, steps_out=None,
                packed=False):
    """One recurrent step, in place on state_H [N,H,d_k,d_k] (or, with packed, the
    cyclic-diagonal form [N,H,d_k/2+1,d_k] of pack_state) and state_G [N,H,d_v,d_k].
    q, k [N,H,d_k], v [N,H,d_v] fp32 or bf16; gamma, beta [N,H]; lam [H,d_k].
    eps / steps_out (int32 [N,H]): CG relative tolerance and iteration counts, through
    mesa_decode_step_tol (or mesa_decode_step_packed).  Returns out [N,H,d_v] fp32."""
    torch = _torch()
    lib = load()
    N, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    _check(state_H, "state_H", (N, H, dk // 2 + 1 if packed else dk, dk), torch.float32, dev)
    _check(state_G, "state_G", (N, H, dv, dk), torch.float32, dev)
    _check(q, "q", (N, H, dk), device=dev)
    _check(k, "k", (N, H, dk), q.dtype, dev)
    _check(v, "v", (N, H, dv), q.dtype, dev)
    _check(gamma, "gamma", (N, H), torch.float32, dev)
    _check(beta, "beta", (N, H), torch.float32, dev)
    _check(lam, "lam", (H, dk), torch.float32, dev)
    if out is None:
        out = torch.empty((N, H, dv), dtype=torch.float32, device=dev)
    _check(out, "out", (N, H, dv), torch.float32, dev)
    if packed:
        if steps_out is not None:
            _check(steps_out, "steps_out", (N, H), torch.int32, dev)
        st = lib.mesa_decode_step_packed(_ptr(state_H), _ptr(state_G), _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(gamma), _ptr(beta), _ptr(lam), N, H, dk, dv, _dtype_code(q),
                                         int(n_cg), float(eps or 0.0), _ptr(out), _ptr(steps_out),
                                         _stream(dev))
        if st != MESA_OK:
            raise MesaError(st, "mesa_decode_step_packed")
        return out
    if eps is not None or steps_out is not None:
        if steps_out is not None:
            _check(steps_out, "steps_out", (N, H), torch.int32, dev)
        st = lib.mesa_decode_step_tol(_ptr(state_H), _ptr(state_G), _ptr(q), _ptr(k), _ptr(v),
                                      _ptr(gamma), _ptr(beta), _ptr(lam), N, H, dk, dv, _dtype_code(q),
                                      int(n_cg), float(eps or 0.0), _ptr(out), _ptr(steps_out),
                                      _stream(dev))
        if st != MESA_OK:
            raise MesaError(st, "mesa_decode_step_tol")
        return out
    st = lib.mesa_decode_step(_ptr(state_H), _ptr(state_G), _ptr(q), _ptr(k), _ptr(v), _ptr(gamma),
                              _ptr(beta), _ptr(lam), N, H, dk, dv, _dtype_code(q), int(n_cg),
                              _ptr(out), _stream(dev))
    if st != MESA_OK:
        raise MesaError(st, "mesa_decode_step")
    return out
