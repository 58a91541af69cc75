"""Helpers shared by the GPU tests: device placement of generator output and
the parity metric (relative L2 over the compared outputs)."""
import numpy as np

# Tolerances on relative L2 of the outputs against the oracle's same-step CG:
# fp32 inputs (fp32 products) and bf16 inputs (fp32 state and CG vectors).
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def rel_l2(got, want):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    return float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))


def to_device(x, dtype, device="cuda:0"):
    """Generator output (fp32 numpy, bf16-exact for bf16 workloads) -> torch tensors."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = {}
    for name, a in x.items():
        t = torch.from_numpy(np.ascontiguousarray(a)).to(device)
        out[name] = t.to(tdt) if name in ("q", "k", "v") else t
    return out


def subset(x, b_idx, h_idx):
    """Rows of a forward input dict for the chosen (batch, head) pairs, as [n, 1, ...]
    (lambda rows follow the heads).  Keeps the oracle's work bounded."""
    sel = {}
    for name in ("q", "k", "v", "gamma", "beta"):
        sel[name] = np.stack([x[name][b, h] for b, h in zip(b_idx, h_idx)])[:, None]
    return sel, [x["lam"][h][None] for h in h_idx]
