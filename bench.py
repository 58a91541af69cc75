#!/usr/bin/env python3
"""Benchmark of the Mesa layer forward (and decode) through libmesa on one MI355X.

A step is one forward pass of the layer over one batch of the 1B-shaped
workload (B=8, heads=16, T=2048, d_k=d_v=128, chunk 64, 15 CG steps, bf16
q/k/v): the chunk-state scan launch, then the chunked CG + read-out launch.
Inputs are resident in HBM before timing starts.  Each launch is bracketed by
HIP events on the stream it runs on; the CG launch is the dominant kernel and
its algorithmic flops per launch divided by its mean event time give the
roofline entry.

The timed steps (the metric) use the single-pass matrix-core products
(MESA_PREC_BF16: chunk states stored in bf16, CG operands rounded to bf16, fp32
accumulation and fp32 CG vectors), the fastest mode within the bf16-input
tolerance on the workloads.  The same workload is also timed with the
fp32-accurate split-operand products (MESA_PREC_BF16X3, the library's default
for bf16 inputs; App. G.5 keeps the solver's products in fp32) and with fp32
products (MESA_PREC_F32), each with its own roofline entry; and the
long-context workload (B=1, heads=16, T=16384, 20 CG steps) in both
matrix-core modes.  Decode (256 sequences x 16 heads, d=128, 15 CG steps,
1024 consecutive steps) is timed after the forward steps.

Context entries run the same forward and decode with Alg. 1's relative
stopping test (eps = 1e-4, at most 30 iterations, the paper's dynamic
test-time compute setting), time the backward pass (mesa_backward, App. D) and
the layer's front and back end (App. E) at the same shapes.
The CPU baseline is the fp64 oracle (the sequential recurrence with
fixed-step CG) on the same workload, run on the host's cores.

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Mesa-layer forward tokens/s on 1 MI355X (+% MFMA peak); decode tokens/s"
PEAKS = {  # MI355X published dense peaks
    "mfma_bf16_tflops": 2500.0,
    "mfma_fp32_tflops": 157.3,
    "hbm_gbps": 8000.0,
}

# What each precision mode computes, as printed in the JSON line.
PREC_TEXT = {
    2: "bf16 q/k/v; chunk states stored as bf16 matrix-core fragments; CG and read-out products on "
       "single bf16 operands (the fp32 state, direction, intra-chunk weights and Lambda rounded to bf16) "
       "with fp32 accumulation; CG vectors, scalars and reductions fp32 (MESA_PREC_BF16)",
    3: "bf16 q/k/v; chunk states fp32-accurate (H_c fp32, G_c as bf16 high + low parts); CG and read-out "
       "products on split operands x = hi + lo (hi*hi + hi*lo + lo*hi, three bf16 matrix-core passes, fp32 "
       "accumulation); Lambda p, CG vectors, scalars and reductions fp32 (MESA_PREC_BF16X3)",
    1: "bf16 q/k/v; fp32 chunk states; fp32 products on the fp32 matrix cores (MESA_PREC_F32)",
}
# The CG kernel each mode runs, and the sources its traffic record is tied to.
CG_KERNEL = {2: "chunk_cg_bf16", 3: "chunk_cg_x3", 1: "chunk_cg_f32"}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def cg_kernel_flops(B, H, T, dk, dv, C, n_cg):
    """Algorithmic flops of one launch of the chunked CG + read-out kernel.
    Per token-head: (n_cg + 1) products (H_t + Lambda) p, each 2 d_k^2 for the
    state term plus 2 (C + 1) d_k for the causal intra-chunk K^T(Z (K p)) term
    (causal halves only), and the read-out 2 d_v d_k + (C + 1)(d_k + d_v).
    The same count serves every precision mode: split operands issue more
    matrix-core work for the same products."""
    per_th = (n_cg + 1) * (2 * dk * dk + 2 * (C + 1) * dk) + 2 * dv * dk + (C + 1) * (dk + dv)
    return B * H * T * per_th


def state_kernel_bytes(B, H, T, dk, dv, C, in_bytes, state_bytes):
    """Algorithmic HBM bytes of the chunk-state launch: the states entering every
    chunk written once (state_bytes per element: 2 for the bf16 fragments of the
    single-pass path, 4 for fp32 or split-operand states), plus k and v read once
    (gates ignored)."""
    nc = (T + C - 1) // C
    return B * H * nc * dk * (dk + dv) * state_bytes + B * H * T * (dk + dv) * in_bytes


def source_hash(kernel):
    """sha256 over the sources a CG kernel is built from and the build script (its flags)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2506_05233_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.startswith(kernel) or name in ("mesa_device.hpp", "mesa_mfma.hpp", "mesa_kernels.hpp"):
            h.update(open(os.path.join(csrc, name), "rb").read())
    h.update(open(os.path.join(ROOT, "paper_2506_05233_amd", "build.py"), "rb").read())
    return h.hexdigest()


def traffic_entry(kernel):
    """HBM bytes per launch of a CG kernel from its committed rocprofv3 --pmc record,
    or None when absent or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "%s_layer1b_traffic.json" % kernel)
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != source_hash(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def device_inputs(torch, x):
    dev = torch.device("cuda:0")
    d = {}
    for name, a in x.items():
        t = torch.from_numpy(a).to(dev)
        d[name] = t.to(torch.bfloat16) if name in ("q", "k", "v") else t
    return d


def time_forward(torch, L, w, d, prec, steps, warmup):
    """Times `steps` forward steps (scan launch + solve launch) after `warmup`
    untimed ones: wall time between two synchronisations and the mean HIP-event
    time of each launch (events on the launch stream)."""
    plan = L.ForwardPlan(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], w.n_cg, w.chunk, prec)
    for _ in range(warmup):
        plan()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record()
        plan.states()
        ev[i][1].record()
        plan.solve()
        ev[i][2].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    state_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / steps
    cg_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / steps
    if not bool(torch.isfinite(plan.out).all()):
        raise RuntimeError("non-finite output")
    return {"plan": plan, "wall": wall, "state_ms": state_ms, "cg_ms": cg_ms}


def roofline(L, w, prec, cg_ms):
    """Roofline entry of the CG launch: algorithmic flops / mean launch time against
    the peak of the matrix cores the mode runs on."""
    flops = cg_kernel_flops(w.batch, w.heads, w.seq_len, w.d_k, w.d_v, w.chunk, w.n_cg)
    achieved = flops / (cg_ms / 1e3) / 1e12
    peak = PEAKS["mfma_fp32_tflops"] if prec == L.MESA_PREC_F32 else PEAKS["mfma_bf16_tflops"]
    kernel = CG_KERNEL[prec]
    return {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
            "traffic": traffic_entry(kernel), "kernel": kernel + " (chunked CG + read-out)",
            "ms_per_launch": cg_ms, "flops_per_launch": flops}


def mode_entry(L, w, prec, t):
    B, H, T, dk, dv = w.batch, w.heads, w.seq_len, w.d_k, w.d_v
    sb = 2 if prec == L.MESA_PREC_BF16 else 4
    st_bytes = state_kernel_bytes(B, H, T, dk, dv, w.chunk, 2, sb)
    return {"inputs": PREC_TEXT[prec], "tokens_per_s": B * T / (t["wall"] / t["steps"]),
            "ms_per_step": t["wall"] / t["steps"] * 1e3,
            "kernels_ms": {"chunk_state": t["state_ms"], "chunk_cg": t["cg_ms"]},
            "state_kernel_hbm": {"GBps": st_bytes / (t["state_ms"] / 1e3) / 1e9,
                                 "frac": st_bytes / (t["state_ms"] / 1e3) / 1e9 / PEAKS["hbm_gbps"]},
            "roofline": roofline(L, w, prec, t["cg_ms"])}


def run_forward(args, torch, L, W):
    w = W.LAYER_1B_BF16
    log("generating %s inputs" % w.name)
    x = W.workload_inputs(w)
    d = device_inputs(torch, x)
    log("warmup %d, timing %d steps (precision %d)" % (args.warmup, args.steps, args.precision))
    t = time_forward(torch, L, w, d, args.precision, args.steps, args.warmup)
    t["steps"] = args.steps
    return {"w": w, "x": x, "d": d, "plan": t["plan"], "t": t}


def run_other_modes(args, torch, L, fw):
    """The headline workload in the other precision modes (5 timed steps each)."""
    w, d = fw["w"], fw["d"]
    out = {}
    for prec, key in ((L.MESA_PREC_BF16X3, "split_operands_bf16x3"), (L.MESA_PREC_F32, "fp32_products")):
        if prec == args.precision:
            continue
        log("forward in precision mode %d" % prec)
        t = time_forward(torch, L, w, d, prec, 5, 2)
        t["steps"] = 5
        out[key] = mode_entry(L, w, prec, t)
        del t["plan"]
    return out


def run_long_context(args, torch, L, W):
    """The long-context workload (B=1, heads=16, T=16384, 20 CG steps) in both
    matrix-core modes: tokens/s and per-launch times."""
    w = W.LONG_BF16
    log("generating %s inputs" % w.name)
    d = device_inputs(torch, W.workload_inputs(w))
    res = {"workload": w.name, "batch": w.batch, "heads": w.heads, "seq_len": w.seq_len, "n_cg": w.n_cg}
    for prec, key in ((L.MESA_PREC_BF16, "single_pass_bf16"), (L.MESA_PREC_BF16X3, "split_operands_bf16x3")):
        log("long context, precision mode %d" % prec)
        t = time_forward(torch, L, w, d, prec, 5, 2)
        t["steps"] = 5
        e = mode_entry(L, w, prec, t)
        e["cg_fraction_of_step"] = t["cg_ms"] / (t["state_ms"] + t["cg_ms"])
        del t["plan"]
        res[key] = e
    return res


def run_layer_ends(args, torch, L, fw):
    """The layer's front end (mesa_frontend: projections -> q, k, v, gates, Lambda) and back
    end (mesa_output_norm: per-head RMSNorm) at the headline workload's shapes, bf16
    projections with a value filter, bf16 normed output.  Both are HBM-bound; the entry
    gives time per call and algorithmic bytes over time against the 8 TB/s peak."""
    w = fw["w"]
    B, H, T, dk, dv = w.batch, w.heads, w.seq_len, w.d_k, w.d_v
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(11)
    bf = torch.bfloat16
    qp = torch.randn((B, T, H, dk), generator=g, device=dev).to(bf)
    kp = torch.randn((B, T, H, dk), generator=g, device=dev).to(bf)
    vp = torch.randn((B, T, H, dv), generator=g, device=dev).to(bf)
    cq, ck = (0.5 * torch.randn((H * dk, 4), generator=g, device=dev) for _ in range(2))
    cv = 0.5 * torch.randn((H * dv, 4), generator=g, device=dev)
    ag = 4.0 + torch.randn((B, T, H), generator=g, device=dev)
    ab = torch.randn((B, T, H), generator=g, device=dev)
    th = torch.randn((H, dk), generator=g, device=dev)
    o = fw["plan"].out
    wt = torch.ones((H, dv), device=dev)

    def timed(fn, reps=10):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    ms_f = timed(lambda: L.frontend(qp, kp, vp, cq, ck, cv, ag, ab, th))
    ms_n = timed(lambda: L.output_norm(o, wt, 1e-6))
    th_ = B * H * T
    bytes_f = th_ * (2 * (2 * dk + dv) * 2 + 4 * 4) + 4 * (H * (2 * dk + dv) * 4 + 2 * H * dk)
    bytes_n = th_ * dv * (4 + 2)
    gbps = lambda b, ms: b / (ms / 1e3) / 1e9
    return {"frontend": {"ms_per_call": ms_f, "tokens_per_s": B * T / (ms_f / 1e3), "bytes": bytes_f,
                         "hbm_GBps": gbps(bytes_f, ms_f), "hbm_frac": gbps(bytes_f, ms_f) / PEAKS["hbm_gbps"],
                         "what": "window-4 convolution + SiLU (q, k, v), unit norm (q, k), gates with the cap, "
                                 "Lambda; bf16 projections [B,T,H,d] -> bf16 [B,H,T,d]"},
            "output_norm": {"ms_per_call": ms_n, "tokens_per_s": B * T / (ms_n / 1e3), "bytes": bytes_n,
                            "hbm_GBps": gbps(bytes_n, ms_n), "hbm_frac": gbps(bytes_n, ms_n) / PEAKS["hbm_gbps"],
                            "what": "per-head RMSNorm, fp32 [B,H,T,d_v] -> bf16 [B,T,H,d_v]"}}


def run_forward_dynamic(args, torch, L, fw):
    """The same forward with Alg. 1's relative stopping test (eps, at most
    args.dyn_max_cg iterations): time per call and the mean iterations per token."""
    w, d, plan = fw["w"], fw["d"], fw["plan"]
    steps = None
    def call():
        return L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], args.dyn_max_cg,
                         w.chunk, precision=args.precision, out=plan.out, workspace=plan.workspace,
                         eps=args.eps, want_steps=True)
    for _ in range(2):
        steps = call()["steps"]
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    reps = 5
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"eps": args.eps, "max_cg": args.dyn_max_cg, "tokens_per_s": w.batch * w.seq_len / (ms / 1e3),
            "ms_per_call": ms, "mean_cg_steps": float(steps.float().mean())}


def run_backward(args, torch, L, fw):
    """mesa_backward on the forward workload: gradients of q, k, v, gamma, beta and
    Lambda given a seeded dL/do and the q* of the forward (computed before timing)."""
    w, d = fw["w"], fw["d"]
    # the backward's solve runs on fp32 products or on the single-pass matrix cores
    prec = L.MESA_PREC_F32 if args.precision == L.MESA_PREC_F32 else L.MESA_PREC_BF16
    res = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], w.n_cg, w.chunk,
                    precision=args.precision, want_qstar=True)
    qstar = res["qstar"]
    gen = torch.Generator(device="cuda").manual_seed(7)
    dout = torch.randn(d["v"].shape, dtype=torch.float32, device="cuda", generator=gen)
    ws = torch.empty(L.backward_workspace_bytes(w.batch, w.heads, w.seq_len, w.d_k, w.d_v),
                     dtype=torch.uint8, device="cuda")
    def call():
        return L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], qstar, dout, w.n_cg,
                          precision=prec, workspace=ws)
    for _ in range(2):
        g = call()
    torch.cuda.synchronize()
    if not all(bool(torch.isfinite(t).all()) for t in g.values()):
        raise RuntimeError("non-finite gradient")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    reps = 5
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del ws
    return {"tokens_per_s": w.batch * w.seq_len / (ms / 1e3), "ms_per_call": ms, "n_cg": w.n_cg,
            "solve": "matrix cores (single-pass bf16 operands)" if prec == L.MESA_PREC_BF16 else "fp32 products",
            "launches": "fp32 and bf16 chunk states, rhs G^T e, CG solve for e*, reverse adjoint scan, "
                        "per-chunk gradients, Lambda sum"}


def run_decode(args, torch, L, W):
    w = W.DECODE_BF16
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(w.seed)
    N, H, d = w.seqs, w.heads, w.d_k
    log("decode: prefilling %d x %d states over %d tokens on the GPU" % (N, H, w.prefill))

    def unit(shape):
        t = torch.randn(shape, generator=g, device=dev)
        return t / t.norm(dim=-1, keepdim=True)

    # prefill in slices of sequences to bound memory
    sH = torch.empty((N, H, d, d), dtype=torch.float32, device=dev)
    sG = torch.empty((N, H, d, d), dtype=torch.float32, device=dev)
    step = 64
    for s0 in range(0, N, step):
        n = min(step, N - s0)
        k = unit((n, H, w.prefill, d)).to(torch.bfloat16)
        v = torch.randn((n, H, w.prefill, d), generator=g, device=dev).to(torch.bfloat16)
        gam = torch.sigmoid(w.gamma_mu + torch.randn((n, H, w.prefill), generator=g, device=dev))
        bet = torch.sigmoid(torch.randn((n, H, w.prefill), generator=g, device=dev))
        fH, fG = L.prefill_states(k, v, gam, bet)
        sH[s0:s0 + n].copy_(fH)
        sG[s0:s0 + n].copy_(fG)
        del k, v, gam, bet, fH, fG
    lam = 0.25 + 0.75 * torch.rand((H, d), generator=g, device=dev)
    S = args.decode_steps
    q = unit((S, N, H, d)).to(torch.bfloat16)
    k = unit((S, N, H, d)).to(torch.bfloat16)
    v = torch.randn((S, N, H, d), generator=g, device=dev).to(torch.bfloat16)
    gam = torch.sigmoid(w.gamma_mu + torch.randn((S, N, H), generator=g, device=dev))
    bet = torch.sigmoid(torch.randn((S, N, H), generator=g, device=dev))
    out = torch.empty((N, H, d), dtype=torch.float32, device=dev)
    for i in range(min(3, S)):  # warm-up on a copy of the state
        L.decode_step(sH.clone(), sG.clone(), q[i], k[i], v[i], gam[i], bet[i], lam, w.n_cg, out=out)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    log("decode: timing %d steps" % S)
    e0.record()
    for i in range(S):
        L.decode_step(sH, sG, q[i], k[i], v[i], gam[i], bet[i], lam, w.n_cg, out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    if not bool(torch.isfinite(out).all()):
        raise RuntimeError("non-finite decode output")
    bytes_per_step = N * H * (2 * d * d * 4 * 2 + 3 * d * 2 + d * 4)
    # the same steps on the packed symmetric state (cyclic diagonals of H)
    sHP = L.pack_state(sH)
    sG2 = sG.clone()
    for i in range(min(3, S)):
        L.decode_step(sHP.clone(), sG2.clone(), q[i], k[i], v[i], gam[i], bet[i], lam, w.n_cg, out=out, packed=True)
    torch.cuda.synchronize()
    log("decode: timing %d steps on the packed state" % S)
    e0.record()
    for i in range(S):
        L.decode_step(sHP, sG2, q[i], k[i], v[i], gam[i], bet[i], lam, w.n_cg, out=out, packed=True)
    e1.record()
    torch.cuda.synchronize()
    msp = e0.elapsed_time(e1)
    bytes_packed = N * H * (2 * (d // 2 + 1) * d * 4 + 2 * d * d * 4 + 3 * d * 2 + d * 4)
    packed = {"tokens_per_s": N * S / (msp / 1e3), "ms_per_step": msp / S,
              "hbm_GBps": bytes_packed * S / (msp / 1e3) / 1e9,
              "hbm_frac": bytes_packed * S / (msp / 1e3) / 1e9 / PEAKS["hbm_gbps"],
              "state": "H as its d/2+1 cyclic diagonals (mesa_decode_step_packed)"}
    del sHP, sG2
    dyn = None
    if args.eps > 0:  # dynamic stopping on the continuing states
        S2 = min(S, 64)
        st = torch.zeros((N, H), dtype=torch.int32, device=dev)
        tot = torch.zeros((N, H), dtype=torch.int64, device=dev)
        log("decode: timing %d steps with eps %g" % (S2, args.eps))
        torch.cuda.synchronize()
        e0.record()
        for i in range(S2):
            L.decode_step(sH, sG, q[i], k[i], v[i], gam[i], bet[i], lam, args.dyn_max_cg, out=out,
                          eps=args.eps, steps_out=st)
            tot += st
        e1.record()
        torch.cuda.synchronize()
        ms2 = e0.elapsed_time(e1)
        dyn = {"eps": args.eps, "max_cg": args.dyn_max_cg, "steps": S2,
               "tokens_per_s": N * S2 / (ms2 / 1e3), "mean_cg_steps": float(tot.float().mean()) / S2}
    return {
        "workload": w.name, "steps": S, "tokens_per_s": N * S / (ms / 1e3),
        "ms_per_step": ms / S,
        "hbm_GBps": bytes_per_step * S / (ms / 1e3) / 1e9,
        "hbm_frac": bytes_per_step * S / (ms / 1e3) / 1e9 / PEAKS["hbm_gbps"],
        "packed_state": packed,
        "dynamic_stopping": dyn,
    }


def cpu_model():
    """Model name of the host CPU from /proc/cpuinfo (None where unreadable)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_quota():
    """CPUs this process may keep busy: the cgroup CPU quota (cgroup v2 cpu.max),
    else the CPUs in its affinity mask."""
    import oracle
    usable = oracle.default_threads()
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        if quota != "max":
            return max(1, min(usable, int(int(quota) // int(period))))
    except (OSError, ValueError):
        pass
    return usable


def cpu_baseline(args, x, w):
    import numpy as np
    import oracle
    n_seq = args.cpu_sequences
    threads = min(n_seq, cpu_quota())
    pairs = [(i // w.heads % w.batch, i % w.heads) for i in range(n_seq)]
    sl = {n: np.stack([x[n][b, h] for b, h in pairs])[:, None] for n in ("q", "k", "v", "gamma", "beta")}
    # one head row of lambda per sequence: run the oracle once per distinct head set
    lam_rows = np.stack([x["lam"][h] for _, h in pairs])
    log("cpu baseline: oracle on %d sequences x T=%d with %d threads" % (n_seq, w.seq_len, threads))
    t0 = time.perf_counter()
    import concurrent.futures as cf

    def one(i):
        return oracle.forward(sl["q"][i:i + 1], sl["k"][i:i + 1], sl["v"][i:i + 1],
                              sl["gamma"][i:i + 1], sl["beta"][i:i + 1], lam_rows[i:i + 1], w.n_cg,
                              threads=1)["out"]
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(one, range(n_seq)))
    el = time.perf_counter() - t0
    token_heads = n_seq * w.seq_len
    return {
        "value": token_heads / w.heads / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
        "host_cpus": os.cpu_count(), "host_cpus_in_affinity": oracle.default_threads(),
        "host_cpus_quota": cpu_quota(), "cpu_model": cpu_model(),
        "sample": "%d of the %d (batch, head) sequences of %s (all of them when equal), %d tokens "
                  "each, fp64 sequential recurrence with %d-step CG, one sequence per thread; "
                  "tokens/s = token-heads/s / %d heads; %.1f s wall"
                  % (n_seq, w.batch * w.heads, w.name, w.seq_len, w.n_cg, w.heads, el),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--precision", type=int, default=2, choices=(1, 2, 3),
                    help="MESA_PREC_* of the timed steps: 2 single-pass bf16 (default), 3 split "
                         "operands, 1 fp32 products")
    ap.add_argument("--decode-steps", type=int, default=1024)
    ap.add_argument("--cpu-sequences", type=int, default=128)
    ap.add_argument("--skip-decode", action="store_true")
    ap.add_argument("--skip-backward", action="store_true")
    ap.add_argument("--skip-modes", action="store_true", help="skip the other precision modes")
    ap.add_argument("--skip-long", action="store_true", help="skip the long-context workload")
    ap.add_argument("--skip-layer-ends", action="store_true", help="skip the front and back end")
    ap.add_argument("--long-only", action="store_true",
                    help="time only the long-context workload and print its entry (a profiling aid; "
                         "not the metric)")
    ap.add_argument("--eps", type=float, default=1e-4,
                    help="relative CG tolerance of the extra dynamic-stopping runs (0: skip them)")
    ap.add_argument("--dyn-max-cg", type=int, default=30, help="iteration limit of those runs")
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, copy this many MiB once with a plain device copy "
                         "(reference dispatch for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: runs on one GPU only (--gpus 1); sharding the (batch, head) "
              "sequences across GPUs is not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_05233_amd import libmesa as L
    from paper_2506_05233_amd import workloads as W
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    L.load()

    if args.long_only:
        print(json.dumps({"long_context": run_long_context(args, torch, L, W)}), flush=True)
        return
    fw = run_forward(args, torch, L, W)
    w, t = fw["w"], fw["t"]
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    head = mode_entry(L, w, args.precision, t)
    modes = None if args.skip_modes else run_other_modes(args, torch, L, fw)
    ends = None if args.skip_layer_ends else run_layer_ends(args, torch, L, fw)
    dyn = run_forward_dynamic(args, torch, L, fw) if args.eps > 0 else None
    bwd = None if args.skip_backward else run_backward(args, torch, L, fw)
    longctx = None if args.skip_long else run_long_context(args, torch, L, W)
    dec = None if args.skip_decode else run_decode(args, torch, L, W)
    cpu = None if args.skip_cpu else cpu_baseline(args, fw["x"], w)

    tokens = w.batch * w.seq_len
    res = {
        "metric": METRIC,
        "value": tokens * args.steps / t["wall"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t["wall"] / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.precision == L.MESA_PREC_F32 else "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "heads": w.heads, "seq_len": w.seq_len,
                   "d_k": w.d_k, "d_v": w.d_v, "chunk": w.chunk, "n_cg": w.n_cg,
                   "inputs": PREC_TEXT[args.precision], "parallelism": "single GPU"},
        "roofline": head["roofline"],
        "kernels_ms": head["kernels_ms"],
        "state_kernel_hbm": head["state_kernel_hbm"],
        "other_precision_modes": modes,
        "long_context": longctx,
        "layer_front_and_back_end": ends,
        "forward_dynamic_stopping": dyn,
        "backward": bwd,
        "decode": dec,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
