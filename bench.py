#!/usr/bin/env python3
"""Benchmark of the Mesa layer forward (and decode) through libmesa on one MI355X.

A step is one forward pass of the layer over one batch of the 1B-shaped
workload (B=8, heads=16, T=2048, d_k=d_v=128, chunk 64, 15 CG steps, bf16
q/k/v, fp32 state and CG): the chunk-state scan launch, then the chunked CG +
read-out launch.  Inputs are resident in HBM before timing starts.  Each launch
is bracketed by HIP events on the stream it runs on; the CG launch is the
dominant kernel and its algorithmic flops per launch divided by its mean event
time give the roofline entry.  Decode (256 sequences x 16 heads, d=128,
15 CG steps, 1024 consecutive steps) is timed after the forward steps.

Two extra entries run the same forward and decode with Alg. 1's relative
stopping test (eps = 1e-4, at most 30 iterations, the paper's dynamic
test-time compute setting) and report tokens/s and the mean iterations used;
they are context, not the metric.  A third times the backward pass
(mesa_backward, App. D) of the same workload given dL/do and the forward's q*.

The CPU baseline is the fp64 oracle (the sequential recurrence with fixed-step
CG) on a bounded sample of the same workload, run on the host's cores.

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
    "fp32_vector_tflops": 157.3,
    "hbm_gbps": 8000.0,
}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def cg_kernel_flops(B, H, T, dk, dv, C, n_cg):
    """Algorithmic flops of one launch of the chunked CG + read-out kernel.
    Per token-head: (n_cg + 1) products (H_t + Lambda) p, each 2 d_k^2 for the
    state term plus 2 (C + 1) d_k for the causal intra-chunk K^T(Z (K p)) term
    (causal halves only), and the read-out 2 d_v d_k + (C + 1)(d_k + d_v)."""
    per_th = (n_cg + 1) * (2 * dk * dk + 2 * (C + 1) * dk) + 2 * dv * dk + (C + 1) * (dk + dv)
    return B * H * T * per_th


def state_kernel_bytes(B, H, T, dk, dv, C, in_bytes, state_bytes):
    """Algorithmic HBM bytes of the chunk-state launch: the states entering every
    chunk written once (state_bytes per element: 2 for the bf16 fragments of the
    bf16 path, 4 for fp32 states), plus k and v read once (gates ignored)."""
    nc = (T + C - 1) // C
    return B * H * nc * dk * (dk + dv) * state_bytes + B * H * T * (dk + dv) * in_bytes


def traffic_entry(kernel_src_hash):
    """HBM traffic of the CG kernel from committed rocprofv3 --pmc summaries, or
    None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "chunk_cg_layer1b_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


def source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2506_05233_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.startswith("chunk_cg") or name in ("mesa_device.hpp", "mesa_mfma.hpp"):
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()


def run_forward(args, torch, L, W):
    w = W.LAYER_1B_BF16
    log("generating %s inputs" % w.name)
    x = W.workload_inputs(w)
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16
    d = {}
    for name, a in x.items():
        t = torch.from_numpy(a).to(dev)
        d[name] = t.to(tdt) if name in ("q", "k", "v") else t
    plan = L.ForwardPlan(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], w.n_cg, w.chunk,
                         args.precision)
    log("warmup %d" % args.warmup)
    for _ in range(args.warmup):
        plan()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    log("timing %d steps" % args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record()
        plan.states()
        ev[i][1].record()
        plan.solve()
        ev[i][2].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    state_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    cg_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    out = plan.out
    if not bool(torch.isfinite(out).all()):
        raise RuntimeError("non-finite output")
    B, H, T, dk, dv = w.batch, w.heads, w.seq_len, w.d_k, w.d_v
    bf16_states = args.precision == L.MESA_PREC_BF16 or (
        args.precision == L.MESA_PREC_AUTO and L.bf16_path_available(dk, dv, w.chunk, T))
    return {
        "w": w, "wall": wall, "state_ms": state_ms, "cg_ms": cg_ms, "d": d, "plan": plan,
        "flops": cg_kernel_flops(B, H, T, dk, dv, w.chunk, w.n_cg),
        "state_bytes": state_kernel_bytes(B, H, T, dk, dv, w.chunk, 2, 2 if bf16_states else 4),
        "x": x,
    }


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
    res = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], w.n_cg, w.chunk,
                    precision=args.precision, want_qstar=True)
    qstar = res["qstar"]
    gen = torch.Generator(device="cuda").manual_seed(7)
    dout = torch.randn(d["v"].shape, dtype=torch.float32, device="cuda", generator=gen)
    ws = torch.empty(L.backward_workspace_bytes(w.batch, w.heads, w.seq_len, w.d_k, w.d_v),
                     dtype=torch.uint8, device="cuda")
    def call():
        return L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], qstar, dout, w.n_cg,
                          precision=args.precision, workspace=ws)
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
            "solve": "matrix cores (bf16 operands)" if args.precision != L.MESA_PREC_F32 else "fp32",
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
    ap.add_argument("--precision", type=int, default=0, help="MESA_PREC_* (0 = auto)")
    ap.add_argument("--decode-steps", type=int, default=1024)
    ap.add_argument("--cpu-sequences", type=int, default=128)
    ap.add_argument("--skip-decode", action="store_true")
    ap.add_argument("--skip-backward", action="store_true")
    ap.add_argument("--eps", type=float, default=1e-4,
                    help="relative CG tolerance of the extra dynamic-stopping runs (0: skip them)")
    ap.add_argument("--dyn-max-cg", type=int, default=30, help="iteration limit of those runs")
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, copy this many MiB once with a plain device copy "
                         "(reference dispatch for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (--gpus 1); the (batch, head) sharding "
              "across GPUs is described in DESIGN.md but not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_05233_amd import libmesa as L
    from paper_2506_05233_amd import workloads as W
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    L.load()

    fw = run_forward(args, torch, L, W)
    w = fw["w"]
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    dyn = run_forward_dynamic(args, torch, L, fw) if args.eps > 0 else None
    bwd = None if args.skip_backward else run_backward(args, torch, L, fw)
    dec = None if args.skip_decode else run_decode(args, torch, L, W)
    cpu = None if args.skip_cpu else cpu_baseline(args, fw["x"], w)

    prec = args.precision
    bf16_path = prec == L.MESA_PREC_BF16 or (prec == L.MESA_PREC_AUTO and
                                              L.bf16_path_available(w.d_k, w.d_v, w.chunk, w.seq_len))
    tokens = w.batch * w.seq_len
    cg_s = fw["cg_ms"] / 1e3
    achieved = fw["flops"] / cg_s / 1e12
    if bf16_path:
        roof = {"bound": "mfma", "peak": PEAKS["mfma_bf16_tflops"]}
    else:
        roof = {"bound": "alu", "peak": PEAKS["fp32_vector_tflops"]}
    roof.update({"achieved": achieved, "unit": "TFLOP/s", "frac": achieved / roof["peak"],
                 "traffic": traffic_entry(source_hash()),
                 "kernel": "chunk_cg (chunked CG + read-out)", "ms_per_launch": fw["cg_ms"],
                 "flops_per_launch": fw["flops"]})
    res = {
        "metric": METRIC,
        "value": tokens * args.steps / fw["wall"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": fw["wall"] / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16_path else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "heads": w.heads, "seq_len": w.seq_len,
                   "d_k": w.d_k, "d_v": w.d_v, "chunk": w.chunk, "n_cg": w.n_cg,
                   "inputs": "bf16 q/k/v, fp32 gates/lambda/state/CG",
                   "parallelism": "single GPU"},
        "roofline": roof,
        "kernels_ms": {"chunk_state": fw["state_ms"], "chunk_cg": fw["cg_ms"]},
        "state_kernel_hbm": {"GBps": fw["state_bytes"] / (fw["state_ms"] / 1e3) / 1e9,
                             "frac": fw["state_bytes"] / (fw["state_ms"] / 1e3) / 1e9 / PEAKS["hbm_gbps"]},
        "forward_dynamic_stopping": dyn,
        "backward": bwd,
        "decode": dec,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
