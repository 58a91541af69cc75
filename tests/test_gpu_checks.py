"""MESA_CHECK_FINITE: the forward and decode calls check their input values before their
launches (MESA_ERR_ARG, nothing launched) and their outputs after them
(MESA_ERR_NONFINITE).  The variable is read once per process, so each case runs in a
child process with it set; the child reports status codes and writes its outputs for
comparison with this process's (unchecked) run.
"""
import json
import os
import subprocess
import sys
import textwrap

import numpy as np
import pytest
import torch

from paper_2506_05233_amd import libmesa as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent('''
    import json, sys
    import numpy as np
    import torch
    sys.path.insert(0, %(root)r)
    from paper_2506_05233_amd import libmesa as L
    dev = "cuda"
    g = torch.Generator(device="cpu").manual_seed(3)
    B, H, T, d = 1, 2, 80, 64
    def unit(*shape):
        x = torch.randn(*shape, generator=g)
        return (x / x.norm(dim=-1, keepdim=True)).to(dev)
    base = dict(q=unit(B, H, T, d), k=unit(B, H, T, d), v=torch.randn(B, H, T, d, generator=g).to(dev),
                gamma=torch.sigmoid(3 + torch.randn(B, H, T, generator=g)).to(dev),
                beta=torch.sigmoid(torch.randn(B, H, T, generator=g)).to(dev),
                lam=(0.25 + 0.75 * torch.rand(H, d, generator=g)).to(dev))
    res = {}
    def run(name, **change):
        a = {k: v.clone() for k, v in base.items()}
        for k, (idx, val) in change.items():
            a[k][idx] = val
        out = torch.full((B, H, T, d), 7.0, device=dev)
        try:
            L.forward(a["q"], a["k"], a["v"], a["gamma"], a["beta"], a["lam"], 10, 64, out=out)
            st = L.MESA_OK
        except L.MesaError as e:
            st = e.status
        torch.cuda.synchronize()
        res[name] = [st, bool((out == 7.0).all())]
        return out
    ok = run("valid")
    np.save(%(out)r, ok.cpu().numpy())
    run("nan_q", q=((0, 1, 5, 3), float("nan")))
    run("inf_v", v=((0, 0, 70, 1), float("inf")))
    run("gamma_above_1", gamma=((0, 1, 40), 1.5))
    run("beta_below_0", beta=((0, 0, 0), -0.1))
    run("lambda_zero", lam=((1, 7), 0.0))
    # finite inputs whose states overflow: every value at the largest float, gates 1
    big = dict(v=((Ellipsis,), 3.0e38), gamma=((Ellipsis,), 1.0), beta=((Ellipsis,), 1.0))
    run("overflow", **big)
    # decode: a NaN in the state, then valid
    N, dk = 3, 64
    sH = torch.eye(dk, device=dev).repeat(N, H, 1, 1).contiguous()
    sG = torch.randn(N, H, dk, dk, generator=g).to(dev)
    q1, k1, v1 = unit(N, H, dk), unit(N, H, dk), torch.randn(N, H, dk, generator=g).to(dev)
    gm, bt = torch.full((N, H), 0.9, device=dev), torch.full((N, H), 0.5, device=dev)
    out1 = torch.full((N, H, dk), 7.0, device=dev)
    bad = sH.clone(); bad[1, 1, 3, 3] = float("nan")
    for name, state in (("decode_nan_state", bad), ("decode_valid", sH.clone())):
        try:
            L.decode_step(state, sG.clone(), q1, k1, v1, gm, bt, base["lam"], 10, out=out1)
            st = L.MESA_OK
        except L.MesaError as e:
            st = e.status
        torch.cuda.synchronize()
        res[name] = [st, bool((out1 == 7.0).all())]
    print("RESULT " + json.dumps(res), flush=True)
''')


@pytest.mark.gpu
def test_check_finite_flags_bad_values_and_leaves_results_alone(tmp_path):
    out_path = str(tmp_path / "checked_out.npy")
    env = dict(os.environ, MESA_CHECK_FINITE="1")
    proc = subprocess.run([sys.executable, "-c", CHILD % {"root": ROOT, "out": out_path}], env=env,
                          capture_output=True, text=True, timeout=300)
    assert proc.returncode == 0, proc.stderr[-3000:]
    line = [l for l in proc.stdout.splitlines() if l.startswith("RESULT ")][-1]
    res = json.loads(line[len("RESULT "):])
    print(res)
    # valid inputs: ok and the output written
    assert res["valid"] == [L.MESA_OK, False]
    # bad inputs: rejected before any launch, the output untouched
    for name in ("nan_q", "inf_v", "gamma_above_1", "beta_below_0", "lambda_zero"):
        assert res[name] == [L.MESA_ERR_ARG, True], name
    # finite inputs, overflowing states: the output check reports it
    assert res["overflow"][0] == L.MESA_ERR_NONFINITE
    assert res["decode_nan_state"] == [L.MESA_ERR_ARG, True]
    assert res["decode_valid"] == [L.MESA_OK, False]
    # the checked run computes what an unchecked run computes, bit for bit
    g = torch.Generator(device="cpu").manual_seed(3)
    B, H, T, d = 1, 2, 80, 64

    def unit(*shape):
        x = torch.randn(*shape, generator=g)
        return (x / x.norm(dim=-1, keepdim=True)).cuda()
    q, k = unit(B, H, T, d), unit(B, H, T, d)
    v = torch.randn(B, H, T, d, generator=g).cuda()
    gamma = torch.sigmoid(3 + torch.randn(B, H, T, generator=g)).cuda()
    beta = torch.sigmoid(torch.randn(B, H, T, generator=g)).cuda()
    lam = (0.25 + 0.75 * torch.rand(H, d, generator=g)).cuda()
    ref = L.forward(q, k, v, gamma, beta, lam, 10, 64).cpu().numpy()
    assert np.array_equal(np.load(out_path), ref)
