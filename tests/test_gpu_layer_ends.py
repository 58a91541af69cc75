"""GPU parity of the layer's front end (mesa_frontend) and back end (mesa_output_norm)
against the fp64 oracle (oracle/layer_ends.py), through the C ABI.

fp32 projections are compared at 1e-5 (fp32 arithmetic with the hardware exponential);
bf16 projections produce bf16 q, k, v, compared with the oracle on the same bf16
inputs at the bf16 rounding of the outputs (relative L2 4e-3, every element within
2^-8 relative plus 1e-6 absolute).  Gates and Lambda are fp32 in both cases."""
import numpy as np
import pytest

from mesa_testutil import rel_l2
from oracle import layer_ends as E
from paper_2506_05233_amd import libmesa as L
from paper_2506_05233_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L.load()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def _inputs(B, T, H, dk, dv, dtype, seed, conv_v=True):
    """Projections like those of a trained layer's input: N(0,1) entries, filters with
    taps of either sign, gate logits around the forget gate's operating range."""
    rng = np.random.default_rng(seed)
    x = {"qp": rng.standard_normal((B, T, H, dk)), "kp": rng.standard_normal((B, T, H, dk)),
         "vp": rng.standard_normal((B, T, H, dv)),
         "conv_q": rng.normal(0, 0.5, (H * dk, 4)), "conv_k": rng.normal(0, 0.5, (H * dk, 4)),
         "conv_v": rng.normal(0, 0.5, (H * dv, 4)) if conv_v else None,
         "a_gamma": rng.normal(4.0, 1.5, (B, T, H)), "a_beta": rng.normal(0.0, 1.5, (B, T, H)),
         "theta": rng.normal(0.0, 1.0, (H, dk))}
    for n in ("qp", "kp", "vp"):
        x[n] = x[n].astype(np.float32)
        if dtype == "bf16":
            x[n] = W.round_to_bf16(x[n])
    for n in ("conv_q", "conv_k", "conv_v", "a_gamma", "a_beta", "theta"):
        if x[n] is not None:
            x[n] = x[n].astype(np.float32)
    return x


def _dev(x, dtype):
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return {n: (None if a is None else torch.from_numpy(a).cuda().to(tdt if n in ("qp", "kp", "vp") else torch.float32))
            for n, a in x.items()}


def _check_front(x, dtype, cap=0.9975, eps=1e-6):
    d = _dev(x, dtype)
    got = L.frontend(d["qp"], d["kp"], d["vp"], d["conv_q"], d["conv_k"], d["conv_v"], d["a_gamma"], d["a_beta"],
                     d["theta"], gamma_cap=cap, l2_eps=eps)
    torch.cuda.synchronize()
    got = {n: t.float().cpu().numpy() for n, t in got.items()}
    ref = E.frontend(**x, gamma_cap=cap, l2_eps=eps)
    errs = {}
    for n in ("q", "k", "v"):
        e = rel_l2(got[n], ref[n])
        errs[n] = e
        if dtype == "bf16":
            assert e <= 4e-3, n
            assert np.all(np.abs(got[n] - ref[n]) <= 2.0 ** -8 * np.abs(ref[n]) + 1e-6), n
        else:
            assert e <= 1e-5, n
    for n in ("gamma", "beta", "lam"):
        errs[n] = float(np.max(np.abs(got[n] - ref[n]) / np.maximum(np.abs(ref[n]), 1e-30)))
        assert errs[n] <= 2e-6, n
    return errs


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_frontend_shapes_ragged(dk, dv, dtype):
    """Several 64-token runs per head plus a ragged one; every output element."""
    x = _inputs(2, 3 * 64 + 11, 3, dk, dv, dtype, seed=dk + dv + (dtype == "bf16"))
    errs = _check_front(x, dtype)
    _say("frontend %s d_k=%d d_v=%d: %s" % (dtype, dk, dv, " ".join("%s %.2e" % kv for kv in errs.items())))


def test_frontend_short_sequences_values_unfiltered_and_caps():
    """Sequences shorter than the filter (T = 1, 2, 3), a value stream without a filter,
    the cap off (b_gamma = 1) and at App. G.5's value, a zero projection row."""
    for T in (1, 2, 3, 65):
        x = _inputs(2, T, 2, 128, 128, "f32", seed=100 + T, conv_v=(T % 2 == 1))
        x["kp"][0, 0, 1] = 0.0
        _check_front(x, "f32", cap=1.0 if T == 2 else 0.9975)


def test_frontend_full_size_layer1b_shapes():
    """The 1B-shaped layer (B=8, heads=16, T=2048, d=128) in bf16, all outputs."""
    x = _inputs(8, 2048, 16, 128, 128, "bf16", seed=7)
    errs = _check_front(x, "bf16")
    _say("frontend full size: %s" % " ".join("%s %.2e" % kv for kv in errs.items()))


@pytest.mark.parametrize("dv", [64, 128])
@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_output_norm(dv, out_dtype):
    rng = np.random.default_rng(dv)
    B, H, T = 2, 3, 2 * 64 + 5
    o = (rng.standard_normal((B, H, T, dv)) * rng.uniform(0.01, 10, (B, H, T, 1))).astype(np.float32)
    wgt = rng.normal(1.0, 0.2, (H, dv)).astype(np.float32)
    tdt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    got = L.output_norm(torch.from_numpy(o).cuda(), torch.from_numpy(wgt).cuda(), 1e-6, out_dtype=tdt)
    torch.cuda.synchronize()
    got = got.float().cpu().numpy()
    ref = E.output_norm(o, wgt, 1e-6)
    e = rel_l2(got, ref)
    _say("output norm d_v=%d %s: %.2e" % (dv, out_dtype, e))
    if out_dtype == "bf16":
        assert e <= 4e-3 and np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6)
    else:
        assert e <= 1e-6


def test_layer_front_to_back_end_to_end():
    """Front end -> forward (split operands) -> back end on the GPU against the oracle's
    front end -> fp64 layer -> back end on the same projections, the oracle's keys,
    queries and values rounded to bf16 as the GPU's are: the composition a model runs.
    A bf16 rounding that lands on the other side of a tie for a few elements moves the
    output by ~1e-3, inside the bf16-input tolerance."""
    import oracle
    from mesa_testutil import TOL_BF16
    x = _inputs(1, 130, 2, 128, 128, "bf16", seed=11)
    d = _dev(x, "bf16")
    fe = L.frontend(d["qp"], d["kp"], d["vp"], d["conv_q"], d["conv_k"], d["conv_v"], d["a_gamma"], d["a_beta"],
                    d["theta"])
    out = L.forward(fe["q"], fe["k"], fe["v"], fe["gamma"], fe["beta"], fe["lam"], 15, 64)
    wgt = np.random.default_rng(3).normal(1.0, 0.1, (2, 128)).astype(np.float32)
    y = L.output_norm(out, torch.from_numpy(wgt).cuda(), 1e-6, out_dtype=torch.float32)
    torch.cuda.synchronize()
    r = E.frontend(**x)
    q, k, v = (W.round_to_bf16(r[n].astype(np.float32)) for n in ("q", "k", "v"))
    ref_o = oracle.forward(q, k, v, r["gamma"], r["beta"], r["lam"], 15)["out"]
    ref_y = E.output_norm(ref_o, wgt, 1e-6)
    e = rel_l2(y.cpu().numpy(), ref_y)
    _say("front end -> layer -> back end: %.2e" % e)
    assert e <= TOL_BF16
