"""GPU parity of the backward pass (mesa_backward) against the fp64 oracle.

q*_t comes from the GPU forward on the fp32 path (mesa_forward_ex, qstar_out);
the oracle's backward recomputes q*_t and e*_t with the same-step CG (Alg. 1,
tolerance zero), so every gradient is compared element by element: at the fp32
tolerance when the solve for e*_t uses fp32 products, at the bf16 tolerance on
the matrix-core route (bf16 chunk states and right-hand sides, as the forward's
bf16 path).  Inputs given to the GPU in bf16 widen exactly for the oracle.
"""
import numpy as np
import pytest

import oracle
from mesa_testutil import TOL_BF16, TOL_F32, rel_l2, to_device
from paper_2506_05233_amd import libmesa as L
from paper_2506_05233_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GRADS = ("dq", "dk", "dv", "dgamma", "dbeta", "dlam")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L.load()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def _dout(x, seed):
    B, H, T, _ = x["v"].shape
    return np.random.default_rng(seed).normal(size=(B, H, T, x["v"].shape[-1])).astype(np.float32)


def _gpu_backward(x, dtype, n_cg, dout, precision=L.MESA_PREC_F32):
    d = to_device(x, dtype)
    fwd = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], n_cg, 64,
                    precision=L.MESA_PREC_F32, want_qstar=True)
    g = L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], fwd["qstar"],
                   torch.from_numpy(dout).cuda(), n_cg, precision=precision)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in g.items()}


def _check(x, dtype, n_cg, dout, label, tol=TOL_F32, precision=L.MESA_PREC_F32):
    got = _gpu_backward(x, dtype, n_cg, dout, precision)
    ref = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], dout, n_cg)
    errs = {k: rel_l2(got[k], ref[k]) for k in GRADS}
    _say("%s: %s" % (label, "  ".join("%s %.2e" % (k, e) for k, e in errs.items())))
    for k in GRADS:
        assert np.isfinite(got[k]).all(), k
        assert errs[k] <= tol, (k, errs[k])
    return got, ref


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_matches_oracle(dk, dv, dtype):
    """Three chunks and a ragged tail, every gradient against the oracle (fp32 solve)."""
    x = W.forward_inputs(1, 2, 3 * 64 + 17, dk, dv, dtype, 3.0, seed=dk + dv)
    _check(x, dtype, 10, _dout(x, 1), "backward %s d_k=%d d_v=%d" % (dtype, dk, dv))


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
def test_backward_matrix_core_solve_matches_oracle(dk, dv):
    """bf16 inputs, the solve for e* on the matrix cores (the default for bf16):
    every gradient within the bf16 tolerance, on two sequences with ragged tails and
    a zero gate."""
    x = W.forward_inputs(2, 2, 4 * 64 + 29, dk, dv, "bf16", 4.0, seed=3 * dk + dv)
    x["gamma"][1, 0, 100] = 0.0
    _check(x, "bf16", 15, _dout(x, 4), "backward matrix-core solve d_k=%d d_v=%d" % (dk, dv),
           tol=TOL_BF16, precision=L.MESA_PREC_AUTO)


@pytest.mark.parametrize("precision,tol", [(L.MESA_PREC_F32, TOL_F32), (L.MESA_PREC_AUTO, TOL_BF16)],
                         ids=["f32_solve", "matrix_core_solve"])
def test_backward_max_ncg(precision, tol):
    """The largest accepted iteration count (MESA_MAX_NCG) in the forward and in the
    solve for e*, bf16 inputs, against the oracle."""
    x = W.forward_inputs(1, 2, 70, 64, 64, "bf16", 4.0, seed=43)
    _check(x, "bf16", L.MESA_MAX_NCG, _dout(x, 5), "backward n_cg=%d" % L.MESA_MAX_NCG, tol=tol,
           precision=precision)


@pytest.mark.parametrize("precision", [L.MESA_PREC_F32, L.MESA_PREC_AUTO], ids=["f32_solve", "matrix_core_solve"])
def test_backward_is_bitwise_deterministic(precision):
    """No atomics and fixed summation orders: two calls give identical bits, also with
    the segmented adjoint walk (one sequence of 40 chunks)."""
    x = W.forward_inputs(1, 2, 40 * 64 - 5, 128, 128, "bf16", 4.0, seed=44)
    dout = _dout(x, 6)
    a = _gpu_backward(x, "bf16", 8, dout, precision)
    b = _gpu_backward(x, "bf16", 8, dout, precision)
    for k in GRADS:
        assert np.array_equal(a[k], b[k]), k


def test_backward_batch_sums_dlambda_and_edge_cases():
    """Three sequences (dLambda sums over the batch), zero forget gates at a chunk
    start, inside and at a chunk end, ignored tokens (beta = 0), a zero query."""
    x = W.forward_inputs(3, 2, 150, 64, 64, "f32", 3.0, seed=23)
    x["gamma"][0, 1, 40] = 0.0
    x["gamma"][1, 0, 64] = 0.0
    x["gamma"][2, 1, 63] = 0.0
    x["beta"][1, 1, 5:9] = 0.0
    x["q"][0, 0, 10] = 0.0
    _check(x, "f32", 12, _dout(x, 2), "backward edge cases")


@pytest.mark.parametrize("T", [1, 2, 63, 64, 65])
def test_backward_short_sequences(T):
    x = W.forward_inputs(1, 1, T, 64, 64, "f32", 3.0, seed=T)
    _check(x, "f32", 6, _dout(x, T), "backward T=%d" % T)


def test_backward_zero_dout_gives_zero_gradients():
    x = W.forward_inputs(1, 2, 100, 64, 64, "f32", 3.0, seed=3)
    got = _gpu_backward(x, "f32", 8, np.zeros((1, 2, 100, 64), np.float32))
    for k in GRADS:
        assert np.all(got[k] == 0.0), k


def test_backward_empty_sequence_zero_dlambda():
    d = to_device(W.forward_inputs(2, 3, 0, 64, 64, "f32", 3.0, 0), "f32")
    qs = torch.empty((2, 3, 0, 64), dtype=torch.float32, device="cuda")
    g = L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], qs,
                   torch.empty((2, 3, 0, 64), dtype=torch.float32, device="cuda"), 5)
    torch.cuda.synchronize()
    assert g["dlam"].shape == (3, 64) and float(g["dlam"].abs().max()) == 0.0


def test_backward_full_size_every_sequence():
    """The 1B-shaped workload (B8 H16 T2048 d128, bf16) in the launch configuration
    the benchmark times (forward on the bf16 path for q*, backward with the
    matrix-core solve), every gradient of every (batch, head) sequence and dLambda
    of every head against the oracle, which recomputes q* and e* in fp64 for the
    whole workload (one host thread per sequence)."""
    w = W.LAYER_1B_BF16
    x = W.workload_inputs(w)
    dout = np.random.default_rng(11).normal(size=x["v"].shape).astype(np.float32)
    d = to_device(x, "bf16")
    fwd = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], w.n_cg, w.chunk, want_qstar=True)
    g = L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], fwd["qstar"], torch.from_numpy(dout).cuda(), w.n_cg)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in g.items()}
    for k in GRADS:
        assert np.isfinite(got[k]).all(), k
    ref = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], dout, w.n_cg)
    errs = {k: rel_l2(got[k], ref[k]) for k in GRADS}
    _say("full-size backward, all sequences: %s" % "  ".join("%s %.2e" % kv for kv in errs.items()))
    for k, e in errs.items():
        assert e <= TOL_BF16, (k, e)
    # and sequence by sequence
    for k in ("dq", "dk", "dv"):
        dd = (got[k].astype(np.float64) - ref[k]) ** 2
        per = np.sqrt(dd.sum(axis=(2, 3)) / np.maximum((ref[k] ** 2).sum(axis=(2, 3)), 1e-300))
        assert per.max() <= TOL_BF16, (k, per.max())


@pytest.mark.parametrize("precision,tol", [(L.MESA_PREC_F32, TOL_F32), (L.MESA_PREC_BF16, TOL_BF16)],
                         ids=["f32_solve", "bf16_solve"])
def test_backward_segmented_walks_long_memory(precision, tol):
    """Two sequences of 36 chunks: the reverse adjoint scan (and, on the bf16 route, the
    state scan) run in 4 segments of 9 chunks.  Gates within 1e-3 of one keep every
    later segment's total relevant to the earlier ones; the workspace starts filled
    with ones, so scratch read before it is written would show.  Every gradient
    against the oracle."""
    T = 35 * 64 + 17
    x = W.forward_inputs(1, 2, T, 128, 128, "bf16", 4.0, seed=71)
    rng = np.random.default_rng(7101)
    x["gamma"][...] = rng.uniform(0.999, 1.0, size=x["gamma"].shape).astype(np.float32)
    dout = _dout(x, 9)
    d = to_device(x, "bf16")
    fwd = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], 15, 64,
                    precision=L.MESA_PREC_F32, want_qstar=True)
    ws = torch.ones(L.backward_workspace_bytes(1, 2, T, 128, 128) // 4, dtype=torch.float32, device="cuda")
    g = L.backward(d["k"], d["v"], d["gamma"], d["beta"], d["lam"], fwd["qstar"], torch.from_numpy(dout).cuda(), 15,
                   precision=precision, workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.backward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], dout, 15)
    errs = {k: rel_l2(g[k].cpu().numpy(), ref[k]) for k in GRADS}
    _say("segmented backward: %s" % "  ".join("%s %.2e" % kv for kv in errs.items()))
    for k, e in errs.items():
        assert e <= tol, (k, e)
