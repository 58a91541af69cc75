"""GPU parity of libmesa against the fp64 oracle's same-step CG.

Every call goes through the C ABI (paper_2506_05233_amd.libmesa).  The oracle
consumes exactly the values the GPU receives (bf16 inputs widen exactly).
Every forward workload is compared element by element in full, the full-size
ones in the launch configuration the benchmark times (the oracle runs them over
all (batch, head) sequences, one host thread per sequence); decode over the
workload's 1024 steps is checked on sampled pairs.
"""
import concurrent.futures as cf
import os

import numpy as np
import pytest

import oracle
from mesa_testutil import TOL_BF16, TOL_F32, rel_l2, to_device
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


def _oracle_pairs(x, pairs, n_cg, **kw):
    """Oracle forward on the listed (b, h) sequences, one thread each."""
    def one(bh):
        b, h = bh
        sl = {n: x[n][b:b + 1, h:h + 1] for n in ("q", "k", "v", "gamma", "beta")}
        return oracle.forward(sl["q"], sl["k"], sl["v"], sl["gamma"], sl["beta"], x["lam"][h:h + 1],
                              n_cg, threads=1, **kw)
    with cf.ThreadPoolExecutor(max_workers=min(16, len(pairs))) as ex:
        return list(ex.map(one, pairs))


def _gpu_forward(x, dtype, n_cg, chunk, **kw):
    d = to_device(x, dtype)
    res = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], n_cg, chunk, **kw)
    torch.cuda.synchronize()
    if isinstance(res, dict):
        return {k: v.cpu().numpy() for k, v in res.items()}
    return res.cpu().numpy()


# ------------------------------------------------------------ small, in full
@pytest.mark.parametrize("w", [W.TINY_F32, W.SMALL_F32], ids=lambda w: w.name)
def test_forward_f32_workloads_full(w):
    _say("forward parity %s" % w.name)
    x = W.workload_inputs(w)
    got = _gpu_forward(x, w.dtype, w.n_cg, w.chunk, want_qstar=True, want_states=True)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], w.n_cg,
                         want_qstar=True, want_states=True)
    e_out = rel_l2(got["out"], ref["out"])
    e_q = rel_l2(got["qstar"], ref["qstar"])
    _say("  out %.3e  qstar %.3e" % (e_out, e_q))
    assert e_out <= TOL_F32 and e_q <= TOL_F32
    assert rel_l2(got["H"], ref["H"]) <= 1e-5 and rel_l2(got["G"], ref["G"]) <= 1e-5


def test_forward_bf16_small_full_auto_precision():
    x = W.forward_inputs(2, 3, 320, 128, 128, "bf16", 4.0, seed=11)
    got = _gpu_forward(x, "bf16", 15, 64)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15)["out"]
    e = rel_l2(got, ref)
    _say("bf16 small auto: %.3e" % e)
    assert e <= TOL_BF16


@pytest.mark.parametrize("dk,dv", [(64, 128), (128, 64), (128, 128)])
@pytest.mark.parametrize("chunk", [16, 32, 64])
def test_forward_shapes_ragged_tail(dk, dv, chunk):
    """T not a multiple of the chunk: several chunks plus a ragged last one."""
    x = W.forward_inputs(1, 2, 3 * chunk + 7, dk, dv, "f32", 3.0, seed=dk + dv + chunk)
    got = _gpu_forward(x, "f32", 9, chunk, precision=L.MESA_PREC_F32, want_states=True)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 9, want_states=True)
    assert rel_l2(got["out"], ref["out"]) <= TOL_F32
    assert rel_l2(got["H"], ref["H"]) <= 1e-5 and rel_l2(got["G"], ref["G"]) <= 1e-5


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
def test_forward_bf16_matrix_core_path_shapes(dk, dv):
    """bf16 inputs, chunk 64 (the matrix-core path): several chunks plus a
    ragged tail, every output and every q* against the oracle."""
    assert L.bf16_path_available(dk, dv, 64)
    x = W.forward_inputs(2, 2, 3 * 64 + 29, dk, dv, "bf16", 4.0, seed=dk + 2 * dv)
    got = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16, want_qstar=True)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15, want_qstar=True)
    e_out, e_q = rel_l2(got["out"], ref["out"]), rel_l2(got["qstar"], ref["qstar"])
    _say("bf16 path d_k=%d d_v=%d: out %.3e qstar %.3e" % (dk, dv, e_out, e_q))
    assert e_out <= TOL_BF16 and e_q <= TOL_BF16


def test_bf16_path_edge_cases():
    x = W.forward_inputs(2, 2, 150, 128, 128, "bf16", 4.0, seed=31)
    x["gamma"][0, 1, 40] = 0.0
    x["gamma"][1, 0, 64] = 0.0
    x["gamma"][1, 1, 63] = 0.0
    x["q"][0, 0, 10] = 0.0
    x["beta"][1, 0, 5:9] = 0.0
    # 0 (Jacobi start only), 1 and 3 (the CG loop's odd tail), 2 and 15 (whole pairs of
    # iterations, then a tail)
    for n_cg in (0, 1, 2, 3, 15):
        got = _gpu_forward(x, "bf16", n_cg, 64, precision=L.MESA_PREC_BF16)
        ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], n_cg)["out"]
        e = rel_l2(got, ref)
        _say("bf16 edge n_cg=%d: %.3e" % (n_cg, e))
        assert e <= TOL_BF16, n_cg
        assert np.all(got[0, 0, 10] == 0.0)


def test_bf16_path_strong_decay():
    """Gates in [0.25, 0.6]: the decay across 32-48 tokens drops below 1e-20, so the
    later sub-chunk states of every chunk are built without the chunk state, and the
    earlier ones carry rank-update weights up to ~1e14 (both regimes of the
    sub-chunk states of the matrix-core path), checked over every output."""
    x = W.forward_inputs(2, 2, 4 * 64 + 17, 128, 128, "bf16", 4.0, seed=43)
    rng = np.random.default_rng(4301)
    x["gamma"][...] = rng.uniform(0.25, 0.6, size=x["gamma"].shape).astype(np.float32)
    for n_cg in (0, 15):
        got = _gpu_forward(x, "bf16", n_cg, 64, precision=L.MESA_PREC_BF16, want_qstar=True)
        ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], n_cg, want_qstar=True)
        e_out, e_q = rel_l2(got["out"], ref["out"]), rel_l2(got["qstar"], ref["qstar"])
        _say("bf16 strong decay n_cg=%d: out %.3e qstar %.3e" % (n_cg, e_out, e_q))
        assert e_out <= TOL_BF16 and e_q <= TOL_BF16, n_cg


def test_bf16_path_query_scale_is_exact():
    """o is positively homogeneous in q (App. C: every CG iterate scales with the
    right-hand side).  The matrix-core path solves each column for q scaled by a power
    of two, so scaling q by 2^k, from 2^-60 to 2^60, must scale out by exactly 2^k, bit
    for bit, and stay within the bf16 tolerance of the oracle."""
    x = W.forward_inputs(1, 2, 128 + 40, 128, 128, "bf16", 4.0, seed=47)
    base = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15)["out"]
    assert rel_l2(base, ref) <= TOL_BF16
    for k in (-60, -20, 7, 60):
        y = dict(x)
        y["q"] = (x["q"].astype(np.float64) * 2.0 ** k).astype(np.float32)
        got = _gpu_forward(y, "bf16", 15, 64, precision=L.MESA_PREC_BF16)
        _say("q scaled by 2^%d: max |got/2^k - base| = %.3e" % (k, np.abs(got * 2.0 ** -k - base).max()))
        assert np.array_equal(got, (base.astype(np.float64) * 2.0 ** k).astype(np.float32)), k


def test_stress_repeated_keys_bf16_path_reported():
    """Single-pass bf16 operands are validated on the workload distributions, not
    on adversarial inputs: on the repeated-key stress input (App. G.5's repeated
    tokens with gates near one) the error exceeds the bf16 tolerance.  It is pinned
    near its measured value (~0.13 with one repeated key) so that a regression shows."""
    x = W.repeated_key_inputs(1, 2, 512, 128, 128, pool=1, dtype="bf16")
    got = _gpu_forward(x, "bf16", 20, 64, precision=L.MESA_PREC_BF16)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 20)["out"]
    e = rel_l2(got, ref)
    _say("stress pool=1 bf16 matrix-core products: %.3e" % e)
    assert np.isfinite(got).all() and e <= 0.15


def test_chunk_size_invariance():
    x = W.forward_inputs(1, 2, 256, 64, 64, "f32", 3.0, seed=5)
    outs = [_gpu_forward(x, "f32", 10, c, precision=L.MESA_PREC_F32) for c in (16, 32, 64)]
    assert rel_l2(outs[0], outs[2]) <= 1e-5 and rel_l2(outs[1], outs[2]) <= 1e-5


def test_edge_cases_zero_gates_zero_queries_short_sequences():
    x = W.forward_inputs(2, 2, 97, 64, 64, "f32", 3.0, seed=21)
    x["gamma"][0, 1, 40] = 0.0      # memory reset inside a chunk
    x["gamma"][1, 0, 64] = 0.0      # reset at a chunk start
    x["gamma"][1, 1, 63] = 0.0      # reset at a chunk end
    x["q"][0, 0, 10] = 0.0          # q = 0 -> o = 0
    x["beta"][1, 0, 5:9] = 0.0      # ignored tokens
    for n_cg in (0, 1, 12):
        got = _gpu_forward(x, "f32", n_cg, 64, precision=L.MESA_PREC_F32)
        ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], n_cg)["out"]
        assert rel_l2(got, ref) <= TOL_F32, n_cg
        assert np.all(got[0, 0, 10] == 0.0)
    for T in (1, 2, 63, 64, 65):
        y = W.forward_inputs(1, 1, T, 64, 64, "f32", 3.0, seed=T)
        got = _gpu_forward(y, "f32", 6, 64, precision=L.MESA_PREC_F32)
        ref = oracle.forward(y["q"], y["k"], y["v"], y["gamma"], y["beta"], y["lam"], 6)["out"]
        assert rel_l2(got, ref) <= TOL_F32, T


def test_empty_sequence_gives_zero_states():
    d = to_device(W.forward_inputs(2, 2, 0, 64, 64, "f32", 3.0, 0), "f32")
    H, G = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"])
    torch.cuda.synchronize()
    assert H.shape == (2, 2, 64, 64) and float(H.abs().max()) == 0.0 and float(G.abs().max()) == 0.0


def test_prefill_states_match_oracle():
    x = W.forward_inputs(2, 2, 200, 128, 64, "bf16", 4.0, seed=8)
    d = to_device(x, "bf16")
    H, G = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"])
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 0, want_states=True)
    assert rel_l2(H.cpu().numpy(), ref["H"]) <= 1e-5
    assert rel_l2(G.cpu().numpy(), ref["G"]) <= 1e-5


@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 64), (64, 128), (128, 128)])
def test_f32_state_scan_ring_tails(dk, dv):
    """fp32 scan (chunk 64): sequences of 1, 3, 4, 5 and 9 chunks, most with a ragged
    last chunk, cover the scan's four-chunk load ring in full passes and with every
    tail length; a zero gate on a chunk's first token and one inside a chunk reset
    memory exactly.  The states-only call's final states and the forward's output
    (which reads every chunk state) and final states against the oracle."""
    for T in (37, 3 * 64, 4 * 64, 4 * 64 + 1, 8 * 64 + 50):
        x = W.forward_inputs(2, 2, T, dk, dv, "f32", 3.0, seed=T + dk + dv)
        x["gamma"][0, 1, T // 2] = 0.0
        if T > 128:
            x["gamma"][1, 0, 128] = 0.0
        d = to_device(x, "f32")
        H, G = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"])
        got = _gpu_forward(x, "f32", 6, 64, precision=L.MESA_PREC_F32, want_states=True)
        ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 6, want_states=True)
        e = [rel_l2(H.cpu().numpy(), ref["H"]), rel_l2(G.cpu().numpy(), ref["G"]),
             rel_l2(got["H"], ref["H"]), rel_l2(got["G"], ref["G"]), rel_l2(got["out"], ref["out"])]
        _say("f32 scan d_k=%d d_v=%d T=%d: H %.2e G %.2e (forward H %.2e G %.2e out %.2e)" % (dk, dv, T, *e))
        assert max(e[:4]) <= 2e-6 and e[4] <= TOL_F32, T


@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 128)])
def test_segmented_state_scan_matches_oracle(dk, dv):
    """Two sequences of 36 chunks (the last ragged): the bf16 scan runs in 4 segments
    of 9 chunks, totals first, then every segment from the state entering it.  Zero
    gates sit inside a segment and on the first token of one (a memory reset the
    entering state must honour).  Every output, the final states (fp32) and the
    states-only call with scratch against the oracle; the states-only call without
    scratch walks unsegmented and must agree with it to fp32 rounding."""
    T = 35 * 64 + 17
    x = W.forward_inputs(1, 2, T, dk, dv, "bf16", 4.0, seed=61 + dk)
    x["gamma"][0, 0, 9 * 64 + 100] = 0.0
    x["gamma"][0, 1, 18 * 64] = 0.0
    got = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16, want_states=True)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15, want_states=True)
    e_out = rel_l2(got["out"], ref["out"])
    e_h, e_g = rel_l2(got["H"], ref["H"]), rel_l2(got["G"], ref["G"])
    _say("segmented scan d_k=%d d_v=%d: out %.3e  H %.3e  G %.3e" % (dk, dv, e_out, e_h, e_g))
    assert e_out <= TOL_BF16 and e_h <= 1e-5 and e_g <= 1e-5
    d = to_device(x, "bf16")
    ws = torch.empty(L.forward_workspace_bytes(1, 2, T, dk, dv, 64), dtype=torch.uint8, device="cuda")
    Hs, Gs = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"], workspace=ws)
    H1, G1 = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"])
    torch.cuda.synchronize()
    assert rel_l2(Hs.cpu().numpy(), ref["H"]) <= 1e-5 and rel_l2(Gs.cpu().numpy(), ref["G"]) <= 1e-5
    assert rel_l2(Hs.cpu().numpy(), H1.cpu().numpy()) <= 1e-6
    assert rel_l2(Gs.cpu().numpy(), G1.cpu().numpy()) <= 1e-6


@pytest.mark.parametrize("d", [64, 128])
def test_segmented_forward_bf16_states_only_path(d):
    """The forward without fp32 final states: the bf16 scan's segment totals and its
    walk both run on the single-product kernels (each of a sequence's two workgroups
    owning half the columns of H and of G^T).  Gates within 1e-3 of one keep every
    earlier segment visible in the outputs, and a zero gate resets memory inside a
    segment; every output against the oracle."""
    T = 35 * 64 + 17
    x = W.forward_inputs(1, 2, T, d, d, "bf16", 4.0, seed=71 + d)
    rng = np.random.default_rng(7101 + d)
    x["gamma"][...] = rng.uniform(0.999, 1.0, size=x["gamma"].shape).astype(np.float32)
    x["gamma"][0, 1, 20 * 64 + 5] = 0.0
    got = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15)["out"]
    e = rel_l2(got, ref)
    _say("segmented forward d=%d, gates near one: out %.3e" % (d, e))
    assert e <= TOL_BF16


def test_segmented_state_scan_long_memory():
    """Gates within 1e-3 of one (a few exactly one): the decay across a 9-chunk segment
    stays above 0.5, so every earlier segment's total reaches the final states with a
    weight the fp32 check sees -- a wrong combination coefficient or a dropped segment
    fails here.  The workspace starts filled with ones, so a read of scratch that the
    scan has not written yet shows too.  The final states of the segmented scan
    (forward and states-only with scratch) against the oracle, and against the
    unsegmented states-only walk; the output against the oracle at the bf16 tolerance."""
    T = 35 * 64 + 17
    x = W.forward_inputs(1, 2, T, 128, 128, "bf16", 4.0, seed=67)
    rng = np.random.default_rng(6701)
    x["gamma"][...] = rng.uniform(0.999, 1.0, size=x["gamma"].shape).astype(np.float32)
    x["gamma"][0, 0, ::97] = 1.0
    need = L.forward_workspace_bytes(1, 2, T, 128, 128, 64)
    got = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16, want_states=True,
                       workspace=torch.ones(need // 4, dtype=torch.float32, device="cuda"))
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 15, want_states=True)
    e_out = rel_l2(got["out"], ref["out"])
    e_h, e_g = rel_l2(got["H"], ref["H"]), rel_l2(got["G"], ref["G"])
    _say("segmented scan, gates near one: out %.3e  H %.3e  G %.3e" % (e_out, e_h, e_g))
    assert e_h <= 1e-5 and e_g <= 1e-5
    assert e_out <= TOL_BF16
    d = to_device(x, "bf16")
    ws = torch.ones(need // 4, dtype=torch.float32, device="cuda")
    Hs, Gs = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"], workspace=ws)
    H1, G1 = L.prefill_states(d["k"], d["v"], d["gamma"], d["beta"])
    torch.cuda.synchronize()
    assert rel_l2(Hs.cpu().numpy(), ref["H"]) <= 1e-5 and rel_l2(Gs.cpu().numpy(), ref["G"]) <= 1e-5
    assert rel_l2(Hs.cpu().numpy(), H1.cpu().numpy()) <= 1e-6
    assert rel_l2(Gs.cpu().numpy(), G1.cpu().numpy()) <= 1e-6


def test_forward_is_bitwise_deterministic():
    x = W.forward_inputs(2, 4, 512, 128, 128, "bf16", 4.0, seed=9)
    a = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16)
    b = _gpu_forward(x, "bf16", 15, 64, precision=L.MESA_PREC_BF16)
    assert np.array_equal(a, b)


def test_stress_repeated_keys_f32_path():
    """Keys from a pool of one vector, gates near one: the ill-conditioned case."""
    x = W.repeated_key_inputs(1, 2, 512, 128, 128, pool=1, dtype="bf16")
    got = _gpu_forward(x, "bf16", 20, 64, precision=L.MESA_PREC_F32)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 20)["out"]
    e = rel_l2(got, ref)
    _say("stress pool=1 f32 products: %.3e" % e)
    assert e <= TOL_F32


# ------------------------------------------------------- full size, in full
def _per_sequence_rel_l2(got, ref):
    """Relative L2 error of each (batch, head) sequence, [B, H]."""
    d = (got.astype(np.float64) - ref) ** 2
    return np.sqrt(d.sum(axis=(2, 3)) / np.maximum((ref ** 2).sum(axis=(2, 3)), 1e-300))


@pytest.mark.parametrize("w", [W.LAYER_1B_BF16, W.LONG_BF16], ids=["layer1b", "longctx"])
def test_forward_full_size_every_sequence(w):
    """Single-pass matrix-core products (the benchmarked mode) at full size, every
    output of every (batch, head) sequence against the oracle (which runs the whole
    workload, one host thread per sequence); the split-operand mode has its own
    full-size test."""
    _say("full-size forward %s, all %d sequences" % (w.name, w.batch * w.heads))
    x = W.workload_inputs(w)
    got = _gpu_forward(x, w.dtype, w.n_cg, w.chunk, precision=L.MESA_PREC_BF16)
    assert np.isfinite(got).all()
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], w.n_cg)["out"]
    e = rel_l2(got, ref)
    per = _per_sequence_rel_l2(got, ref)
    _say("  rel L2 %.3e, worst sequence %.3e at %s" % (e, per.max(), np.unravel_index(per.argmax(), per.shape)))
    tol = TOL_BF16 if w.dtype == "bf16" else TOL_F32
    assert e <= tol and per.max() <= tol


# ------------------------------------------------------------------- decode
def _decode_state_pool(w, n_pool):
    """Oracle-prefilled states of the first n_pool sequences' head-0..H-1 pairs."""
    toks = W.decode_prefill_tokens(w, 0, n_pool)
    H, G = oracle.unrolled_states(toks["k"], toks["v"], toks["gamma"], toks["beta"])
    return H.astype(np.float32), G.astype(np.float32)   # [n_pool, H, d, d]


def test_decode_full_workload_1024_steps():
    """The decode workload as specified: 256 sequences x 16 heads, d = 128, 15 CG
    steps, 1024 consecutive steps, on the full layout and (separately) on the packed
    symmetric state.  Every pair starts from an oracle-prefilled state (4096 gated
    updates; 8 distinct sequences' states, sequence s taking those of s % 8) and
    receives its own seeded token at every step.  Checked against the oracle:
    every pair over the first 16 steps; 64 sampled pairs (four sequences with
    distinct prefill states x 16 heads) at every one of the 1024 steps, and their
    states after the last step."""
    w = W.DECODE_BF16
    n_pool, n_all = 8, 16
    _say("decode %s: 1024 steps on the full batch" % w.name)
    Hp, Gp = _decode_state_pool(w, n_pool)
    Hp = np.triu(Hp) + np.swapaxes(np.triu(Hp, 1), -1, -2)   # exactly symmetric fp32
    idx = np.arange(w.seqs) % n_pool
    H0 = np.ascontiguousarray(Hp[idx])
    G0 = np.ascontiguousarray(Gp[idx])
    lam = W.decode_lambda(w)
    dlam = torch.from_numpy(lam).cuda()
    dH, dG = torch.from_numpy(H0).cuda(), torch.from_numpy(G0).cuda()
    pH, pG = L.pack_state(dH), dG.clone()
    sample = [0, 13, 130, 255]                # prefill states 0, 5, 2, 7
    rH = H0[sample].astype(np.float64)
    rG = G0[sample].astype(np.float64)
    first_in, first_out = [], []
    worst_full, worst_packed, worst_at = 0.0, 0.0, {}
    for step in range(w.steps):
        x = W.decode_step_inputs(w, step)
        d = to_device(x, w.dtype)
        of = L.decode_step(dH, dG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], dlam, w.n_cg)
        op = L.decode_step(pH, pG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], dlam, w.n_cg, packed=True)
        torch.cuda.synchronize()
        of, op = of.cpu().numpy(), op.cpu().numpy()
        assert np.isfinite(of).all() and np.isfinite(op).all(), step
        if step < n_all:
            first_in.append(x)
            first_out.append((of, op))
        sx = {n: x[n][sample] for n in x}
        ro, rH, rG = oracle.decode_step(rH, rG, sx["q"], sx["k"], sx["v"], sx["gamma"], sx["beta"],
                                        lam, w.n_cg, threads=16)
        ef, ep = rel_l2(of[sample], ro), rel_l2(op[sample], ro)
        worst_full, worst_packed = max(worst_full, ef), max(worst_packed, ep)
        if step + 1 in (1, 16, 64, 256, 1024):
            worst_at[step + 1] = (ef, ep)
        if (step + 1) % 128 == 0:
            _say("  step %d: sampled pairs rel L2 full %.2e packed %.2e" % (step + 1, ef, ep))
    _say("  worst over 1024 steps: full %.3e packed %.3e; at steps %s" % (worst_full, worst_packed, worst_at))
    assert worst_full <= TOL_BF16 and worst_packed <= TOL_BF16
    eH, eG = rel_l2(dH.cpu().numpy()[sample], rH), rel_l2(dG.cpu().numpy()[sample], rG)
    ePH = rel_l2(L.unpack_state(pH).cpu().numpy()[sample], rH)
    ePG = rel_l2(pG.cpu().numpy()[sample], rG)
    _say("  final states rel L2: H %.2e G %.2e (packed H %.2e G %.2e)" % (eH, eG, ePH, ePG))
    assert max(eH, eG, ePH, ePG) <= 1e-5
    # every pair over the first 16 steps, the oracle run in slices of 32 sequences
    worst_all = 0.0
    for s0 in range(0, w.seqs, 32):
        sl = slice(s0, s0 + 32)
        qH, qG = H0[sl].astype(np.float64), G0[sl].astype(np.float64)
        for step in range(n_all):
            x = first_in[step]
            ro, qH, qG = oracle.decode_step(qH, qG, x["q"][sl], x["k"][sl], x["v"][sl], x["gamma"][sl],
                                            x["beta"][sl], lam, w.n_cg, threads=16)
            of, op = first_out[step]
            worst_all = max(worst_all, rel_l2(of[sl], ro), rel_l2(op[sl], ro))
    _say("  all 4096 pairs, first %d steps: worst rel L2 %.3e" % (n_all, worst_all))
    assert worst_all <= TOL_BF16


def test_decode_f32_matches_oracle_tightly():
    x = W.forward_inputs(3, 2, 1, 64, 128, "f32", 3.0, seed=3)
    rng = np.random.default_rng(0)
    H0, G0 = oracle.unrolled_states(rng.standard_normal((3, 2, 50, 64)) / 8,
                                    rng.standard_normal((3, 2, 50, 128)),
                                    np.full((3, 2, 50), 0.97), np.full((3, 2, 50), 0.5))
    H0 = H0.astype(np.float32)
    G0 = G0.astype(np.float32)
    d = to_device({k: v[:, :, 0] for k, v in x.items() if k != "lam"}, "f32")
    dH, dG = torch.from_numpy(H0).cuda(), torch.from_numpy(G0).cuda()
    lam = torch.from_numpy(x["lam"]).cuda()
    out = L.decode_step(dH, dG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], lam, 12)
    ro, rH, rG = oracle.decode_step(H0, G0, x["q"][:, :, 0], x["k"][:, :, 0], x["v"][:, :, 0],
                                    x["gamma"][:, :, 0], x["beta"][:, :, 0], x["lam"], 12)
    assert rel_l2(out.cpu().numpy(), ro) <= TOL_F32
    assert rel_l2(dH.cpu().numpy(), rH) <= 1e-6 and rel_l2(dG.cpu().numpy(), rG) <= 1e-6


def test_max_ncg_forward_and_decode():
    """The largest accepted iteration count, MESA_MAX_NCG, on small inputs: the forward's
    CG loop on both matrix-core paths (bf16 operands: 512 pairs of iterations; fp32), the
    scalar fp32 kernel (chunk 32) and
    the decode step run every iteration (eps = 0, so fp32 columns keep iterating on a
    residual at the rounding floor) and still agree with the oracle's fp64 CG."""
    n = L.MESA_MAX_NCG
    x = W.forward_inputs(1, 2, 70, 64, 64, "bf16", 4.0, seed=41)
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], n)["out"]
    e_b = rel_l2(_gpu_forward(x, "bf16", n, 64, precision=L.MESA_PREC_BF16), ref)
    e_f = rel_l2(_gpu_forward(x, "bf16", n, 64, precision=L.MESA_PREC_F32), ref)
    e_s = rel_l2(_gpu_forward(x, "bf16", n, 32, precision=L.MESA_PREC_F32), ref)  # scalar fp32 kernel
    _say("n_cg = %d: bf16 operands %.3e, fp32 %.3e, fp32 chunk 32 %.3e" % (n, e_b, e_f, e_s))
    assert e_b <= TOL_BF16 and e_f <= TOL_F32 and e_s <= TOL_F32
    y = W.forward_inputs(2, 2, 1, 64, 64, "f32", 3.0, seed=42)
    rng = np.random.default_rng(1)
    H0, G0 = oracle.unrolled_states(rng.standard_normal((2, 2, 40, 64)) / 8,
                                    rng.standard_normal((2, 2, 40, 64)),
                                    np.full((2, 2, 40), 0.95), np.full((2, 2, 40), 0.5))
    H0, G0 = H0.astype(np.float32), G0.astype(np.float32)
    d = to_device({k: v[:, :, 0] for k, v in y.items() if k != "lam"}, "f32")
    dH, dG = torch.from_numpy(H0).cuda(), torch.from_numpy(G0).cuda()
    out = L.decode_step(dH, dG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], torch.from_numpy(y["lam"]).cuda(), n)
    ro, _, _ = oracle.decode_step(H0, G0, y["q"][:, :, 0], y["k"][:, :, 0], y["v"][:, :, 0],
                                  y["gamma"][:, :, 0], y["beta"][:, :, 0], y["lam"], n)
    e_d = rel_l2(out.cpu().numpy(), ro)
    _say("n_cg = %d: decode %.3e" % (n, e_d))
    assert e_d <= TOL_F32


def test_decode_steps_from_zero_equal_forward():
    x = W.forward_inputs(2, 2, 70, 128, 128, "bf16", 4.0, seed=12)
    fwd = _gpu_forward(x, "bf16", 10, 64, precision=L.MESA_PREC_F32)
    d = to_device(x, "bf16")
    dH = torch.zeros((2, 2, 128, 128), device="cuda")
    dG = torch.zeros((2, 2, 128, 128), device="cuda")
    outs = []
    for t in range(70):
        outs.append(L.decode_step(dH, dG, d["q"][:, :, t].contiguous(), d["k"][:, :, t].contiguous(),
                                  d["v"][:, :, t].contiguous(), d["gamma"][:, :, t].contiguous(),
                                  d["beta"][:, :, t].contiguous(), d["lam"], 10).cpu().numpy())
    dec = np.stack(outs, axis=2)
    assert rel_l2(dec, fwd) <= 1e-4


# --------------------------------------------- dynamic stopping (App. C, Alg. 1, eps > 0)
def _steps_agreement(got_steps, ref_steps, what):
    diff = np.abs(got_steps.astype(np.int64) - ref_steps.astype(np.int64))
    _say("%s: steps equal %.4f, max |diff| %d, mean steps gpu %.2f oracle %.2f"
         % (what, np.mean(diff == 0), diff.max(), got_steps.mean(), ref_steps.mean()))
    return diff


@pytest.mark.parametrize("eps", [1e-2, 1e-4])
def test_forward_tolerance_f32_matches_oracle(eps):
    """fp32 path: the iteration counts match the oracle's except where a residual
    sits within rounding of the threshold (then by one step); outputs of tokens
    with equal counts match to the fp32 tolerance, the others to O(eps)."""
    x = W.forward_inputs(2, 2, 3 * 64 + 21, 64, 64, "f32", 3.0, seed=61)
    d = to_device(x, "f32")
    res = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], 40, 64,
                    precision=L.MESA_PREC_F32, eps=eps, want_steps=True)
    torch.cuda.synchronize()
    out, steps = res["out"].cpu().numpy(), res["steps"].cpu().numpy()
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 40, eps=eps, want_steps=True)
    diff = _steps_agreement(steps, ref["steps"], "f32 eps=%g" % eps)
    assert diff.max() <= 1 and np.mean(diff == 0) >= 0.98
    same = diff == 0
    assert rel_l2(out[same], ref["out"][same]) <= TOL_F32
    assert rel_l2(out, ref["out"]) <= 20 * eps + TOL_F32
    assert steps.max() < 40  # the tolerance, not the limit, ended every solve


@pytest.mark.parametrize("eps", [1e-2, 1e-4])
def test_forward_tolerance_bf16_path_matches_oracle(eps):
    """Matrix-core path: recursive residuals stay within rounding of the oracle's,
    so counts agree to a step or two and outputs to the bf16 tolerance."""
    x = W.forward_inputs(2, 2, 2 * 64 + 40, 128, 128, "bf16", 4.0, seed=62)
    d = to_device(x, "bf16")
    res = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], 40, 64,
                    precision=L.MESA_PREC_BF16, eps=eps, want_steps=True)
    torch.cuda.synchronize()
    out, steps = res["out"].cpu().numpy(), res["steps"].cpu().numpy()
    ref = oracle.forward(x["q"], x["k"], x["v"], x["gamma"], x["beta"], x["lam"], 40, eps=eps, want_steps=True)
    diff = _steps_agreement(steps, ref["steps"], "bf16 eps=%g" % eps)
    assert diff.max() <= 3 and np.mean(diff) <= 0.5
    e = rel_l2(out, ref["out"])
    _say("  bf16 eps=%g out %.3e" % (eps, e))
    assert e <= TOL_BF16


def test_tolerance_zero_equals_fixed_steps_bitwise():
    x = W.forward_inputs(1, 2, 150, 128, 128, "bf16", 4.0, seed=63)
    d = to_device(x, "bf16")
    for prec in (L.MESA_PREC_BF16, L.MESA_PREC_F32):
        a = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], 15, 64, precision=prec)
        b = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], 15, 64, precision=prec,
                      eps=0.0, want_steps=True)
        torch.cuda.synchronize()
        assert torch.equal(a, b["out"]), prec
        assert int(b["steps"].max()) == 15


def test_decode_tolerance_matches_oracle():
    x = W.forward_inputs(3, 2, 1, 128, 128, "f32", 3.0, seed=64)
    rng = np.random.default_rng(64)
    H0, G0 = oracle.unrolled_states(rng.standard_normal((3, 2, 300, 128)) / 11,
                                    rng.standard_normal((3, 2, 300, 128)),
                                    np.full((3, 2, 300), 0.99), np.full((3, 2, 300), 0.5))
    H0, G0 = H0.astype(np.float32), G0.astype(np.float32)
    d = to_device({k: v[:, :, 0] for k, v in x.items() if k != "lam"}, "f32")
    lam = torch.from_numpy(x["lam"]).cuda()
    for eps in (0.0, 1e-3, 1e-5):
        dH, dG = torch.from_numpy(H0).cuda(), torch.from_numpy(G0).cuda()
        st = torch.zeros((3, 2), dtype=torch.int32, device="cuda")
        out = L.decode_step(dH, dG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], lam, 40, eps=eps,
                            steps_out=st)
        rst = np.zeros((3, 2), dtype=np.int32)
        ro, rH, rG = oracle.decode_step(H0, G0, x["q"][:, :, 0], x["k"][:, :, 0], x["v"][:, :, 0],
                                        x["gamma"][:, :, 0], x["beta"][:, :, 0], x["lam"], 40, eps=eps,
                                        steps_out=rst)
        got = st.cpu().numpy()
        _say("decode eps=%g steps gpu %s oracle %s" % (eps, got.ravel().tolist(), rst.ravel().tolist()))
        assert np.abs(got - rst).max() <= 1
        same = got == rst
        assert rel_l2(out.cpu().numpy()[same], ro[same]) <= TOL_F32
        assert rel_l2(dH.cpu().numpy(), rH) <= 1e-6 and rel_l2(dG.cpu().numpy(), rG) <= 1e-6


# ------------------------------------------------------ packed symmetric decode state
def _np_pack(H):
    """Cyclic diagonals of symmetric H [..., d, d]: HP[..., k, i] = H[..., i, (i + k) mod d]."""
    d = H.shape[-1]
    i = np.arange(d)
    return np.stack([H[..., i, (i + k) % d] for k in range(d // 2 + 1)], axis=-2)


@pytest.mark.parametrize("dk", [64, 128])
def test_pack_unpack_state_roundtrip(dk):
    rng = np.random.default_rng(dk)
    A = rng.standard_normal((3, 2, dk, dk)).astype(np.float32)
    H = (A + np.swapaxes(A, -1, -2)).astype(np.float32)   # exactly symmetric
    hp = L.pack_state(torch.from_numpy(H).cuda())
    back = L.unpack_state(hp)
    torch.cuda.synchronize()
    assert np.array_equal(hp.cpu().numpy(), _np_pack(H))
    assert np.array_equal(back.cpu().numpy(), H)


@pytest.mark.parametrize("dk,dv,dtype", [(128, 128, "bf16"), (64, 128, "f32"), (128, 64, "f32")])
def test_packed_decode_matches_full_layout_and_oracle(dk, dv, dtype):
    """Twelve steps on the packed state and on the full state from the same prefilled
    (symmetric) states: outputs agree to fp32 rounding, the unpacked state matches the
    full one, and both match the oracle's decode."""
    rng = np.random.default_rng(dk + dv)
    N, Hh = 5, 2
    H0, G0 = oracle.unrolled_states(rng.standard_normal((N, Hh, 200, dk)) / np.sqrt(dk),
                                    rng.standard_normal((N, Hh, 200, dv)),
                                    np.full((N, Hh, 200), 0.98), np.full((N, Hh, 200), 0.5))
    H0 = H0.astype(np.float32)
    H0 = np.triu(H0) + np.swapaxes(np.triu(H0, 1), -1, -2)   # exactly symmetric fp32
    G0 = G0.astype(np.float32)
    lam = W.forward_inputs(1, Hh, 1, dk, dv, "f32", 3.0, seed=1)["lam"]
    dlam = torch.from_numpy(lam).cuda()
    fH, fG = torch.from_numpy(H0).cuda(), torch.from_numpy(G0).cuda()
    pG = torch.from_numpy(G0).cuda()
    pH = L.pack_state(fH.clone())
    rH, rG = H0.astype(np.float64), G0.astype(np.float64)
    worst_fp, worst_or = 0.0, 0.0
    for step in range(12):
        x = W.forward_inputs(N, Hh, 1, dk, dv, dtype, 3.0, seed=100 + step)
        d = to_device({k: v[:, :, 0] for k, v in x.items() if k != "lam"}, dtype)
        of = L.decode_step(fH, fG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], dlam, 15)
        op = L.decode_step(pH, pG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], dlam, 15, packed=True)
        torch.cuda.synchronize()
        ro, rH, rG = oracle.decode_step(rH, rG, x["q"][:, :, 0], x["k"][:, :, 0], x["v"][:, :, 0],
                                        x["gamma"][:, :, 0], x["beta"][:, :, 0], lam, 15)
        worst_fp = max(worst_fp, rel_l2(op.cpu().numpy(), of.cpu().numpy()))
        worst_or = max(worst_or, rel_l2(op.cpu().numpy(), ro))
    _say("packed decode d_k=%d d_v=%d %s: vs full layout %.2e, vs oracle %.2e" % (dk, dv, dtype, worst_fp, worst_or))
    assert worst_fp <= 1e-5
    assert worst_or <= (TOL_BF16 if dtype == "bf16" else TOL_F32)
    full_from_packed = L.unpack_state(pH).cpu().numpy()
    assert rel_l2(full_from_packed, fH.cpu().numpy()) <= 1e-6
    assert rel_l2(full_from_packed, rH) <= 1e-6 and rel_l2(pG.cpu().numpy(), rG) <= 1e-6
    # the stored diagonals stay exactly those of a symmetric matrix
    assert np.array_equal(L.pack_state(torch.from_numpy(full_from_packed).cuda()).cpu().numpy()[:, :, :dk // 2],
                          pH.cpu().numpy()[:, :, :dk // 2])


def test_packed_decode_tolerance_counts():
    x = W.forward_inputs(3, 2, 1, 128, 128, "f32", 3.0, seed=65)
    rng = np.random.default_rng(65)
    H0, G0 = oracle.unrolled_states(rng.standard_normal((3, 2, 300, 128)) / 11,
                                    rng.standard_normal((3, 2, 300, 128)),
                                    np.full((3, 2, 300), 0.99), np.full((3, 2, 300), 0.5))
    H0 = H0.astype(np.float32)
    H0 = np.triu(H0) + np.swapaxes(np.triu(H0, 1), -1, -2)
    G0 = G0.astype(np.float32)
    d = to_device({k: v[:, :, 0] for k, v in x.items() if k != "lam"}, "f32")
    lam = torch.from_numpy(x["lam"]).cuda()
    pH = L.pack_state(torch.from_numpy(H0).cuda())
    pG = torch.from_numpy(G0).cuda()
    st = torch.zeros((3, 2), dtype=torch.int32, device="cuda")
    out = L.decode_step(pH, pG, d["q"], d["k"], d["v"], d["gamma"], d["beta"], lam, 40, eps=1e-4,
                        steps_out=st, packed=True)
    rst = np.zeros((3, 2), dtype=np.int32)
    ro, _, _ = oracle.decode_step(H0, G0, x["q"][:, :, 0], x["k"][:, :, 0], x["v"][:, :, 0], x["gamma"][:, :, 0],
                                  x["beta"][:, :, 0], x["lam"], 40, eps=1e-4, steps_out=rst)
    got = st.cpu().numpy()
    assert np.abs(got - rst).max() <= 1
    same = got == rst
    assert rel_l2(out.cpu().numpy()[same], ro[same]) <= TOL_F32
