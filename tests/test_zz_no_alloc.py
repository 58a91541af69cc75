"""mesa_forward_noalloc: the forward with the chunk states in the library's own
fixed device buffer, for callers that cannot allocate.  Called through the C ABI
and checked against mesa_forward (same kernels, so bit for bit) on two calls in a
row, the second with a smaller input, and against the oracle on the small one."""
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


def _both(x, dtype, n_cg, chunk):
    d = to_device(x, dtype)
    a = L.forward_noalloc(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], n_cg, chunk)
    b = L.forward(d["q"], d["k"], d["v"], d["gamma"], d["beta"], d["lam"], n_cg, chunk)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


def test_noalloc_forward_matches_forward_twice_then_smaller():
    # 1: bf16, d = 128, 4 x 16 sequences of 4 chunks (the segmented scan does not
    #    apply: 64 sequences); 512 sequence-chunks, the buffer's limit at d = 128
    x1 = W.forward_inputs(4, 16, 8 * 64, 128, 128, "bf16", 4.0, seed=501)
    assert L.forward_workspace_bytes(4, 16, 8 * 64, 128, 128, 64) == L.MESA_NOALLOC_SCRATCH_BYTES
    a1, b1 = _both(x1, "bf16", 15, 64)
    print("noalloc call 1: equal %s" % np.array_equal(a1, b1), flush=True)
    assert np.array_equal(a1, b1)
    # 2: smaller: two sequences of 18 chunks (the segmented scan: segment totals in the
    #    buffer's second half), ragged tail; against the oracle too
    x2 = W.forward_inputs(1, 2, 17 * 64 + 13, 128, 128, "bf16", 4.0, seed=502)
    a2, b2 = _both(x2, "bf16", 15, 64)
    ref = oracle.forward(x2["q"], x2["k"], x2["v"], x2["gamma"], x2["beta"], x2["lam"], 15)["out"]
    e = rel_l2(a2, ref)
    print("noalloc call 2: equal %s, vs oracle %.3e" % (np.array_equal(a2, b2), e), flush=True)
    assert np.array_equal(a2, b2) and e <= TOL_BF16
    # 3: fp32 inputs, chunk 32 (fp32 states in the buffer)
    x3 = W.forward_inputs(2, 2, 100, 64, 64, "f32", 3.0, seed=503)
    a3, b3 = _both(x3, "f32", 10, 32)
    ref3 = oracle.forward(x3["q"], x3["k"], x3["v"], x3["gamma"], x3["beta"], x3["lam"], 10)["out"]
    assert np.array_equal(a3, b3) and rel_l2(a3, ref3) <= TOL_F32


def test_noalloc_rejects_shapes_beyond_the_buffer():
    x = W.forward_inputs(1, 1, 1, 128, 128, "bf16", 4.0, seed=504)
    d = to_device(x, "bf16")
    # 513 sequence-chunks at d = 128 need more than the buffer: rejected before any launch
    T = 513 * 64
    q = torch.zeros((1, 1, T, 128), dtype=torch.bfloat16, device="cuda")
    g = torch.ones((1, 1, T), dtype=torch.float32, device="cuda")
    with pytest.raises(L.MesaError) as e:
        L.forward_noalloc(q, q.clone(), q.clone(), g, g.clone(), d["lam"], 15, 64)
    assert e.value.status == L.MESA_ERR_WORKSPACE
