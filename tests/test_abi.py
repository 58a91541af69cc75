"""The C ABI on the host: the library loads, exports every entry point that
include/libmesa.h declares, and rejects bad arguments before any launch.

No test here reaches a kernel launch: every call fails validation, so the
suite runs without a GPU.  Fake device pointers are plain integers.
"""
import ctypes
import os
import re

import pytest

from paper_2506_05233_amd import libmesa as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "libmesa.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return L.load()


def _declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?(?:int|size_t|char\s*\*|const char\s*\*)\s*\**\s*(mesa_\w+)\s*\(",
                                 text, flags=re.M)))


def _declared_constants():
    text = open(HEADER).read()
    return {m.group(1): int(m.group(2)) for m in re.finditer(r"#define\s+(MESA_\w+)\s+(-?\d+)", text)}


def test_header_declares_the_expected_entry_points():
    assert _declared_functions() == sorted(L.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_binding_constants_match_header():
    for name, value in _declared_constants().items():
        assert getattr(L, name) == value, name


def test_status_strings(lib):
    for s in range(8):
        assert L.status_string(s) not in ("", "unknown status")
    assert L.status_string(99) == "unknown status"
    assert L.version() == 101


def test_workspace_bytes(lib):
    # states entering every chunk: H_c (d_k x d_k) and G_c^T (d_k x d_v), fp32
    assert L.forward_workspace_bytes(8, 16, 2048, 128, 128, 64) == 8 * 16 * 32 * 128 * 256 * 4
    assert L.forward_workspace_bytes(1, 2, 100, 64, 128, 32) == 2 * 4 * 64 * 192 * 4
    assert L.forward_workspace_bytes(1, 1, 0, 64, 64, 64) == 0
    assert L.forward_workspace_bytes(1, 1, 64, 96, 64, 64) == 0
    assert L.forward_workspace_bytes(1, 1, 64, 64, 64, 48) == 0
    # few long sequences: room for the segment totals of the segmented scan after the
    # states, min(B H floor(chunks / 8), 128) totals of d_k (d_k + d_v) floats, + 128 floats
    states = 16 * 256 * 128 * 256 * 4
    assert L.forward_workspace_bytes(1, 16, 16384, 128, 128, 64) == states + 128 * 128 * 256 * 4 + 512
    assert L.forward_workspace_bytes(1, 2, 17 * 64 + 13, 64, 128, 64) == 2 * 18 * 64 * 192 * 4 + 4 * 64 * 192 * 4 + 512
    assert L.forward_workspace_bytes(65, 1, 16 * 64, 128, 128, 64) == 65 * 16 * 128 * 256 * 4


# fake, non-overlapping device addresses
P = {n: 0x10000000 * (i + 1) for i, n in enumerate(
    ["q", "k", "v", "g", "b", "lam", "out", "qs", "fh", "fg", "ws", "H", "G", "st", "dl"])}


def _fwd(lib, **kw):
    a = dict(q=P["q"], k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"], lam=P["lam"], B=2, H=3, T=128,
             dk=64, dv=64, dtype=0, n_cg=5, chunk=64, prec=0, out=P["out"], qstar=None, fH=None,
             fG=None, ws=P["ws"], ws_bytes=1 << 40)
    a.update(kw)
    return lib.mesa_forward_ex(a["q"], a["k"], a["v"], a["gamma"], a["beta"], a["lam"], a["B"],
                               a["H"], a["T"], a["dk"], a["dv"], a["dtype"], a["n_cg"], a["chunk"],
                               a["prec"], a["out"], a["qstar"], a["fH"], a["fG"], a["ws"],
                               a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), L.MESA_ERR_NULL),
    (dict(k=None), L.MESA_ERR_NULL),
    (dict(lam=None), L.MESA_ERR_NULL),
    (dict(ws=None), L.MESA_ERR_NULL),
    (dict(B=-1), L.MESA_ERR_SHAPE),
    (dict(T=-5), L.MESA_ERR_SHAPE),
    (dict(dk=96), L.MESA_ERR_UNSUPPORTED),
    (dict(dv=32), L.MESA_ERR_UNSUPPORTED),
    (dict(chunk=48), L.MESA_ERR_UNSUPPORTED),
    (dict(chunk=128), L.MESA_ERR_UNSUPPORTED),
    (dict(dtype=2), L.MESA_ERR_UNSUPPORTED),
    (dict(prec=7), L.MESA_ERR_UNSUPPORTED),
    (dict(prec=L.MESA_PREC_BF16X3), L.MESA_ERR_UNSUPPORTED),               # split operands need bf16 inputs
    (dict(prec=L.MESA_PREC_BF16X3, dtype=1, chunk=32), L.MESA_ERR_UNSUPPORTED),  # ... and chunk 64
    (dict(n_cg=-1), L.MESA_ERR_ARG),
    (dict(n_cg=L.MESA_MAX_NCG + 1), L.MESA_ERR_ARG),
    (dict(ws_bytes=100), L.MESA_ERR_WORKSPACE),
    (dict(prec=L.MESA_PREC_BF16X3, dtype=1, ws_bytes=100), L.MESA_ERR_WORKSPACE),
    (dict(out=P["q"] + 64), L.MESA_ERR_ARG),          # out overlaps q
    (dict(k=P["k"] + 2), L.MESA_ERR_ARG),             # k not 16-byte aligned
    (dict(ws=P["ws"] + 8), L.MESA_ERR_ARG),           # workspace not 16-byte aligned
    (dict(out=P["ws"]), L.MESA_ERR_ARG),               # out overlaps the workspace
    (dict(qstar=P["out"]), L.MESA_ERR_ARG),            # two outputs overlap
    (dict(out=None, fH=P["fh"], fG=None), L.MESA_ERR_NULL),    # states only needs both states
    (dict(out=None, fH=P["fh"], fG=P["fg"], qstar=P["qs"]), L.MESA_ERR_NULL),
    (dict(out=None, fH=P["fh"], fG=P["fg"], ws_bytes=100), L.MESA_ERR_WORKSPACE),  # states only, scratch too small
    (dict(out=None, fH=P["ws"] + 256, fG=P["fg"]), L.MESA_ERR_ARG),  # states only, scratch overlaps final_H
])
def test_forward_rejects_bad_arguments(lib, kw, status):
    assert _fwd(lib, **kw) == status


def test_forward_empty_batch_is_a_noop(lib):
    assert _fwd(lib, B=0) == L.MESA_OK
    assert _fwd(lib, H=0, q=None) == L.MESA_OK


def test_plain_forward_requires_out(lib):
    assert lib.mesa_forward(P["q"], P["k"], P["v"], P["g"], P["b"], P["lam"], 1, 1, 64, 64, 64, 0, 3,
                            64, None, P["ws"], 1 << 30, None) == L.MESA_ERR_NULL


def _fwd_tol(lib, **kw):
    a = dict(q=P["q"], k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"], lam=P["lam"], B=2, H=3, T=128,
             dk=64, dv=64, dtype=0, n_cg=30, eps=1e-4, chunk=64, prec=0, out=P["out"], qstar=None,
             steps=P["st"], ws=P["ws"], ws_bytes=1 << 40)
    a.update(kw)
    return lib.mesa_forward_tol(a["q"], a["k"], a["v"], a["gamma"], a["beta"], a["lam"], a["B"],
                                a["H"], a["T"], a["dk"], a["dv"], a["dtype"], a["n_cg"], a["eps"],
                                a["chunk"], a["prec"], a["out"], a["qstar"], a["steps"], a["ws"],
                                a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(eps=-1e-3), L.MESA_ERR_ARG),
    (dict(eps=float("nan")), L.MESA_ERR_ARG),
    (dict(eps=float("inf")), L.MESA_ERR_ARG),
    (dict(out=None), L.MESA_ERR_NULL),
    (dict(n_cg=L.MESA_MAX_NCG + 1), L.MESA_ERR_ARG),
    (dict(steps=P["st"] + 2), L.MESA_ERR_ARG),        # steps not 4-byte aligned
    (dict(steps=P["q"] + 16), L.MESA_ERR_ARG),        # steps overlaps q
    (dict(steps=P["out"] + 64), L.MESA_ERR_ARG),      # steps overlaps out
    (dict(dk=96), L.MESA_ERR_UNSUPPORTED),
    (dict(ws_bytes=16), L.MESA_ERR_WORKSPACE),
])
def test_forward_tol_rejects_bad_arguments(lib, kw, status):
    assert _fwd_tol(lib, **kw) == status


def test_forward_tol_empty_batch_is_a_noop(lib):
    assert _fwd_tol(lib, B=0) == L.MESA_OK


def _dec_tol(lib, **kw):
    a = dict(H=P["H"], G=P["G"], q=P["q"], k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"],
             lam=P["lam"], N=4, Hh=2, dk=128, dv=128, dtype=1, n_cg=30, eps=1e-4, out=P["out"],
             steps=P["st"])
    a.update(kw)
    return lib.mesa_decode_step_tol(a["H"], a["G"], a["q"], a["k"], a["v"], a["gamma"], a["beta"],
                                    a["lam"], a["N"], a["Hh"], a["dk"], a["dv"], a["dtype"], a["n_cg"],
                                    a["eps"], a["out"], a["steps"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(eps=-0.5), L.MESA_ERR_ARG),
    (dict(eps=float("nan")), L.MESA_ERR_ARG),
    (dict(steps=P["st"] + 1), L.MESA_ERR_ARG),
    (dict(steps=P["H"] + 4), L.MESA_ERR_ARG),         # steps overlaps the H state
    (dict(steps=P["g"]), L.MESA_ERR_ARG),             # steps overlaps gamma
    (dict(out=None), L.MESA_ERR_NULL),
    (dict(n_cg=-1), L.MESA_ERR_ARG),
])
def test_decode_tol_rejects_bad_arguments(lib, kw, status):
    assert _dec_tol(lib, **kw) == status


def test_decode_tol_empty_is_a_noop(lib):
    assert _dec_tol(lib, N=0) == L.MESA_OK


def _dec(lib, **kw):
    a = dict(H=P["H"], G=P["G"], q=P["q"], k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"],
             lam=P["lam"], N=4, Hh=2, dk=128, dv=128, dtype=1, n_cg=15, out=P["out"])
    a.update(kw)
    return lib.mesa_decode_step(a["H"], a["G"], a["q"], a["k"], a["v"], a["gamma"], a["beta"],
                                a["lam"], a["N"], a["Hh"], a["dk"], a["dv"], a["dtype"], a["n_cg"],
                                a["out"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=None), L.MESA_ERR_NULL),
    (dict(out=None), L.MESA_ERR_NULL),
    (dict(lam=None), L.MESA_ERR_NULL),
    (dict(N=-2), L.MESA_ERR_SHAPE),
    (dict(dk=256), L.MESA_ERR_UNSUPPORTED),
    (dict(dtype=5), L.MESA_ERR_UNSUPPORTED),
    (dict(n_cg=-3), L.MESA_ERR_ARG),
    (dict(out=P["q"]), L.MESA_ERR_ARG),
    (dict(G=P["H"] + 1024), L.MESA_ERR_ARG),
])
def test_decode_rejects_bad_arguments(lib, kw, status):
    assert _dec(lib, **kw) == status


def test_decode_empty_is_a_noop(lib):
    assert _dec(lib, N=0) == L.MESA_OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        L.load()


def _bwd(lib, **kw):
    a = dict(k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"], lam=P["lam"], B=2, H=3, T=128, dk=64, dv=64,
             dtype=0, n_cg=10, prec=0, qs=P["qs"], dout=P["out"], dq=P["fh"], dk_=P["fg"], dv_=P["H"], dg=P["G"],
             db=P["st"], dl=P["dl"], ws=P["ws"], ws_bytes=1 << 40)
    a.update(kw)
    return lib.mesa_backward(a["k"], a["v"], a["gamma"], a["beta"], a["lam"], a["B"], a["H"], a["T"], a["dk"],
                             a["dv"], a["dtype"], a["n_cg"], a["prec"], a["qs"], a["dout"], a["dq"], a["dk_"], a["dv_"],
                             a["dg"], a["db"], a["dl"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(qs=None), L.MESA_ERR_NULL),
    (dict(dout=None), L.MESA_ERR_NULL),
    (dict(dl=None), L.MESA_ERR_NULL),
    (dict(ws=None), L.MESA_ERR_NULL),
    (dict(dk=96), L.MESA_ERR_UNSUPPORTED),
    (dict(n_cg=-1), L.MESA_ERR_ARG),
    (dict(prec=5), L.MESA_ERR_UNSUPPORTED),
    (dict(prec=L.MESA_PREC_BF16), L.MESA_ERR_UNSUPPORTED),  # fp32 inputs have no matrix-core solve
    (dict(T=-1), L.MESA_ERR_SHAPE),
    (dict(ws_bytes=64), L.MESA_ERR_WORKSPACE),
    (dict(qs=P["qs"] + 4), L.MESA_ERR_ARG),          # q* not 16-byte aligned
    (dict(k=P["k"] + 2), L.MESA_ERR_ARG),            # k not 16-byte aligned
    (dict(dq=P["fh"] + 8), L.MESA_ERR_ARG),          # dq not 16-byte aligned
    (dict(dq=P["k"] + 64), L.MESA_ERR_ARG),          # dq overlaps k
    (dict(db=P["fh"] + 8), L.MESA_ERR_ARG),          # two gradients overlap
    (dict(dl=P["ws"] + 4096), L.MESA_ERR_ARG),       # dlambda inside the workspace
])
def test_backward_rejects_bad_arguments(lib, kw, status):
    assert _bwd(lib, **kw) == status


def test_backward_workspace_size(lib):
    # fp32: H_c, G_c, S^H, A^G per 64-token chunk, u per token, dLambda parts per chunk;
    # bf16: H_c, G_c fragments per chunk, u per token
    B, H, T, dk, dv = 2, 3, 130, 64, 128
    nc = 3
    want = 4 * (2 * B * H * nc * dk * (dk + dv) + B * H * T * dk + B * H * nc * dk)
    want += 2 * (B * H * nc * dk * (dk + dv) + B * H * T * dk)
    assert lib.mesa_backward_workspace_bytes(B, H, T, dk, dv) == want
    assert lib.mesa_backward_workspace_bytes(B, H, 0, dk, dv) == 0
    assert _bwd(lib, B=0) == L.MESA_OK


def test_packed_state_entry_points_reject_bad_arguments(lib):
    assert lib.mesa_pack_state(None, P["H"], 2, 2, 128, None) == L.MESA_ERR_NULL
    assert lib.mesa_pack_state(P["H"], P["H"] + 64, 2, 2, 128, None) == L.MESA_ERR_ARG   # overlap
    assert lib.mesa_unpack_state(P["H"], P["G"], 2, 2, 96, None) == L.MESA_ERR_UNSUPPORTED
    assert lib.mesa_unpack_state(P["H"], P["G"], -1, 2, 64, None) == L.MESA_ERR_SHAPE
    assert lib.mesa_pack_state(P["H"], P["G"], 0, 2, 64, None) == L.MESA_OK
    args = [P["H"], P["G"], P["q"], P["k"], P["v"], P["g"], P["b"], P["lam"], 4, 2, 128, 128, 1, 15]
    assert lib.mesa_decode_step_packed(*args[:8], 4, 2, 128, 128, 1, 15, -1.0, P["out"], None, None) == L.MESA_ERR_ARG
    assert lib.mesa_decode_step_packed(None, *args[1:], 0.0, P["out"], None, None) == L.MESA_ERR_NULL
    # the packed H of 8 pairs spans 8 * 65 * 128 floats: an output inside that extent overlaps
    assert lib.mesa_decode_step_packed(*args, 0.0, P["H"] + 8 * 65 * 128 * 4 - 4, None, None) == L.MESA_ERR_ARG


def _noalloc(lib, **kw):
    a = dict(q=P["q"], k=P["k"], v=P["v"], gamma=P["g"], beta=P["b"], lam=P["lam"], B=2, H=3, T=128,
             dk=64, dv=64, dtype=0, n_cg=5, chunk=64, out=P["out"])
    a.update(kw)
    return lib.mesa_forward_noalloc(a["q"], a["k"], a["v"], a["gamma"], a["beta"], a["lam"], a["B"], a["H"],
                                    a["T"], a["dk"], a["dv"], a["dtype"], a["n_cg"], a["chunk"], a["out"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(out=None), L.MESA_ERR_NULL),
    (dict(q=None), L.MESA_ERR_NULL),
    (dict(dk=96), L.MESA_ERR_UNSUPPORTED),
    (dict(chunk=48), L.MESA_ERR_UNSUPPORTED),
    (dict(n_cg=1025), L.MESA_ERR_ARG),
    (dict(out=P["k"] + 16), L.MESA_ERR_ARG),          # out overlaps k
    (dict(B=0), L.MESA_OK),                           # nothing to do, nothing touched
    # more than MESA_NOALLOC_SCRATCH_BYTES of chunk states: 513 sequence-chunks at d = 128
    (dict(B=1, H=1, T=513 * 64, dk=128, dv=128), L.MESA_ERR_WORKSPACE),
    (dict(B=8, H=16, T=2048, dk=128, dv=128, dtype=1), L.MESA_ERR_WORKSPACE),
])
def test_noalloc_forward_rejects_before_touching_the_device(lib, kw, status):
    """Every check of mesa_forward_noalloc, the buffer size included, runs before the
    library looks up its device buffer: these calls need no GPU."""
    assert _noalloc(lib, **kw) == status


def test_noalloc_buffer_size_constant():
    assert L.MESA_NOALLOC_SCRATCH_BYTES == 64 << 20
    # exactly the buffer: 512 sequence-chunks of fp32 H_c and G_c at d_k = d_v = 128
    assert L.forward_workspace_bytes(4, 16, 512, 128, 128, 64) == L.MESA_NOALLOC_SCRATCH_BYTES


def _front(lib, **kw):
    a = dict(qp=P["q"], kp=P["k"], vp=P["v"], cq=P["g"], ck=P["b"], cv=None, ag=P["lam"], ab=P["H"],
             th=P["G"], cap=0.9975, eps=1e-6, B=2, H=3, T=100, dk=128, dv=64, dtype=1, q=P["out"], k=P["qs"],
             v=P["fh"], gam=P["fg"], bet=P["ws"], lam=P["st"])
    a.update(kw)
    return lib.mesa_frontend(a["qp"], a["kp"], a["vp"], a["cq"], a["ck"], a["cv"], a["ag"], a["ab"], a["th"],
                             a["cap"], a["eps"], a["B"], a["H"], a["T"], a["dk"], a["dv"], a["dtype"], a["q"],
                             a["k"], a["v"], a["gam"], a["bet"], a["lam"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(qp=None), L.MESA_ERR_NULL),
    (dict(th=None), L.MESA_ERR_NULL),
    (dict(lam=None, T=0), L.MESA_ERR_NULL),          # Lambda is written even without tokens
    (dict(dk=96), L.MESA_ERR_UNSUPPORTED),
    (dict(dtype=5), L.MESA_ERR_UNSUPPORTED),
    (dict(B=-1), L.MESA_ERR_SHAPE),
    (dict(cap=1.5), L.MESA_ERR_ARG),
    (dict(cap=float("nan")), L.MESA_ERR_ARG),
    (dict(eps=-1.0), L.MESA_ERR_ARG),
    (dict(qp=P["q"] + 1), L.MESA_ERR_ARG),            # projections move in 16-byte pieces
    (dict(vp=P["v"] + 8), L.MESA_ERR_ARG),
    (dict(v=P["fh"] + 8), L.MESA_ERR_ARG),
    (dict(ck=P["b"] + 4), L.MESA_ERR_ARG),            # so do the filter rows
    (dict(ag=P["lam"] + 2), L.MESA_ERR_ARG),          # gate projections: 4-byte alignment
    (dict(q=P["k"] + 64), L.MESA_ERR_ARG),            # output overlaps an input
    (dict(k=P["out"] + 64), L.MESA_ERR_ARG),          # two outputs overlap
    (dict(H=0), L.MESA_OK),
])
def test_frontend_rejects_bad_arguments(lib, kw, status):
    assert _front(lib, **kw) == status


def test_output_norm_rejects_bad_arguments(lib):
    f = lib.mesa_output_norm
    assert f(None, P["lam"], 1e-6, 1, 2, 10, 128, 1, P["out"], None) == L.MESA_ERR_NULL
    assert f(P["q"], P["lam"], -1e-6, 1, 2, 10, 128, 1, P["out"], None) == L.MESA_ERR_ARG
    assert f(P["q"], P["lam"], 1e-6, 1, 2, 10, 96, 1, P["out"], None) == L.MESA_ERR_UNSUPPORTED
    assert f(P["q"], P["lam"], 1e-6, 1, 2, 10, 128, 3, P["out"], None) == L.MESA_ERR_UNSUPPORTED
    assert f(P["q"], P["lam"], 1e-6, 1, 2, 10, 128, 1, P["q"] + 64, None) == L.MESA_ERR_ARG
    assert f(P["q"], P["lam"], 1e-6, 0, 2, 10, 128, 1, P["out"], None) == L.MESA_OK
    assert f(P["q"] + 4, P["lam"], 1e-6, 1, 2, 10, 128, 1, P["out"], None) == L.MESA_ERR_ARG
    assert f(P["q"], P["lam"] + 4, 1e-6, 1, 2, 10, 128, 1, P["out"], None) == L.MESA_ERR_ARG
    assert f(P["q"], P["lam"], 1e-6, 1, 2, 10, 128, 1, P["out"] + 8, None) == L.MESA_ERR_ARG
