"""Register and scratch use of every libmesa kernel, from the compiler's resource report.

The kernels are built to hold their working sets in registers: a spilled register goes
to scratch memory, and reloading it waits on the vector memory counter, which also
covers every load in flight (one such case, 64-bit tile addresses held across the
phases of the backward gradient kernel, cost 12% of that kernel).  These tests
recompile each source for gfx950 with the library's own flags and read the compiler's
resource remarks: no kernel may use scratch memory beyond the few known, measured cases
below, and none may exceed the register file.  CPU only (hipcc cross-compiles).
"""
import concurrent.futures
import os
import re
import shutil
import subprocess

import pytest

from paper_2506_05233_amd import build as B

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Kernels whose small spills were measured and left: (name pattern, maximum scratch bytes
# per lane).  The split-operand CG keeps one or two values of its chunk set-up in a spill
# slot (reloaded once per chunk, outside the CG loop); the state scan's fp32-plain-state
# variant (the backward's state pass) spills a few values that are reloaded off its
# critical path (removing them by other address forms made the kernel slower).
KNOWN_SPILLS = [
    (r"chunk_cg_x3_kernel<128, (64|128), true>", 16),
    (r"chunk_state_wide_kernel<128, (64|128), true, true, true, false>", 48),
]


def _demangler():
    for c in ("/opt/rocm/llvm/bin/llvm-cxxfilt", shutil.which("llvm-cxxfilt"), shutil.which("c++filt")):
        if c and os.path.exists(c):
            return c
    return None


def _demangle(names):
    out = subprocess.run([_demangler()], input="\n".join(names), capture_output=True, text=True,
                         check=True).stdout.splitlines()
    return dict(zip(names, out))


def _report(src):
    """Resource remarks of one source: {mangled kernel name: {field: value}}."""
    cmd = [HIPCC] + B.HIPCC_FLAGS + B.EXTRA_FLAGS.get(os.path.basename(src), []) + [
        "--cuda-device-only", "-Rpass-analysis=kernel-resource-usage", "-c", "-o", os.devnull, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    kernels, cur = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+(VGPRs|AGPRs|VGPRs Spill|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)",
                      line)
        if m and cur is not None:
            cur[m.group(1)] = int(m.group(2))
    return kernels


@pytest.fixture(scope="module")
def reports():
    if not os.path.exists(HIPCC) or _demangler() is None:
        pytest.skip("hipcc or a C++ demangler is not available")
    srcs = B.sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(len(srcs), 8)) as ex:
        reps = list(ex.map(_report, srcs))
    merged = {}
    for r in reps:
        merged.update(r)
    names = _demangle(sorted(merged))
    return {names[k]: v for k, v in merged.items()}


def test_every_source_reports_its_kernels(reports):
    kinds = ["chunk_cg_bf16_kernel", "chunk_cg_x3_kernel", "chunk_cg_f32_mma_kernel", "chunk_state_wide_kernel",
             "decode_step_kernel", "bwd_grad_kernel", "bwd_adjoint_kernel", "bwd_rhs_kernel", "frontend_kernel",
             "output_norm_kernel"]
    for k in kinds:
        assert any(k in name for name in reports), k


def test_no_kernel_uses_scratch_beyond_the_known_cases(reports):
    bad = []
    for name, r in sorted(reports.items()):
        scratch = r.get("ScratchSize [bytes/lane]", 0)
        if scratch == 0:
            continue
        allowed = next((lim for pat, lim in KNOWN_SPILLS if re.search(pat, name)), 0)
        if scratch > allowed:
            bad.append("%s: %d bytes/lane of scratch (%d spilled VGPRs)" % (name, scratch, r.get("VGPRs Spill", 0)))
    assert not bad, "\n".join(bad)


def test_hot_kernels_have_no_spills(reports):
    # the kernels every benchmark step runs, at d = 128
    hot = [r"chunk_cg_bf16_kernel<128, 128, (true|false)>", r"chunk_state_wide_kernel<128, 128, true, false, false, false>",
           r"bwd_grad_kernel<mesa::bf16_t, 128, 128>", r"bwd_adjoint_kernel<128, 128, true>",
           r"bwd_rhs_kernel<mesa::bf16_t, 128, 128>", r"decode_step_kernel<mesa::bf16_t, 128, 128, (true|false)>"]
    for pat in hot:
        found = [(n, r) for n, r in reports.items() if re.search(pat, n)]
        assert found, pat
        for n, r in found:
            assert r.get("VGPRs Spill", 0) == 0 and r.get("ScratchSize [bytes/lane]", 0) == 0, n


def test_registers_fit_the_occupancy_each_kernel_is_built_for(reports):
    # every kernel compiles to at least one wave per SIMD with at most 512 registers per lane
    for name, r in reports.items():
        assert r.get("VGPRs", 0) <= 512 and r.get("AGPRs", 0) <= 256, name
        assert r.get("Occupancy [waves/SIMD]", 1) >= 1, name
