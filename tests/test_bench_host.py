"""Host-side parts of bench.py: the algorithmic counts its roofline divides by, the traffic
record lookup, and the one-GPU guard.  CPU only; nothing here launches a kernel."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_cg_flops_per_token_head_at_the_1b_shape():
    # d_k = d_v = 128, chunk 64, 15 CG steps: 16 products of 2 d^2 + 2 (C+1) d flops, then the
    # read-out 2 d^2 + (C+1) 2d: 17 x 49408 = 839,936 flops per token-head
    per_th = 16 * (2 * 128 * 128 + 2 * 65 * 128) + 2 * 128 * 128 + 65 * 256
    assert per_th == 839936
    assert bench.cg_kernel_flops(1, 1, 1, 128, 128, 64, 15) == per_th
    # linear in the token-heads
    assert bench.cg_kernel_flops(8, 16, 2048, 128, 128, 64, 15) == 8 * 16 * 2048 * per_th


def test_state_bytes_at_the_1b_shape():
    # 128 sequences x 32 chunks of bf16 H and G (128 x 256 each) plus k, v read once
    states = 128 * 32 * 128 * 256 * 2
    inputs = 128 * 2048 * 256 * 2
    assert bench.state_kernel_bytes(8, 16, 2048, 128, 128, 64, 2, 2) == states + inputs == 402653184
    # a ragged last chunk still stores its entering state
    assert bench.state_kernel_bytes(1, 1, 65, 128, 128, 64, 2, 4) == 2 * 128 * 256 * 4 + 65 * 256 * 2


@pytest.mark.parametrize("kernel", ["chunk_cg_bf16", "chunk_cg_x3", "chunk_cg_f32"])
def test_traffic_record_is_used_only_for_the_sources_it_was_taken_on(kernel, monkeypatch):
    path = os.path.join(ROOT, "profiles", "%s_layer1b_traffic.json" % kernel)
    if not os.path.exists(path):
        pytest.skip("no traffic record for " + kernel)
    rec = json.load(open(path))
    monkeypatch.setattr(bench, "source_hash", lambda k: rec["kernel_source_sha256"])
    assert bench.traffic_entry(kernel) == rec["hbm_bytes_per_launch"]
    monkeypatch.setattr(bench, "source_hash", lambda k: "0" * 64)
    assert bench.traffic_entry(kernel) is None


def test_source_hash_covers_the_kernel_and_its_headers():
    h = bench.source_hash("chunk_cg_bf16")
    assert len(h) == 64 and h != bench.source_hash("chunk_cg_x3")


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU only" in res.stderr
    assert res.stdout == ""
