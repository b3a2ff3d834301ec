"""Host logic of bench.py (no GPU): the algorithmic byte count behind every bandwidth and roofline
figure, and the one-GPU contract.

The byte counts are pinned to figures derived independently from the model shapes: every weight
of the verify layers read once, plus the frozen head, plus keys and values of the verify layers
over the average context (prompt + half the new tokens), plus the logits written.
"""
import os
import subprocess
import sys

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _verify_bytes(shape, batch, ctx, k_spec):
    layers = shape.n_layers - shape.split_k
    es = 2
    weights = layers * shape.layer_params() * es + shape.vocab * shape.d_model * es
    # keys and values of every verify layer at positions 0..ctx+k_spec-1
    kv_per_token_layer = shape.n_kv_heads * shape.head_dim * 2 * es
    kv = batch * layers * (ctx + k_spec) * kv_per_token_layer
    logits = batch * k_spec * shape.vocab * 4
    return weights + kv + logits


@pytest.mark.parametrize("shape,batch,prompt,new,k_spec,approx_gb", [
    (synth.SHAPE_7B, 1, 512, 512, 4, 6.94),      # 7B shape, batch 1
    (synth.SHAPE_7B, 8, 2048, 256, 8, 11.32),    # 7B shape, batch 8, long prompts
    (synth.SHAPE_13B, 1, 1024, 512, 6, 13.54),   # 13B shape
])
def test_verify_bytes_match_the_shape_arithmetic(shape, batch, prompt, new, k_spec, approx_gb):
    ctx = prompt + new // 2
    got = bench.algorithmic_bytes(shape, shape.n_layers - shape.split_k, k_spec, [ctx] * batch, batch * k_spec)
    assert got == _verify_bytes(shape, batch, ctx, k_spec)
    assert abs(got / 1e9 - approx_gb) / approx_gb < 0.01


def test_layer_params_of_the_7b_shape():
    # q, k, v, o (4 d^2 with MHA), gate, up, down (3 d F), two norm gains (2 d)
    s = synth.SHAPE_7B
    assert s.layer_params() == 4 * 4096 * 4096 + 3 * 4096 * 11008 + 2 * 4096 == 202383360


def test_draft_pass_counts_the_lora_factors():
    s = synth.SHAPE_13B
    plain = bench.algorithmic_bytes(s, s.split_k, 1, [1024], 1)
    lora = bench.algorithmic_bytes(s, s.split_k, 1, [1024], 1, lora=True)
    assert lora - plain == (s.vocab * s.lora_rank + s.lora_rank * s.d_model) * 4


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_profile_is_used_only_for_its_sources_and_workload(tmp_path, monkeypatch):
    # a counter summary names the kernel sources' SHA-256, the workload and k_spec it was taken
    # with; bench.py takes its traffic figure only when all three match
    prof = tmp_path / "traffic.md"
    prof.write_text("- `kernel_sources_sha256`: `abc`\n- `workload`: `7b`\n- `k_spec`: `4`\n"
                    "- `traffic_bytes_per_launch`: `181040071`\n")
    monkeypatch.setattr(bench, "TRAFFIC_PROFILES", {"gate_up": str(prof)})
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: "abc")
    assert bench.measured_traffic("gate_up", "7b", 4) == 181040071
    assert bench.measured_traffic("gate_up", "7b", 6) is None
    assert bench.measured_traffic("gate_up", "13b", 4) is None
    assert bench.measured_traffic("qkv", "7b", 4) is None
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: "def")
    assert bench.measured_traffic("gate_up", "7b", 4) is None


def test_kernel_sources_hash_covers_both_device_files():
    assert len(bench.KERNEL_SOURCES) == 2
    assert all(os.path.exists(os.path.join(ROOT, f)) for f in bench.KERNEL_SOURCES)
    assert len(bench.kernel_sources_sha256()) == 64
