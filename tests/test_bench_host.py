"""Host-side logic of bench.py, on the CPU: the one-GPU refusal, the
source-hash lookup of committed counter summaries, and the oracle's CPU
baseline on the small fp32 matmul workload."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2401_11202_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "error" in line and line["n_gpus"] == 2


def test_roles_map_to_the_files_their_kernels_come_from():
    assert "attention_bwd.hip" in bench.role_sources("attn.bwd")
    assert "attention.hip" in bench.role_sources("attn.core")
    assert "attention.hip" in bench.role_sources("attn.combine")
    assert "elementwise.hip" in bench.role_sources("rmsnorm")
    assert "backward.hip" in bench.role_sources("mlp.bwd.act")
    # every other role is a bf16 GEMM
    assert "gemm_bf16.hip" in bench.role_sources("mlp.up")
    assert "gemm_bf16.hip" in bench.role_sources("attn.qkv.fixup")
    assert bench.kernel_source_hash("mlp.up") == bench.kernel_source_hash("attn.out")
    assert bench.kernel_source_hash("mlp.up") != bench.kernel_source_hash("attn.core")


def test_profile_values_are_read_only_while_the_sources_match(tmp_path):
    h = bench.kernel_source_hash("mlp.up")
    good = tmp_path / "good.md"
    good.write_text(f"mfma_busy mlp.up: 0.7123\nkernel_source_sha256 mlp.up: {h}\n")
    assert bench._profile_value(str(good), "mfma_busy", "mlp.up") == pytest.approx(0.7123)
    stale = tmp_path / "stale.md"
    stale.write_text("mfma_busy mlp.up: 0.7123\nkernel_source_sha256 mlp.up: " + "0" * 64 + "\n")
    assert bench._profile_value(str(stale), "mfma_busy", "mlp.up") is None
    assert bench._profile_value(str(tmp_path / "missing.md"), "mfma_busy", "mlp.up") is None
    # another role's line does not answer for this one
    assert bench._profile_value(str(good), "mfma_busy", "mlp.down") is None


def test_committed_profiles_match_the_headline_kernels():
    """The default workload's counter summaries were taken on the kernels in
    this tree (regenerate profiles/ after changing a GEMM source)."""
    for role in ("mlp.up", "mlp.down"):
        assert bench.mfma_busy_from_profile("mlp_batch_x_megatron", role) is not None, role
        assert bench.traffic_from_profile("mlp_batch_x_megatron", role) is not None, role


def test_cpu_baseline_on_the_small_matmul_states_its_host():
    w = W.WORKLOADS["matmul_f32_sumK"]
    r = bench.cpu_baseline(w, W.make_inputs(w), 0.2)
    assert r["kind"] == "oracle" and r["unit"] == "TFLOP/s" and r["value"] > 0
    assert r["cores"] >= 1 and r["affinity_cores"] >= 1
    assert isinstance(r["sample"], str) and r["sample"]
    assert r["extrapolated_full_output_s"] >= 0 and "extrapolation" in r
