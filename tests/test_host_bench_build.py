"""Host logic of the build script and of bench.py (no GPU): the compiler-output
filter and spill detection of the build, the benchmark's mirror of the GEMM
engine's kernel choice for the step's shapes, the HBM-traffic record lookup
and its source digest, and the one-GPU guard."""
import importlib.util
import os
import shutil
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the package's build script as a module of its own (importing the package
# would load the library)
_spec = importlib.util.spec_from_file_location("mdnn_build_script",
                                               os.path.join(ROOT, "paper_2011_11188_amd", "build.py"))
build = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(build)

R = build.RESOURCE_REMARK


def test_diagnostics_drop_resource_remarks_with_their_context():
    lines = [
        "In file included from a.hip:6:",
        f"k.h:555:1: remark: k: VGPRs: 128 [-Rpass-analysis={R}]",
        "  555 | kernel(int x) {",
        "      | ^",
        "warning: unknown target feature 'packed-fp32-ops'",
        "In file included from b.hip:2:",
        "w.h:7:3: warning: unused variable 'q'",
        "    7 |   int q;",
        "      |       ^",
        "",
    ]
    assert build._diagnostics(lines) == [
        "In file included from b.hip:2:", "w.h:7:3: warning: unused variable 'q'", "    7 |   int q;",
        "      |       ^"]


def test_spills_report_only_vector_register_spills():
    lines = [
        f"x.hip:1:1: remark: Function Name: kern_a [-Rpass-analysis={R}]",
        f"x.hip:1:1: remark:     SGPRs Spill: 4 [-Rpass-analysis={R}]",
        f"x.hip:1:1: remark:     VGPRs Spill: 0 [-Rpass-analysis={R}]",
        f"x.hip:9:1: remark: Function Name: kern_b [-Rpass-analysis={R}]",
        f"x.hip:9:1: remark:     VGPRs Spill: 12 [-Rpass-analysis={R}]",
    ]
    assert build._spills(lines) == ["kern_b: VGPRs Spill: 12"]


@pytest.mark.parametrize("shape,kernel", [
    (("NN", 4096, 4096, 4096), "gemm_lds_kernel (256x256 direct-to-LDS pipeline)"),
    (("NN", 4096, 4096, 1024), "gemm_lds_kernel (256x256 direct-to-LDS pipeline)"),
    (("TN", 1024, 4096, 4096), "gemm_lds_kernel (128x128 direct-to-LDS pipeline with 3 stages)"),
    (("NN", 4096, 1, 4096), "skinny rows kernel"),
    (("TN", 4096, 1, 4096), "skinny cols kernel"),
    (("NT", 4096, 4096, 1), "skinny depth kernel"),
    (("NN", 100, 136, 100), "gemm_mfma_kernel 64x64"),
    (("NT", 1024, 1024, 1024), "gemm_lds_kernel (64x64 direct-to-LDS pipeline)"),
])
def test_kernel_choice_for_the_step_shapes(shape, kernel):
    assert bench._kernel_choice(*shape) == kernel


def test_traffic_record_lookup(monkeypatch):
    """The committed record holds one entry per step GEMM kernel; it is used
    only while the sources it was measured on are unchanged (the digest is
    forced to the recorded one here, so the lookup itself is what is tested)."""
    path = os.path.join(ROOT, "profiles", "gemm_lds_kernel_traffic.txt")
    sha = [ln.split(":", 1)[1].strip() for ln in open(path) if ln.startswith("source_sha256:")][0]
    monkeypatch.setattr(bench, "gemm_lds_source_digest", lambda: sha)
    desc = "gemm_lds_kernel (256x256 direct-to-LDS pipeline), {} f16 -> {}, 3 launches per step"
    for lay, out in (("NN", "f16"), ("NT", "f16"), ("TN", bench.UPDATE_OUT)):
        rec = bench._traffic_record(desc.format(lay, out))
        assert rec is not None and rec > 0, lay
    assert bench._traffic_record("skinny rows kernel, NN f16 -> f32, 1 launches per step") is None
    monkeypatch.setattr(bench, "gemm_lds_source_digest", lambda: "0" * 64)
    assert bench._traffic_record(desc.format("NN", "f16")) is None


def test_traffic_record_dropped_when_a_kernel_source_changes(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2011_11188_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in bench.TRAFFIC_SOURCES:
        shutil.copy(os.path.join(ROOT, "paper_2011_11188_amd", "csrc", f), csrc / f)
    shutil.copytree(os.path.join(ROOT, "profiles"), tmp_path / "profiles")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # a record measured on exactly these sources
    prof = tmp_path / "profiles" / "gemm_lds_kernel_traffic.txt"
    lines = [f"source_sha256: {bench.gemm_lds_source_digest()}\n" if ln.startswith("source_sha256:") else ln
             for ln in open(prof)]
    prof.write_text("".join(lines))
    desc = "gemm_lds_kernel (256x256 direct-to-LDS pipeline), NN f16 -> f16, 4 launches per step"
    assert bench._traffic_record(desc) is not None
    with open(csrc / "gemm_core.h", "a") as fh:   # the epilogue's header, not the pipeline's own
        fh.write("\n")
    assert bench._traffic_record(desc) is None


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr


def test_fused_layers_of_the_step():
    """bench.py's mirror of the library's fuse_update rule: the wide MLP's
    first layer (1024 x 4096) and three 4096 x 4096 hidden layers are updated
    in their weight-gradient products, the one-output head is not; LeNet
    (bf16 FC layers too small to skip the K split) and fp32 nets never."""
    import workloads as W
    cfg = W.wide_mlp_fp16()
    assert [bench._fused(cfg, i) for i in range(len(cfg.layers))] == [True, True, True, True, False]
    tn = [g for g in bench._step_gemms(cfg, True) if g[0] == "TN"]
    assert [g[4] for g in tn] == [bench.UPDATE_OUT] * 4 + ["f32"]
    assert all(g[4] == "f32" for g in bench._step_gemms(cfg, False) if g[0] == "TN")
    small = W.wide_mlp_fp16(batch=512, width=1024)   # 64 tiles: the unfused step splits K
    assert not any(bench._fused(small, i) for i in range(len(small.layers)))
    for c in (W.lenet_bf16(), W.mlp784_fp32()):
        assert not any(bench._fused(c, i) for i in range(len(c.layers)))
