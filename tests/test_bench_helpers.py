"""CPU tests of bench.py's bookkeeping: the roofline each fused layer is graded
against, the HBM-traffic record that is valid only for unchanged kernel
sources, and the refusal to run on more than one GPU."""
import hashlib
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_wide_layers_are_matrix_core_bound_narrow_bf16_is_valu_bound():
    nb = 13  # G = 10
    for dt in ("bf16", "f32"):
        assert bench.layer_roofline(dt, 65536, 784, 256, nb)["bound"] == "mfma"
        assert bench.layer_roofline(dt, 65536, 256, 256, nb)["bound"] == "mfma"
    # out = 10: 38 lane-ops per (row, feature) at 78.6 T/s outlast 2 x 10 x 14
    # flops at 2516.6 TFLOP/s, but not at the fp32 matrix-core peak of 157.3
    assert bench.layer_roofline("bf16", 65536, 256, 10, nb)["bound"] == "alu"
    assert bench.layer_roofline("f32", 65536, 256, 10, nb)["bound"] == "mfma"


def test_layer_roofline_work_counts():
    k = bench.layer_roofline("bf16", 65536, 784, 256, 13)
    # dense contraction: 2 * B * out * in * (G + 4) flops
    assert k["algorithmic"] == pytest.approx(2.0 * 65536 * 256 * 784 * 14 / 1e12)
    assert k["peak"] == bench.PEAK_TFLOPS["bf16"]
    n = bench.layer_roofline("bf16", 65536, 256, 10, 13)
    assert n["unit"] == "Gop/s"
    assert n["algorithmic"] == pytest.approx(38.0 * 65536 * 256 / 1e9)
    assert n["peak"] == pytest.approx(256 * 4 * 32 * 2.4)


def test_narrow_kernel_layer_roofline():
    # the vector-ALU kernel: 36 lane-ops of basis generation plus 5 x out fmas
    # per (row, feature), against the VALU peak
    k = bench.layer_roofline("f32", 65536, 256, 10, 13, narrow=True)
    assert k["bound"] == "alu" and k["unit"] == "Gop/s"
    assert k["algorithmic"] == pytest.approx((36.0 + 50.0) * 65536 * 256 / 1e9)
    assert k["peak"] == pytest.approx(256 * 4 * 32 * 2.4)


def _fake_tree(tmp_path, record_md5):
    csrc = tmp_path / "paper_2609_01956_amd" / "csrc"
    csrc.mkdir(parents=True)
    h = hashlib.md5()
    for f in bench.KERNEL_SOURCES:
        data = f"// {f}\n".encode()
        (csrc / f).write_bytes(data)
        h.update(data)
    md5 = h.hexdigest() if record_md5 is None else record_md5
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "kan_mlp_c5_bf16_hbm_traffic.md").write_text(
        "# summary\n\n```\ntraffic-record\n"
        f"kernel_sources_md5: {md5}\ndtype: bf16\nkernel: layer1_784x256\n"
        "fetch_kib: 100.0\nwrite_kib: 50.0\nfetch_factor: 2.0\nwrite_factor: 1.0\n```\n")
    return str(tmp_path)


def test_traffic_record_scaled_bytes(tmp_path):
    root = _fake_tree(tmp_path, None)
    assert bench.traffic_record("bf16", "layer1_784x256", root) == pytest.approx(250.0 * 1024)


def test_traffic_record_void_when_sources_changed_or_other_kernel(tmp_path):
    root = _fake_tree(tmp_path, "0" * 32)
    assert bench.traffic_record("bf16", "layer1_784x256", root) is None
    root2 = _fake_tree(tmp_path / "b", None)
    assert bench.traffic_record("bf16", "layer2_256x256", root2) is None
    assert bench.traffic_record("f32", "layer1_784x256", root2) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_sample_is_sized_by_a_sizing_run():
    """The oracle baseline sizes its sample from a second, longer run (the
    64-row warm-up is mostly fixed cost), reports the median of three runs
    and the threads it used."""
    from paper_2609_01956_amd import workloads as wl

    W = wl.make_workload("c2_layer_64x64_g5")
    r = bench.cpu_baseline(W, 0.6)
    assert r["kind"] == "oracle" and r["unit"] == "samples/s" and r["value"] > 0
    assert r["cores"] >= 1
    assert "sizing run" in r["sample"] and "median of 3 runs" in r["sample"]
    rows = int(r["sample"].split("first ")[1].split(" rows")[0])
    assert 64 <= rows <= W["x"].shape[0]
