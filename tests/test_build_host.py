"""Host checks of the build step's bookkeeping (no GPU): the device-code hashes
written beside the library, and the benchmark's use of them to decide
whether a stored counter summary still describes the built GEMM kernel."""
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_01844_amd")


def test_device_text_hashes_cover_every_source():
    from paper_2607_01844_amd import build
    path = build.DEVICE_TEXT
    if not os.path.exists(path):
        pytest.skip("library not built")
    hashes = json.load(open(path))
    assert set(hashes) == set(build.SOURCES)
    # sources with kernels have a hash; host-only sources none
    for src, h in hashes.items():
        if h is not None:
            assert len(h) == 64 and int(h, 16) >= 0
    assert hashes["gemm.hip"] is not None and hashes["api.hip"] is None


def test_device_text_hash_ignores_host_only_changes(tmp_path):
    """Two objects compiled from the same kernel, one with an extra host
    function, have the same device-code hash; a changed kernel does not."""
    import subprocess
    from paper_2607_01844_amd import build
    base = "__global__ void k(float* p) { p[threadIdx.x] = %s; }\n"
    srcs = {"a": base % "1.0f", "b": base % "1.0f" + "int host_only(int v) { return v + 1; }\n",
            "c": base % "2.0f"}
    objs = {}
    for name, text in srcs.items():
        src = tmp_path / f"{name}.hip"
        src.write_text("#include <hip/hip_runtime.h>\n" + text)
        obj = tmp_path / f"{name}.o"
        subprocess.run([build.HIPCC, f"--offload-arch={build.ARCH}", "-O2", "-fPIC", "-c",
                        str(src), "-o", str(obj)], check=True, capture_output=True)
        objs[name] = build.device_text_sha256(str(obj))
    assert objs["a"] == objs["b"]
    assert objs["a"] != objs["c"]


def test_stored_traffic_follows_the_gemm_code(tmp_path, monkeypatch):
    import bench
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    (tmp_path / "paper_2607_01844_amd").mkdir()
    built = tmp_path / "paper_2607_01844_amd" / "libmoe.device_text.json"
    prof = tmp_path / "profiles" / "moe_layer_mid_hbm_traffic.txt"
    prof.write_text("# comment\ndevice_text_sha256 gemm.hip abc\n"
                    "kernel gemm_wgrad_gate_up read_bytes=100 write_bytes=20\n")
    built.write_text(json.dumps({"gemm.hip": "abc"}))
    assert bench.stored_traffic("mid", "gemm_wgrad_gate_up") == 120
    assert bench.stored_traffic("mid", "gemm_fwd_down") is None      # no such line
    assert bench.stored_traffic("large_skew", "gemm_wgrad_gate_up") is None  # no summary
    built.write_text(json.dumps({"gemm.hip": "def"}))                # kernel changed
    assert bench.stored_traffic("mid", "gemm_wgrad_gate_up") is None
