"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Two builds made for this test only, each driven from a child process that
preloads the sanitizer runtime and stops at the first report (any report
fails the test):
  * the oracle (oracle/moe_oracle.cpp, g++ with the sanitizers), running a
    small layer forward and backward and its edge cases (one token, one
    expert, k = E, renormalised gates, an expert-parallel subset with tokens
    that have no local expert, NaN router bias, no tokens) through the
    oracle's Python wrapper;
  * the library (hipcc with the sanitizers on the host pass only; the gfx950
    code is built as usual), driving the host side of the C ABI: every
    invalid-argument case, workspaces one byte short, the workspace queries
    at small, large and overflowing sizes, and the status strings.
No GPU work happens: without a GPU, validation returns before any HIP call
and the queries are host arithmetic.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_01844_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = "-fsanitize=address,undefined"


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


pytestmark = pytest.mark.skipif(not _no_gpu(), reason="host-only checks; dummy pointers")


def _run_child(code: str, preload: str, env_extra: dict):
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2",
               PYTHONPATH=ROOT, **env_extra)
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0 and "CHILD OK" in r.stdout, out[-4000:]
    return out


ORACLE_CHILD = r'''
import numpy as np
import oracle

rng = np.random.default_rng(0)


def bf(a):
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


# T, d, E, k, f, expert_begin, num_local, renorm, NaN bias experts
CASES = [(64, 32, 8, 2, 24, 0, 8, 0, ()), (1, 8, 3, 2, 8, 0, 3, 0, ()),
         (20, 16, 1, 1, 16, 0, 1, 0, ()), (12, 16, 4, 4, 8, 0, 4, 1, ()),
         (40, 24, 16, 2, 16, 5, 3, 0, ()), (30, 16, 9, 3, 8, 0, 9, 0, (0, 4)),
         (0, 16, 4, 2, 8, 0, 4, 0, ())]
for (T, d, E, k, f, eb, el, rn, nan_e) in CASES:
    x = bf(rng.standard_normal((T, d)))
    w_r = (0.02 * rng.standard_normal((d, E))).astype(np.float32)
    bias = (0.1 * rng.standard_normal(E)).astype(np.float32)
    bias[list(nan_e)] = np.nan
    wg, wu = bf(0.02 * rng.standard_normal((el, d, f))), bf(0.02 * rng.standard_normal((el, d, f)))
    wd = bf(0.02 * rng.standard_normal((el, f, d)))
    dy = bf(rng.standard_normal((T, d)))
    for prec in ("f32", "f64"):
        o = oracle.layer(x, w_r, bias, wg, wu, wd, dy, k, e_begin=eb, E_loc=el, renorm=rn,
                         prec=prec)
        assert o["dx"].shape == (T, d)
    if o["M"]:
        n0 = int(o["offsets"][1])
        oracle.wgrad_entries(o["x_perm"][:n0], o["dy_perm"][:n0], wg[0], wu[0], wd[0],
                             [0, 1, 2], [0, 1, 0], [0, 1, 2], prec="f64")
    w64 = [(a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
           for a in (x, wg, wu, wd, dy)]
    o = oracle.layer(w64[0], w_r.astype(np.float64), bias.astype(np.float64), *w64[1:4],
                     w64[4], k, e_begin=eb, E_loc=el, renorm=rn, prec="f64_f64",
                     router_grad=True)
    assert o["dx_total"].shape == (T, d)
print("CHILD OK")
'''


def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    src = os.path.join(ROOT, "oracle", "moe_oracle.cpp")
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fopenmp", "-mavx2", "-mfma",
                    "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC", SAN,
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", src, "-o", lib],
                   check=True, capture_output=True, text=True)
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], check=True,
                          capture_output=True, text=True).stdout.strip()
    _run_child(ORACLE_CHILD, asan, {"MOE_ORACLE_LIB": lib})


LIB_CHILD = r'''
import ctypes
import sys

from paper_2607_01844_amd import _abi
from tests.abi_cases import INVALID, TOO_SMALL

L = _abi.load(sys.argv[1] if len(sys.argv) > 1 else None)
for name, call in INVALID:
    assert call(L) == -1, name
    assert len(L.moe_last_error()) > 0, name
for call in TOO_SMALL:
    assert call(L) == -3
for s in range(-8, 2):
    L.moe_status_string(s)
n = ctypes.c_size_t()
B = 1 << 40
# small, large and absurd sizes: each query answers or refuses, with no
# undefined arithmetic on the way
for T in (0, 1, 4096, 1 << 31, B):
    L.moe_route_workspace_bytes(T, 1024, ctypes.byref(n))
    L.moe_route_bwd_workspace_bytes(T, 262144, 1024, ctypes.byref(n))
    L.moe_permute_workspace_bytes(T, 1024, 16, 1024, ctypes.byref(n))
    L.moe_grouped_swiglu_workspace_bytes(T, 1024, 262144, 262144, 3, ctypes.byref(n))
    L.moe_ffn_fwd_chunked_workspace_bytes(T, 262144, 1024, 16, 1024, 262144, ctypes.byref(n))
    L.moe_ffn_fwd_row_chunked_workspace_bytes(T, 1024, 16, 1024, 262144, 262144, B, ctypes.byref(n))
    L.moe_ffn_fwd_row_chunked_workspace_bytes(T, 64, 6, 64, 2048, 1408, 1, ctypes.byref(n))
    L.moe_vocab_loss_workspace_bytes(T, 262144, B, 1 << 32, ctypes.byref(n))
    L.moe_vocab_loss_workspace_bytes(T, 8, 9, 8, ctypes.byref(n))
print("CHILD OK")
'''


def test_library_host_side_under_asan_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2607_01844_amd import build as B
    flags = list(B.CFLAGS) + [
        "-Xarch_host", SAN, "-Xarch_host", "-fno-sanitize-recover=undefined",
        "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-O1", "-Xarch_host", "-g"]
    procs, objs = [], []
    for src in B.SOURCES:
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for p in procs:
        out, _ = p.communicate(timeout=900)
        assert p.returncode == 0, out[-3000:]
    lib = str(tmp_path / "libmoe_san.so")
    subprocess.run([HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, "-o", lib,
                    "-Xarch_host", SAN], check=True, capture_output=True, text=True)
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    assert rt, "clang's AddressSanitizer runtime is missing"
    _run_child(LIB_CHILD.replace("sys.argv[1] if len(sys.argv) > 1 else None", repr(lib)),
               rt[-1], {})
