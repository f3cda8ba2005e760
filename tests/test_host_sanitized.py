"""The C-ABI shim built for the host alone with AddressSanitizer,
UndefinedBehaviorSanitizer and the checked C++ standard library, its HIP
runtime calls and kernel launches replaced by host stand-ins
(tests/host/hip_stubs.cpp), and driven by tests/host/abi_host_check.cpp:

* the host-only table builders and the depth search write and read exactly
  the buffers the interface states (heap blocks of that size), including
  refused calls that must leave a too-small buffer untouched and malformed
  caller tables that must be rejected;
* every runtime or launch failure surfaces as BF1_ERR_HIP;
* the plan cache builds each plan once, refuses to build one under graph
  capture (BF1_ERR_CAPTURE) and frees everything it allocated;
* the tables it prints equal the oracle's.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import bf1_oracle as orc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = os.path.join(ROOT, "tests", "host")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def report(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir(os.path.join(ROCM, "include", "hip")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path_factory.mktemp("asan") / "abi_host_check")
    cmd = [gxx, "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D_GLIBCXX_DEBUG", "-D_GLIBCXX_ASSERTIONS", f"-I{ROCM}/include", "-D__HIP_PLATFORM_AMD__",
           os.path.join(ROOT, "paper_2608_20427_amd", "csrc", "bf1_api.cpp"),
           os.path.join(HOST, "hip_stubs.cpp"), os.path.join(HOST, "abi_host_check.cpp"), "-o", exe]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stdout[-6000:]
    assert "ERROR: AddressSanitizer" not in r.stdout and "runtime error" not in r.stdout, r.stdout[-6000:]
    assert r.stdout.rstrip().endswith("ALL OK"), r.stdout[-3000:]
    return r.stdout.splitlines()


def _tables(lines):
    out = {}
    for line in lines:
        if line.startswith("table "):
            head, tail = line.split(" |")
            _, kind, n, B, L, *rp = head.split()
            out[(kind, int(n), int(B), int(L))] = (np.array(rp, dtype=np.int64),
                                                   np.array(tail.split(), dtype=np.int64))
    return out


def test_sanitized_build_runs_clean(report):
    assert any(l.startswith("allocations ") for l in report)


def test_sanitized_tables_match_oracle(report):
    tables = _tables(report)
    assert len(tables) == 40
    for (kind, n, B, L), (rp, ci) in tables.items():
        if kind == "transposed":
            rp_o, ci_o = orc.csr_transposed(n, B, L)
        else:
            rp_o, ci_o = orc.variant_csr(kind, n, B, L, 17)
        assert rp.tolist() == list(rp_o) and ci.tolist() == list(ci_o), (kind, n, B, L)


def test_sanitized_depths_match_oracle(report):
    depths = [l.split() for l in report if l.startswith("depth ")]
    assert len(depths) == 30
    tables = _tables(report)
    for _, kind, n, B, L, d in depths:
        rp, ci = tables[(kind, int(n), int(B), int(L))]
        try:
            want = orc.max_shortest_path_csr(rp, ci)
        except AssertionError:          # the oracle refuses unreachable blocks; the ABI says -1
            want = -1
        assert int(d) == want, (kind, n, B, L)


def test_sanitized_sizes_match_the_library(report):
    import paper_2608_20427_amd as bf1
    for l in report:
        if l.startswith("bwd_ws "):
            batch, n, Hq, Hkv, d, B, L, nbytes = map(int, l.split()[1:])
            assert bf1.bwd_workspace_size(batch, n, Hq, Hkv, d, B, L) == nbytes
        if l.startswith("decode "):
            stride, nbytes = map(int, l.split()[1:])
            assert stride == bf1.decode_plan_stride(65536, 64, 2)
            assert nbytes == bf1.decode_workspace_size(32, 16, 8, 128, stride)


def test_sanitizer_reports_a_planted_overflow(tmp_path):
    # negative control: the same flags catch a one-past-the-end heap write
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("needs g++")
    src = tmp_path / "overflow.cpp"
    src.write_text("#include <vector>\nint main(){ std::vector<int> v(7); int* p = v.data(); p[7] = 1;"
                   " return p[0]; }\n")
    exe = str(tmp_path / "overflow")
    r = subprocess.run([gxx, "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                        str(src), "-o", exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    env = dict(os.environ, ASAN_OPTIONS="verify_asan_link_order=0")
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stdout
