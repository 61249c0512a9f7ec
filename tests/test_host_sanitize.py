"""The HIP-free host part of the library (paper_2609_14237_amd/csrc/ods_host.cpp:
allocator, sizing, validation and launch planning) built with the host
compiler under AddressSanitizer and UndefinedBehaviorSanitizer, and run over
every operator range of the evaluated workload shapes (tests/host/host_check.cpp).
No GPU is involved."""
import os
import shutil
import subprocess

import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CXX = os.environ.get("CXX", "g++")


@pytest.mark.skipif(shutil.which(CXX) is None, reason="no host C++ compiler")
def test_host_part_is_clean_under_asan_and_ubsan(tmp_path):
    works = tmp_path / "workloads.txt"
    with open(works, "w") as fh:
        for w in W.ALL + W.SHARES:
            fh.write(f"{w.name} {w.batch} {w.max_pages} {len(w.layers)}")
            for c in w.layers:
                fh.write(f" {c.hidden} {c.n_q} {c.n_kv} {c.head_dim} {c.ffn} {c.n_experts} {c.top_k} "
                         f"{c.moe_ffn} {c.window}")
            fh.write("\n")
    exe = tmp_path / "host_check"
    cmd = [CXX, "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2609_14237_amd", "csrc", "ods_host.cpp"),
           os.path.join(ROOT, "tests", "host", "host_check.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), str(works)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "host_check OK" in r.stdout
