"""Host code of the library under ThreadSanitizer: a build of liblinattn
whose host code is instrumented (the GPU code is built as usual), driven
by eight threads that call the host entry points at once
(tests/tsan/host_threads.cpp).  Every call there is answered on the host,
so no GPU is needed.  The test passes when the driver reports no mismatch
and ThreadSanitizer reports no data race."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANGXX = "/opt/rocm/llvm/bin/clang++"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="ROCm toolchain not found")
def test_host_entry_points_have_no_data_race(tmp_path):
    lib = tmp_path / "liblinattn_tsan.so"
    src = os.path.join(ROOT, "paper_2609_15030_amd", "csrc", "linattn.hip")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_15030_amd", "csrc")]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-Xarch_host", "-fsanitize=thread", *inc, src, "-o", str(lib)],
                   check=True, capture_output=True, timeout=600)
    exe = tmp_path / "host_threads"
    subprocess.run([CLANGXX, "-O1", "-g", "-std=c++17", "-fsanitize=thread", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "tsan", "host_threads.cpp"), "-L", str(tmp_path), "-llinattn_tsan",
                    f"-Wl,-rpath,{tmp_path}", "-o", str(exe)], check=True, capture_output=True, timeout=300)
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert "ThreadSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, (r.stdout, r.stderr[-4000:])
    assert "0 mismatches" in r.stdout
