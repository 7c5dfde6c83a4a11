"""The host runtime (oled.cpp) built with g++ under AddressSanitizer +
UndefinedBehaviorSanitizer (leak checking on), linked with a host-only stand-in
for the HIP runtime and the kernel launchers (tests/native/fake_hip.cpp), and
driven through the C ABI by tests/native/runtime_sanitize.cpp: oled_create's
argument checks, the per-layer call order, record draining, profiling and
inspection, the rollback after a miss copy that cannot be enqueued, the wait
deadline and the reset after it, layer-adaptive sizing and the comparison
policies, and teardown. No GPU is used."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_33385_amd", "csrc")
SRC = [os.path.join(HERE, "native", "runtime_sanitize.cpp"),
       os.path.join(HERE, "native", "fake_hip.cpp"),
       os.path.join(CSRC, "oled.cpp"), os.path.join(CSRC, "cpu_ffn.cpp")]


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the HIP headers")
def test_runtime_asan_ubsan(tmp_path):
    exe = str(tmp_path / "runtime_asan")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, "-ffp-contract=off"] + SRC + ["-o", exe, "-lpthread"]
    subprocess.run(cmd, check=True, capture_output=True, timeout=600)
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "Sanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.stdout.rstrip().endswith("ALL OK")
    assert "could not be enqueued" in r.stdout
    assert "not complete within 5 ms" in r.stdout
