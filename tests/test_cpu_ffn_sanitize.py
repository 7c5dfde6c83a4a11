"""The host expert kernels of the cooperative compensation (cpu_ffn.cpp) built
with g++ under AddressSanitizer + UndefinedBehaviorSanitizer and under
ThreadSanitizer, and run over ragged shapes on both instruction-set paths
(AVX-512 BF16 where the CPU has it, and the AVX2 path forced by
OLED_CPU_FFN_AVX2=1). Both paths must give the same sums."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2609_33385_amd", "csrc")
SRC = [os.path.join(HERE, "native", "cpu_ffn_sanitize.cpp"), os.path.join(CSRC, "cpu_ffn.cpp")]


def _build(tmp_path, flags, name):
    exe = str(tmp_path / name)
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=fast",
           "-I", CSRC] + flags + SRC + ["-o", exe, "-lpthread"]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    return exe


def _run(exe, avx2):
    env = dict(os.environ)
    env.pop("OLED_CPU_FFN_AVX2", None)
    if avx2:
        env["OLED_CPU_FFN_AVX2"] = "1"
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["TSAN_OPTIONS"] = "halt_on_error=1"
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "Sanitizer" not in r.stderr, r.stderr[-4000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("bf16=")]
    assert len(lines) == 10
    return lines


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_cpu_ffn_asan_ubsan(tmp_path):
    exe = _build(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"],
                 "asan")
    assert _run(exe, avx2=False) == _run(exe, avx2=True)


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_cpu_ffn_tsan(tmp_path):
    exe = _build(tmp_path, ["-fsanitize=thread"], "tsan")
    _run(exe, avx2=False)
