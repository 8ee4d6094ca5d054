"""The segment turnstile and the P-epoch runner (host code) under
ThreadSanitizer and under AddressSanitizer + UndefinedBehaviorSanitizer.

The library's own csrc/turnstile.cpp is compiled with g++ (host only) into
tests/native/turnstile_stress.cpp, a driver that runs the controller from a P
thread and a D thread, then the runner's thread against a D thread over
host-only stand-ins of the layer calls, and checks the protocol's outcomes
and its transition log.  The test passes when the driver exits cleanly with
no sanitizer report; it is skipped when the toolchain lacks the sanitizer's
runtime.

The host compiler is ROCm's clang++ (its sanitizer runtimes ship with it).
GCC 11's ThreadSanitizer runtime does not intercept pthread_cond_clockwait,
which libstdc++ uses for condition-variable waits on the steady clock, so it
misses the unlock inside such a wait and reports a double lock that is not
there; it is used only when clang++ is absent."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_00993_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

MODES = {
    "thread": ["-fsanitize=thread"],
    "address-undefined": ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"],
}


def build(mode, tmp_path):
    cxx = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not os.path.exists(cxx):
        cxx = shutil.which("g++")
        if cxx is None:
            pytest.skip("no host C++ compiler")
    exe = str(tmp_path / f"turnstile_stress_{mode}")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-pthread", *MODES[mode],
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "turnstile_stress.cpp"), os.path.join(CSRC, "turnstile.cpp"),
           "-o", exe]
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if p.returncode != 0:
        if "cannot find" in p.stdout and ("tsan" in p.stdout or "asan" in p.stdout or "ubsan" in p.stdout):
            pytest.skip(f"sanitizer runtime missing: {p.stdout.strip().splitlines()[-1]}")
        raise AssertionError(f"build failed:\n{' '.join(cmd)}\n{p.stdout}")
    return exe


@pytest.mark.parametrize("mode", list(MODES))
def test_turnstile_under_sanitizer(mode, tmp_path):
    exe = build(mode, tmp_path)
    env = dict(os.environ)
    env["TSAN_OPTIONS"] = "halt_on_error=1 second_deadlock_stack=1"
    env["ASAN_OPTIONS"] = "detect_leaks=1 halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1 print_stacktrace=1"
    p = subprocess.run([exe, "200"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env,
                       timeout=240)
    out = p.stdout
    assert p.returncode == 0, out[-4000:]
    for marker in ("WARNING: ThreadSanitizer", "ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer"):
        assert marker not in out, out[-4000:]
    assert out.strip().endswith("ok"), out[-2000:]
