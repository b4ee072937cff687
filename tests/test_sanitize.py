"""The oracle and the library's host-side validation built with
AddressSanitizer and UndefinedBehaviorSanitizer (CPU only) and driven over
a spread of valid, invalid and extreme inputs (tests/sanitize/): any
out-of-bounds access, use of freed memory or undefined arithmetic fails the
test.  The library's kernel launches are replaced by stand-ins that launch
nothing."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
CLANG = "/opt/rocm/llvm/bin/clang++"


def run(cmd, env=None):
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=600, env=env)
    return p.returncode, p.stdout + p.stderr


def sanitizer_env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    return env


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    rc, out = run(["gcc", "-std=gnu99", "-O1", "-g", "-ffp-contract=off", "-fno-fast-math", "-Wall"] + SAN +
                  ["-o", exe, os.path.join(HERE, "sanitize", "oracle_driver.c"), "-lm", "-lpthread"])
    assert rc == 0, out
    rc, out = run([exe], env=dict(sanitizer_env(), ASAN_OPTIONS="detect_leaks=1"))
    assert rc == 0 and "runtime error" not in out and "AddressSanitizer" not in out, out
    assert "0 failures" in out


@pytest.mark.skipif(not os.path.exists(CLANG), reason="the ROCm clang is not installed")
def test_host_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "api_driver")
    rc, out = run([CLANG, "-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                   "-I", os.path.join(ROOT, "include")] + SAN +
                  ["-o", exe, os.path.join(HERE, "sanitize", "api_driver.cpp"),
                   os.path.join(HERE, "sanitize", "launch_stubs.cpp"),
                   os.path.join(ROOT, "paper_2111_05426_amd", "csrc", "api.cpp"),
                   "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    assert rc == 0, out
    rc, out = run([exe], env=sanitizer_env())
    assert rc == 0 and "runtime error" not in out and "AddressSanitizer" not in out, out
    assert "reached a launch" in out


@pytest.mark.skipif(not os.path.exists(CLANG), reason="the ROCm clang is not installed")
def test_front_end_under_sanitizers(tmp_path):
    """The parser, interpreter and lowering over valid programs (Fig. 4's
    snippet, GPT-2-shaped layers, random programs) and 4000 mutated ones."""
    import json
    import sys
    sys.path.insert(0, HERE)
    from random_programs import random_program
    from paper_2111_05426_amd import programs
    with open(os.path.join(HERE, "golden", "fig4_reshape.json")) as f:
        fig4 = json.load(f)["program"]
    texts = [fig4.replace("%3114", "%flat"), programs.gpt2_layers(3, 64, n_layers=2, tp=2, pp=2)] + \
        [random_program(s, n_ops=30, n_dev=1 + s % 4) for s in range(6)]
    files = []
    for i, t in enumerate(texts):
        files.append(str(tmp_path / ("p%d.txt" % i)))
        with open(files[-1], "w") as f:
            f.write(t)
    exe = str(tmp_path / "frontend_driver")
    rc, out = run([CLANG, "-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                   "-I", os.path.join(ROOT, "include")] + SAN +
                  ["-o", exe, os.path.join(HERE, "sanitize", "frontend_driver.cpp"),
                   os.path.join(ROOT, "paper_2111_05426_amd", "csrc", "frontend.cpp"),
                   os.path.join(HERE, "sanitize", "launch_stubs.cpp"),
                   os.path.join(ROOT, "paper_2111_05426_amd", "csrc", "api.cpp"),
                   "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    assert rc == 0, out
    rc, out = run([exe] + files, env=dict(sanitizer_env(), ASAN_OPTIONS="detect_leaks=1"))
    assert rc == 0 and "runtime error" not in out and "AddressSanitizer" not in out, out
    assert "0 failures" in out
