"""The host-side C++ (host_plan.h: checks, plans, workspace layout and cache)
and the C oracle, built with AddressSanitizer and UndefinedBehaviorSanitizer
for the CPU (g++ / gcc, no GPU code) and run by tests/c_abi/sanitize_host.cpp."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="no host compiler")
def test_host_code_under_sanitizers(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
    obj = tmp_path / "oracle_topk.o"
    subprocess.run(["gcc", "-std=c11", "-c", os.path.join(ROOT, "oracle", "oracle_topk.c"), "-o", str(obj)] + san,
                   check=True)
    exe = tmp_path / "sanitize_host"
    subprocess.run(["g++", "-std=c++17", "-I" + os.path.join(ROOT, "include"),
                    "-I" + os.path.join(ROOT, "paper_2604_22312_amd", "csrc"),
                    os.path.join(ROOT, "tests", "c_abi", "sanitize_host.cpp"), str(obj), "-o", str(exe)] + san,
                   check=True)
    # (verify_asan_link_order=0: the environment may preload a library ahead of the sanitizer runtime)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
