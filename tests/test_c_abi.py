"""The library used through its C ABI alone: tests/c_abi/abi_host.cpp is a
host program (HIP runtime for device memory and a stream, the calls of
include/gvr_topk.h, no Python or torch) that compares gvr_topk, radix_topk
and gvr_topk_ex (8-wave and 4-wave shapes, the paper's Phase 4 and Phase 2/3
options) with the C oracle, linked in as a test dependency. On the CPU the
program is compiled and linked; on the GPU it runs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "abi_host.cpp")


def _libs():
    import oracle
    import paper_2604_22312_amd as g
    if not os.path.exists(g.library_path()):
        from paper_2604_22312_amd import build
        build.build()
    oracle.build(force=False)
    return os.path.dirname(g.library_path()), os.path.dirname(oracle.LIBRARY)


def build_host(out_dir):
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else shutil.which("hipcc")
    if hipcc is None:
        pytest.skip("hipcc not found")
    pkg, orc = _libs()
    exe = os.path.join(out_dir, "abi_host")
    cmd = [hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"), SRC, "-o", exe,
           "-L" + pkg, "-lgvr_topk", "-L" + orc, "-loracle_topk", "-Wl,-rpath," + pkg + ":" + orc]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_c_abi_host_program_builds(tmp_path):
    exe = build_host(str(tmp_path))
    assert os.access(exe, os.X_OK)


@pytest.mark.gpu
def test_c_abi_host_program_matches_the_oracle(tmp_path):
    exe = build_host(str(tmp_path))
    print("running the C-ABI host program", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok")
    assert "DIFFERS" not in r.stdout
