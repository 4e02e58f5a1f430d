"""Host-only unit tests of the C++ residency planner, built with g++ and
AddressSanitizer / UndefinedBehaviorSanitizer (no GPU)."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_plan_core(tmp_path):
    exe = str(tmp_path / "plan_core_test")
    src = [os.path.join(ROOT, "tests", "cpp", "plan_core_test.cpp"),
           os.path.join(ROOT, "paper_2608_23805_amd", "csrc", "plan_core.cpp")]
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"),
                    "-o", exe] + src, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
