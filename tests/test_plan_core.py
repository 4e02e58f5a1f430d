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


def _source_test(tmp_path, sanitize):
    exe = str(tmp_path / f"source_test_{sanitize.split(',')[0]}")
    src = [os.path.join(ROOT, "tests", "cpp", "source_test.cpp"),
           os.path.join(ROOT, "paper_2608_23805_amd", "csrc", "source.cpp")]
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-pthread", f"-fsanitize={sanitize}",
                    "-o", exe] + src, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr


def test_source_service_asan(tmp_path):
    """Bounded source service under AddressSanitizer / UBSan."""
    _source_test(tmp_path, "address,undefined")


def test_source_service_tsan(tmp_path):
    """The same under ThreadSanitizer (I/O workers and the collecting thread)."""
    _source_test(tmp_path, "thread")
