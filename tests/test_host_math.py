"""Host-side arithmetic of the library, compiled and run on the CPU."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# host programs: built with AddressSanitizer and UndefinedBehaviorSanitizer
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_stride_division_is_exact(tmp_path):
    exe = tmp_path / "check_divl"
    subprocess.run([HIPCC, "-O2", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "paper_1904_10509_amd", "csrc"),
                    os.path.join(ROOT, "tests", "host", "check_divl.cpp"), "-o", str(exe)], check=True,
                   capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert out.returncode == 0 and out.stdout.startswith("ok"), out.stdout + out.stderr


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_decode_set_enumerates_s_pos(tmp_path):
    exe = tmp_path / "check_decode_set"
    subprocess.run([HIPCC, "-O2", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "paper_1904_10509_amd", "csrc"),
                    os.path.join(ROOT, "tests", "host", "check_decode_set.cpp"), "-o", str(exe)], check=True,
                   capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert out.returncode == 0 and out.stdout.startswith("ok"), out.stdout + out.stderr


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_summary_window_closed_forms(tmp_path):
    exe = tmp_path / "check_pattern_window"
    subprocess.run([HIPCC, "-O2", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "paper_1904_10509_amd", "csrc"),
                    os.path.join(ROOT, "tests", "host", "check_pattern_window.cpp"), "-o", str(exe)], check=True,
                   capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert out.returncode == 0 and out.stdout.startswith("ok"), out.stdout + out.stderr
