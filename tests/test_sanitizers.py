"""AddressSanitizer and UndefinedBehaviorSanitizer runs on the CPU.

- The oracle (oracle/memoplan_oracle.c) built with gcc under
  -fsanitize=address,undefined together with tests/sanitize/oracle_driver.c,
  which calls every oracle entry point on a hand-worked example and seeded
  random traces and checks results that hold by definition.
- The host side of the C ABI: the library sources and
  tests/sanitize/abi_driver.cpp built with hipcc, the sanitizers on the host
  pass only (-Xarch_host before each -fsanitize=), run without a GPU: status
  strings, workspace and capacity queries over their whole argument ranges,
  and every entry point with arguments its host checks must reject.
Any sanitizer report ends the child with a nonzero status.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(exe, tmp_path):
    r = subprocess.run([exe], cwd=tmp_path, capture_output=True, text=True, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out
    assert "runtime error" not in out and "AddressSanitizer" not in out, out
    return out


def test_oracle_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", *SAN, "-I", os.path.join(ROOT, "oracle"),
                    os.path.join(ROOT, "oracle", "memoplan_oracle.c"),
                    os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), "-o", exe],
                   check=True)
    assert "all checks passed" in _run(exe, tmp_path)


def test_abi_host_under_asan_ubsan(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    csrc = os.path.join(ROOT, "paper_2203_00448_amd", "csrc")
    srcs = sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))
    host_san = [a for flag in SAN for a in ("-Xarch_host", flag)]
    exe = str(tmp_path / "abi_driver")
    subprocess.run([hipcc, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", *host_san,
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", os.path.join(ROOT, "include"), "-I", csrc,
                    os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp"), *srcs, "-o", exe],
                   check=True, capture_output=True)
    assert "all checks passed" in _run(exe, tmp_path)
