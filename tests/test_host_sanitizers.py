"""Host-only native code under the compiler's sanitizers.

The 8-bit quantiser runs under AddressSanitizer + UndefinedBehaviorSanitizer,
and under ThreadSanitizer over its threaded path.  MD5 runs under
AddressSanitizer + UndefinedBehaviorSanitizer.  Each is driven by a small C++
harness (tests/native/) on exactly sized buffers, built with g++ (host code
only; no GPU code is involved)."""

from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_24204_amd", "csrc")
NATIVE = os.path.join(ROOT, "tests", "native")
GXX = shutil.which("g++")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

pytestmark = pytest.mark.skipif(GXX is None, reason="g++ not available")

ASAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _build_and_run(tmp_path, name, sources, flags, link=(), args=()):
    exe = str(tmp_path / name)
    cmd = [GXX, "-O1", "-g", "-std=c++17", "-pthread", *flags, *sources, "-o", exe, *link]
    b = subprocess.run(cmd, capture_output=True, text=True)
    assert b.returncode == 0, b.stderr[-4000:]
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert r.stdout.strip().startswith("ok"), r.stdout


def test_quantiser_address_and_undefined_behaviour(tmp_path):
    _build_and_run(tmp_path, "q_asan",
                   [os.path.join(NATIVE, "quant_harness.cpp"), os.path.join(CSRC, "quant.cpp")],
                   ASAN)


def test_quantiser_threads(tmp_path):
    _build_and_run(tmp_path, "q_tsan",
                   [os.path.join(NATIVE, "quant_harness.cpp"), os.path.join(CSRC, "quant.cpp")],
                   ["-fsanitize=thread"], args=("threads",))


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")),
                    reason="HIP runtime library not available")
def test_md5_address_and_undefined_behaviour(tmp_path):
    # cache.cpp also holds the cached weight loader, which calls the HIP runtime
    # and the model's entry points; the harness calls only wici_md5, so those
    # references are left unresolved.
    _build_and_run(tmp_path, "md5_asan",
                   [os.path.join(NATIVE, "md5_harness.cpp"), os.path.join(CSRC, "cache.cpp")],
                   ASAN + ["-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include"],
                   link=[f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib",
                         "-Wl,--unresolved-symbols=ignore-in-object-files"])
