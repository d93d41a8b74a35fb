"""The host code that parses and writes the stored model -- the packer, the
blob validation, the pruning-structure helpers (pack.cpp, project.cpp) --
built with AddressSanitizer and UndefinedBehaviorSanitizer for the CPU and
run (a) by a seeded C++ driver that packs random layers and feeds
truncated, bit-flipped and overwritten blobs to the validation, and (b) in a
Python process that byte-compares the packer with the oracle's packer and
repeats the corruption checks.  Any out-of-bounds access, leak in the
driver, or undefined behaviour aborts the run."""
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2004_11250_amd", "csrc")
GXX = shutil.which("g++")
pytestmark = pytest.mark.skipif(GXX is None, reason="g++ not found")

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
HOST_SOURCES = [os.path.join(CSRC, "pack.cpp"), os.path.join(CSRC, "project.cpp")]


@pytest.fixture(scope="module")
def tmp():
    d = tempfile.mkdtemp(prefix="pp_san_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def _env(leaks):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = f"detect_leaks={1 if leaks else 0}:verify_asan_link_order=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


def test_fuzz_driver_under_sanitizers(tmp):
    exe = os.path.join(tmp, "fuzz_host")
    subprocess.run([GXX, "-std=c++17", *SAN, f"-I{ROOT}/include", f"-I{CSRC}",
                    os.path.join(ROOT, "tests", "sanitize", "fuzz_host.cpp"), *HOST_SOURCES, "-o", exe], check=True)
    r = subprocess.run([exe], env=_env(True), capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


def test_packer_parity_under_sanitizers(tmp):
    so = os.path.join(tmp, "libppconv_host_asan.so")
    subprocess.run([GXX, "-std=c++17", *SAN, "-fPIC", "-shared", f"-I{ROOT}/include", f"-I{CSRC}", *HOST_SOURCES,
                    "-o", so], check=True)
    runtime = subprocess.run([GXX, "-print-file-name=libasan.so"], capture_output=True, text=True,
                             check=True).stdout.strip()
    env = _env(False)   # the interpreter's own allocations are not this code's
    env["LD_PRELOAD"] = runtime + (" " + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "sanitize", "asan_pack.py"), so, ROOT], env=env,
                       capture_output=True, text=True, timeout=900, cwd=ROOT)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "blobs identical" in r.stdout
