"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

tests/c/host_abi_check.cpp drives the routing templates, coverage accounting, template fitting,
the automatic group size and the validation and workspace plans of every entry point over many
geometries, on a build of the library sources whose host code carries both sanitizers (device
code is built as usual but never launched).  A second run passes a routing buffer one word
short, which AddressSanitizer must report: the instrumentation is live."""

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_17336_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fhip-fp32-correctly-rounded-divide-sqrt",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("hostsan")
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))

    def compile_one(src):
        obj = str(out / (os.path.basename(src) + ".o"))
        r = subprocess.run([HIPCC, *FLAGS, *SAN, "-c", src, "-o", obj], capture_output=True,
                           text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = str(out / "host_abi_check")
    r = subprocess.run([HIPCC, *FLAGS, *SAN, "-x", "c++",
                        os.path.join(ROOT, "tests", "c", "host_abi_check.cpp"), "-x", "none", *objs,
                        "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def test_host_code_clean_under_sanitizers(checker):
    r = subprocess.run([checker], capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-6000:]
    assert "host ABI checks ok" in r.stdout


def test_sanitizer_is_live(checker):
    r = subprocess.run([checker, "undersized"], capture_output=True, text=True, env=ENV,
                       timeout=300)
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stderr
