"""The host library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU, no GPU).

The C ABI and launch planning (pic_api.cpp, pic_plan.cpp) are built with both sanitizers
against a CPU emulation of every kernel launch (tests/sanitize/emulated_launchers.cpp), which
derives each row a kernel addresses with the kernels' own clamping helpers (pic_bounds.h) and
touches it in host buffers of exactly the documented sizes.  The driver
(tests/sanitize/sanitize_driver.cpp) fuzzes the planners, feeds garbage device tables (gather
blocks, group starts, slot and tile maps, lengths, positions) to every entry point, and checks
that failing calls launch nothing.  A planted mistake (a cache one row short) must be caught.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang++"
SOURCES = [os.path.join(ROOT, "paper_2607_28069_amd", "csrc", "pic_api.cpp"),
           os.path.join(ROOT, "paper_2607_28069_amd", "csrc", "pic_plan.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "emulated_launchers.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "sanitize_driver.cpp")]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("no clang++ in this image")
    out = tmp_path_factory.mktemp("san")
    flags = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *SAN, "-fno-sanitize-recover=all",
             "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{os.path.join(ROOT, 'include')}",
             f"-I{os.path.join(ROOT, 'paper_2607_28069_amd', 'csrc')}"]
    objs = []
    for src in SOURCES:
        obj = str(out / (os.path.basename(src) + ".o"))
        r = subprocess.run([CLANG, *flags, "-c", src, "-o", obj], capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-3000:]
        objs.append(obj)
    exe = str(out / "sanitize_driver")
    r = subprocess.run([CLANG, *SAN, *objs, "-o", exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=600, env=env)


@pytest.mark.parametrize("seed", ["1", "2", "3"])
def test_host_library_clean_under_asan_and_ubsan(driver, seed):
    r = _run(driver, seed, "3")
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "sanitizer driver: OK" in r.stdout


def test_planted_short_buffer_is_caught(driver):
    r = _run(driver, "--plant")
    assert r.returncode != 0
    assert "AddressSanitizer: heap-buffer-overflow" in r.stderr
