"""The library's host code (argument checks, planning, workspace sizing, error reporting)
under AddressSanitizer and UndefinedBehaviorSanitizer.

libsdblock.so is rebuilt with the sanitizers on its host side only (each ``-fsanitize=``
behind ``-Xarch_host``; the gfx950 device code is built as usual but never launched here), and
the host-only ABI tests (``tests/test_abi.py``: every declared symbol, workspace queries, every
shape and argument error path, the binding's loud failure without a library) run against it
in a child interpreter with the sanitizer runtime preloaded.  No call reaches a device.
"""
import glob
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_31315_amd", "csrc", "sd_block.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(_clang_asan_runtime() is None or not os.path.exists(HIPCC),
                    reason="hipcc or its AddressSanitizer runtime is missing")
def test_abi_host_code_clean_under_asan_ubsan(tmp_path):
    lib = tmp_path / "libsdblock_asan.so"
    san = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all"):
        san += ["-Xarch_host", f]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC", "-shared", *san, "-shared-libsan",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", os.path.join(ROOT, "include"), "-o", str(lib), SRC], check=True, capture_output=True)
    child = textwrap.dedent(f"""
        import sys
        sys.path.insert(0, {ROOT!r})
        import pytest
        from paper_2606_31315_amd import _lib
        _lib.LIB_PATH = {str(lib)!r}
        sys.exit(pytest.main([{os.path.join(ROOT, "tests", "test_abi.py")!r}, "-q", "-s", "-p", "no:cacheprovider",
                              "-m", "not gpu"]))
    """)
    env = dict(os.environ, LD_PRELOAD=_clang_asan_runtime(), ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", HIP_VISIBLE_DEVICES="")
    p = subprocess.run([sys.executable, "-c", child], env=env, capture_output=True, text=True, timeout=600,
                       cwd=str(tmp_path))
    report = (p.stdout + p.stderr)[-4000:]
    assert p.returncode == 0, report
    assert "runtime error" not in p.stderr and "AddressSanitizer" not in p.stderr, report
    assert " passed" in p.stdout, report
