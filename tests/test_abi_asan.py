"""The C ABI's host-side code under AddressSanitizer (CPU only).

The library is rebuilt with the host half instrumented (device code is built as usual), and the
host-side ABI tests (exports, argument checks, workspace queries, error strings) run against it
in a child process with the ASan runtime preloaded.  Any heap or stack error in the host code
that those calls reach aborts the child with an AddressSanitizer report.
"""
import glob
import os
import subprocess
import sys

import pytest

from paper_2609_16450_amd import build as eb_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    pats = ["/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so",
            "/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"]
    for pat in pats:
        hits = sorted(glob.glob(pat))
        if hits:
            return hits[-1]
    return None


def test_host_code_is_clean_under_asan(tmp_path):
    try:
        hipcc = eb_build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not found")
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("ASan runtime not found")
    lib = str(tmp_path / "libeb_asan.so")
    # host-only instrumentation: every -fsanitize flag goes to the host compile
    cmd = [hipcc, *eb_build.HIPCC_FLAGS,
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
           "-shared-libasan", "-I", os.path.join(ROOT, "include"),
           *[os.path.join(eb_build.CSRC, s) for s in eb_build.SOURCES], "-o", lib]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert res.returncode == 0, res.stderr[-2000:]
    driver = tmp_path / "run_abi.py"
    driver.write_text(
        "import sys\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "import pytest\n"
        "import paper_2609_16450_amd.binding as B\n"
        f"B._LIB_PATH = {lib!r}\n"
        "code = pytest.main(['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu',\n"
        f"                   {os.path.join(ROOT, 'tests', 'test_abi.py')!r}])\n"
        "import ctypes\n"
        "lib = B.load()\n"
        "assert B._LIB_PATH.endswith('libeb_asan.so')\n"
        "ctypes.CDLL(None).__asan_init  # the ASan runtime is loaded\n"
        "sys.exit(int(code))\n")
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    res = subprocess.run([sys.executable, str(driver)], capture_output=True, text=True,
                         timeout=600, env=env, cwd=str(tmp_path))
    out = res.stdout + res.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in out
