"""The runtime's host code under AddressSanitizer: the library built with ASan
on its host code only (paper_2504_16083_amd/build.py, ASAN_LIB; the GPU
code unchanged) runs in a subprocess with the ASan runtime preloaded, on the
CPU, through every host-side validation case of the C-ABI (shapes, strides,
head configs, modality layouts, key-layout and tile limits). A heap or stack
error in that code aborts the subprocess. (Not run in a GPU process: the
ASan runtime also intercepts the HSA device allocator there.)"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))


def _asan_env():
    from paper_2504_16083_amd import build as B
    if not os.path.exists(B.ASAN_LIB):
        pytest.skip("host-ASan build missing: run __graft_entry__.build()")
    rt = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True).stdout.strip()
    if not os.path.exists(rt):
        pytest.skip("ASan runtime not found")
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1")
    return B.ASAN_LIB, env


def _run(code, timeout):
    lib, env = _asan_env()
    prog = (f"import sys; sys.path.insert(0, {ROOT!r}); sys.path.insert(0, {HERE!r})\n"
            f"from paper_2504_16083_amd import mmi\nmmi.LIB_PATH = {lib!r}\nmmi.lib()\n"
            # the sanitizer runtime and the sanitized library are the ones mapped
            f"maps = open('/proc/self/maps').read()\n"
            f"assert 'libclang_rt.asan' in maps and {lib!r} in maps\n" + code + "\nprint('asan-run-ok')\n")
    r = subprocess.run([sys.executable, "-c", prog], env=env, capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0 and "asan-run-ok" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-4000:])


def test_validation_under_asan():
    _run("import test_abi\n"
         "test_abi.test_every_declared_symbol_is_exported()\n"
         "test_abi.test_struct_sizes_match_header()\n"
         "test_abi.test_validation_codes_without_device()\n"
         "test_abi.test_search_arguments_without_device()\n", timeout=300)

