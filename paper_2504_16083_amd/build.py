"""Build libmmi.so (gfx950) in-tree: hipcc on every csrc/*.hip, then link."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(os.path.dirname(HERE), "_build")
LIB = os.path.join(HERE, "libmmi.so")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         # no packed-fp32 instructions from the compiler
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd)}\n{err}")
    return err


# The same library with AddressSanitizer on the host code only (the GPU code
# is built as usual): a test build for the runtime's validation, layout and
# plan code, loaded with the ASan runtime preloaded.
ASAN_DIR = os.path.join(OBJ, "asan")
ASAN_LIB = os.path.join(HERE, "libmmi_asan.so")
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def build(verbose: bool = False, asan: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    obj_dir, lib, extra = (ASAN_DIR, ASAN_LIB, ASAN_FLAGS) if asan else (OBJ, LIB, [])
    os.makedirs(obj_dir, exist_ok=True)
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    objs = [os.path.join(obj_dir, f[:-4] + ".o") for f in srcs]
    jobs = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")))
    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        futs = [ex.submit(_run, [hipcc, *FLAGS, *extra, "-c", os.path.join(CSRC, s), "-o", o])
                for s, o in zip(srcs, objs)]
        for f in futs:
            msg = f.result()
            if verbose and msg:
                print(msg, file=sys.stderr)
    tmp = lib + ".tmp"
    link_extra = ["-Xarch_host", "-fsanitize=address", "-shared-libsan"] if asan else ["-Wl,--no-undefined"]
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", *link_extra, "-o", tmp, *objs])
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True, asan="--asan" in sys.argv))
