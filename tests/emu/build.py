"""Build of the CPU emulation library (test infrastructure; never loaded by the package).

libsobek_emu.so is the library's own host code (csrc/api.cpp, plan.cpp, tables.cpp) compiled for
the host against a stand-in HIP runtime (hip/hip_runtime.h, mock_hip.cpp) and a plan compiler
that builds the generated kernels for the host (mock_jit.cpp, emu_device.h).  Outputs go to
tests/emu/_build (or _build_asan for the AddressSanitizer variant).
"""

from __future__ import annotations

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2607_18074_amd", "csrc")
CLANG = "/opt/rocm/llvm/bin/clang++"


def available():
    return os.path.exists(CLANG)


def out_dir(asan=False):
    return os.path.join(HERE, "_build_asan" if asan else "_build")


def build(asan=False, force=False):
    """Compile libsobek_emu.so (skipped when it is newer than every source); returns its path."""
    from paper_2607_18074_amd import build as pkg_build
    pkg_build.embed_prelude()   # the device prelude the plan compiler embeds (a generated header)
    out = out_dir(asan)
    lib = os.path.join(out, "libsobek_emu.so")
    units = [os.path.join(CSRC, f) for f in ("api.cpp", "plan.cpp", "tables.cpp")] + \
            [os.path.join(HERE, f) for f in ("mock_jit.cpp", "mock_hip.cpp")]
    deps = units + [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".h", ".inc"))] + \
        [os.path.join(HERE, f) for f in ("emu_rt.h", "emu_device.h", os.path.join("hip", "hip_runtime.h"))] + \
        [os.path.join(ROOT, "include", "sobek.h")]
    if not force and os.path.exists(lib) and os.path.getmtime(lib) >= max(os.path.getmtime(d) for d in deps):
        return lib
    os.makedirs(out, exist_ok=True)
    flags = ["-std=c++17", "-O1", "-g", "-fPIC", "-I" + HERE, "-I" + CSRC]
    if asan:
        flags += ["-fsanitize=address", "-fno-omit-frame-pointer"]

    def cc(src):
        obj = os.path.join(out, os.path.basename(src)[:-4] + ".o")
        r = subprocess.run([CLANG] + flags + ["-c", src, "-o", obj], capture_output=True, text=True)
        if r.returncode:
            raise RuntimeError(f"emulation build of {src} failed:\n{r.stderr[-3000:]}")
        return obj

    with ThreadPoolExecutor(max_workers=min(len(units), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(cc, units))
    link = [CLANG, "-shared"] + (["-fsanitize=address", "-shared-libasan"] if asan else []) + \
        ["-o", lib + ".tmp"] + objs + ["-ldl", "-lpthread", "-Wl,-soname,libsobek_emu.so", "-Wl,-Bsymbolic"]
    r = subprocess.run(link, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError(f"emulation link failed:\n{r.stderr[-3000:]}")
    os.replace(lib + ".tmp", lib)
    return lib


def clean():
    for asan in (False, True):
        shutil.rmtree(out_dir(asan), ignore_errors=True)


if __name__ == "__main__":
    import sys
    print(build(asan="asan" in sys.argv[1:], force="force" in sys.argv[1:]))
