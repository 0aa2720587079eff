"""Build libsobek_hip.so in-tree.

1. Embed csrc/device/prelude.hip (hand-written device code) into the library as
   a string; the library prepends it to every generated plan and compiles the
   result with hipRTC for gfx950.  csrc/device/gemm_bf16.hip is embedded the same
   way and appended to the plans built with the bf16 GEMM option.
2. Compile the host runtime (C ABI, plan builder, kernel generator, hipRTC
   driver) into paper_2607_18074_amd/libsobek_hip.so.
3. Optionally pre-compile the kernels of the given operator signatures into the
   on-disk code-object cache (paper_2607_18074_amd/_jitcache/), so a GPU process
   loads them instead of compiling.  This needs no GPU.
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsobek_hip.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SOURCES = ["api.cpp", "plan.cpp", "tables.cpp", "jit.cpp"]


def _embed(name, delim):
    src = os.path.join(CSRC, "device", name + ".hip")
    with open(src) as f:
        text = f.read()
    assert f"){delim}\"" not in text
    out = os.path.join(CSRC, name + "_embed.inc")
    content = f'R"{delim}(\n{text}\n){delim}"\n'
    if not os.path.exists(out) or open(out).read() != content:
        with open(out, "w") as f:
            f.write(content)


def embed_prelude():
    _embed("prelude", "SOBEKPRELUDE")
    _embed("gemm_bf16", "SOBEKBF16")


def build_library(verbose=False):
    embed_prelude()
    cmd = ["g++", "-O2", "-g", "-std=c++17", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
           f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", "-Wall", "-Wno-unused-function",
           *[os.path.join(CSRC, s) for s in SOURCES],
           f"-L{ROCM}/lib", "-lamdhip64", "-lhiprtc", f"-Wl,-rpath,{ROCM}/lib", "-o", LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _compile_one(sig):
    sys.path.insert(0, ROOT)
    from paper_2607_18074_amd import _lib
    _lib.jit_compile(*sig)
    return sig


def prewarm(signatures, jobs=None, groups=False):
    """JIT-compile kernels for (irreps_in, lmax, irreps_out, K[, layout, norm]) signatures.

    Each signature compiles in a process of its own (hipRTC holds one compilation per
    process at a time); the code-object cache publishes every result atomically.
    groups: also the per-output-group state kernels (the per-group scratch policy).
    """
    import multiprocessing as mp
    jobs = jobs or max(1, min(len(signatures), 4, os.cpu_count() or 1))
    old = os.environ.get("SOBEK_JIT_GROUPS")
    os.environ["SOBEK_JIT_GROUPS"] = "1" if groups else "0"
    try:
        if jobs == 1:
            for sig in signatures:
                _compile_one(sig)
            return
        with mp.get_context("spawn").Pool(jobs) as pool:
            for _ in pool.imap_unordered(_compile_one, signatures):
                pass
    finally:
        if old is None:
            del os.environ["SOBEK_JIT_GROUPS"]
        else:
            os.environ["SOBEK_JIT_GROUPS"] = old


def prune_cache(since):
    """Delete code objects of the in-tree cache that no compile or cache hit touched since `since`."""
    import glob
    removed = 0
    for f in glob.glob(os.path.join(HERE, "_jitcache", "sobek_*.co")):
        if os.path.getmtime(f) < since - 1.0:
            os.remove(f)
            removed += 1
    return removed


if __name__ == "__main__":
    build_library(verbose=True)
    print("built", LIB)
