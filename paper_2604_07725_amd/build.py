"""Builds the native parts in-tree.

* ``libsevo.so``       — the HIP library (every ``csrc/*.hip`` for gfx950)
* ``libsynth_host.so`` — host twin of the synthetic-input generator (gcc)

Run ``python -m paper_2604_07725_amd.build`` or call :func:`build`.  Object
files go to ``paper_2604_07725_amd/_build``; sources are compiled in parallel.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsevo.so")
SYNTH_LIB = os.path.join(PKG, "libsynth_host.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    # packed fp32 ALU forms stay off: plain fp32 code must not be turned into them
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-Wno-unused-command-line-argument",
]


# Per-source additions.  The causal prefill attention assumes no NaN in its
# arithmetic: its masked scores are assigned -inf (which replaces a NaN score)
# and the value slots past a sequence's last key are zeroed before use.  Under
# IEEE NaN rules every fmaxf of the block max first canonicalised both MFMA
# outputs, about 40 extra VALU instructions per 64-key block on a path the
# vector ALU bounds.
EXTRA_FLAGS = {"attn_prefill.hip": ["-fno-honor-nans"]}


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libsevo)")


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "is not a recognized feature for this target" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if out.strip():
        print(out)


def build_synth() -> str:
    _run(["gcc", "-O3", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC",
          os.path.join(PKG, "synth_host.c"), "-o", SYNTH_LIB + ".tmp"])
    os.replace(SYNTH_LIB + ".tmp", SYNTH_LIB)
    return SYNTH_LIB


# Host-side sanitizers for the checking build: AddressSanitizer and
# UndefinedBehaviorSanitizer on the host code only (argument validation,
# planning, layouts), each flag scoped to the host pass; device code is built
# as in the product library.
SANITIZE_HOST_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                       "-Xarch_host", "-fno-sanitize-recover=undefined",
                       "-Xarch_host", "-fno-omit-frame-pointer"]
SANITIZED_LIB = os.path.join(PKG, "_build_sanitized", "libsevo_sanitized.so")


def build_sevo(jobs: int = 8, sanitize: bool = False) -> str:
    """Compile every csrc/*.hip for gfx950 and link libsevo.so (or, with
    ``sanitize``, the host-sanitized checking build at SANITIZED_LIB)."""
    hipcc = _hipcc()
    out_dir = os.path.dirname(SANITIZED_LIB) if sanitize else BUILD
    lib = SANITIZED_LIB if sanitize else LIB
    extra = SANITIZE_HOST_FLAGS if sanitize else []
    os.makedirs(out_dir, exist_ok=True)
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    objs = []

    def compile_one(src: str) -> str:
        obj = os.path.join(out_dir, src[:-4] + ".o")
        _run([hipcc, *HIPCC_FLAGS, *EXTRA_FLAGS.get(src, []), *extra, "-c",
              os.path.join(CSRC, src), "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(srcs)))) as ex:
        objs = list(ex.map(compile_one, srcs))
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, *objs, "-o",
          lib + ".tmp"])
    os.replace(lib + ".tmp", lib)
    return lib


def asan_runtime() -> str:
    """The clang AddressSanitizer runtime the sanitized build needs preloaded
    into a host process that was not itself built with it."""
    import glob
    root = os.path.dirname(os.path.dirname(_hipcc()))
    hits = sorted(glob.glob(os.path.join(root, "llvm", "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    if not hits:
        raise RuntimeError("clang AddressSanitizer runtime not found under " + root)
    return hits[-1]


def build(jobs: int = 8) -> None:
    build_synth()
    build_sevo(jobs)


if __name__ == "__main__":
    build(int(sys.argv[1]) if len(sys.argv) > 1 else 8)
    print("built", LIB, SYNTH_LIB)
