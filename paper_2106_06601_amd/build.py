"""Builds libcosta_mi355x.so (the C-ABI library) in place with hipcc for gfx950.

Also builds the seeded-input fill library used by tests and benchmarks
(synth/libcosta_synth.so); the CPU oracle is built separately by oracle.build().
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libcosta_mi355x.so")
SYNTH_SRC = os.path.join(ROOT, "synth", "fill.hip")
SYNTH_LIB = os.path.join(ROOT, "synth", "libcosta_synth.so")
BUILD_DIR = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# -ffp-contract=off: no FMA contraction, so a*b + c is rounded twice exactly as written.
# packed-fp32-ops disabled: no packed fp32 instructions are generated.
COMMON = ["-O3", "-fPIC", "-std=c++17", "-ffp-contract=off",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function"]
SOURCES = ["layout.cpp", "lap.cpp", "plan.cpp", "api.cpp", "scalapack.cpp", "kernels.hip"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + out)
    return out


# Host-side sanitizers (AddressSanitizer + UndefinedBehaviorSanitizer) for the
# library's host code only: each flag is scoped to the host pass, the device
# code is compiled as usual.
SANITIZE_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def sanitizer_runtime() -> str:
    """The AddressSanitizer runtime of the compiler that builds the library
    (to be preloaded into an uninstrumented host process)."""
    import glob
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise RuntimeError("libclang_rt.asan-x86_64.so not found under /opt/rocm/llvm")
    return found[-1]


def build(verbose: bool = False, defines=(), out=None, build_dir=None, synth=True, sanitize=False) -> str:
    """defines: extra -D flags (tuning experiments); out: library path;
    sanitize: instrument the host code with ASan and UBSan."""
    lib = out or LIB
    bdir = build_dir or BUILD_DIR
    os.makedirs(bdir, exist_ok=True)
    objs = []
    jobs = []
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        obj = os.path.join(bdir, src + ".o")
        objs.append(obj)
        lang = ["-x", "hip"]
        jobs.append([HIPCC, f"--offload-arch={ARCH}", *COMMON, *(SANITIZE_HOST if sanitize else []),
                     *[f"-D{d}" for d in defines], *lang, "-c", path, "-o", obj])
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        outs = list(ex.map(_run, jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = lib + ".tmp"
    link_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"]
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *(link_san if sanitize else []), "-o", tmp, *objs])
    os.replace(tmp, lib)
    if not synth:
        return lib
    tmp = SYNTH_LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", *COMMON, "-shared", "-o", tmp, SYNTH_SRC])
    os.replace(tmp, SYNTH_LIB)
    return lib


if __name__ == "__main__":
    # python paper_2106_06601_amd/build.py [-v] [--define NAME=VALUE ...] [--out LIB]
    # (tuning switches of the kernels and planner; a library built with
    # --out elsewhere is loaded by setting COSTA_LIB to its path)
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("-v", action="store_true")
    ap.add_argument("--define", action="append", default=[])
    ap.add_argument("--out")
    a = ap.parse_args()
    out = os.path.abspath(a.out) if a.out else None
    bdir = os.path.join(BUILD_DIR, "variant_" + os.path.basename(out)) if out else None
    print(build(verbose=a.v, defines=a.define, out=out, build_dir=bdir, synth=out is None))
