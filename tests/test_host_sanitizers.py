"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Builds the library with its host code instrumented (the device code as
usual) and the oracle with the same compiler and sanitizers, then runs the
host-side test modules against those builds in a child process with the
sanitizer runtime preloaded.  Any sanitizer report fails the test: out of
bounds or use-after-free in the layouts, the planner, the relabeling or the
oracle, signed overflow, invalid enum values passed through the C ABI, and
the like.  No device work (the planner's plans are exported and replayed on
the host).
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang"

pytestmark = pytest.mark.spawns

# host-side modules only (the GPU modules are deselected by the marker)
MODULES = ["tests/test_library_host.py", "tests/test_scalapack_host.py", "tests/test_relabel_variants.py",
           "tests/test_oracle_pins.py", "tests/test_oracle_scalapack.py", "tests/test_plan_replay.py"]


def _load_build_script():
    import importlib.util
    spec = importlib.util.spec_from_file_location("costa_build", os.path.join(ROOT, "paper_2106_06601_amd",
                                                                              "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.slow
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    if not os.path.exists(CLANG):
        pytest.skip("no clang under /opt/rocm/llvm")
    b = _load_build_script()
    os.makedirs(BUILD, exist_ok=True)
    lib = b.build(out=os.path.join(BUILD, "libcosta_mi355x.so"), build_dir=os.path.join(BUILD, "obj"),
                  synth=False, sanitize=True)
    import oracle
    olib = oracle.build(out=os.path.join(BUILD, "liboracle.so"), cc=CLANG,
                        extra=["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                               "-fno-omit-frame-pointer", "-shared-libsan"])
    log = str(tmp_path / "san")
    opts = f"halt_on_error=1:log_path={log}"
    env = dict(os.environ, LD_PRELOAD=b.sanitizer_runtime(), COSTA_LIB=lib, COSTA_ORACLE_LIB=olib,
               ASAN_OPTIONS="detect_leaks=0:" + opts, UBSAN_OPTIONS="print_stacktrace=1:" + opts)
    # the full-size plans, the short-walk layouts and the larger random cases are left to the
    # uninstrumented run; everything else runs instrumented
    r = subprocess.run([sys.executable, "-m", "pytest", *MODULES, "-q", "-x", "-m", "not gpu and not slow",
                        "-p", "no:cacheprovider", "-k", "not full_size and not short_row_walks"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=1200)
    reports = sorted(glob.glob(log + "*"))
    text = "".join(open(f).read()[:4000] for f in reports)
    assert not reports, f"sanitizer reports:\n{text}"
    assert r.returncode == 0, r.stdout[-4000:]
