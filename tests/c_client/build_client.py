"""Builds tests/c_client/costa_client (and libcosta_client.so, the same code
without main): the C99 client of the tests, compiled with gcc against
include/costa.h and linked against the in-tree libcosta_mi355x.so and the HIP
runtime (no C++ and no torch involved)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "costa_client.c")
OUT = os.path.join(HERE, "costa_client")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


LIB_OUT = os.path.join(HERE, "libcosta_client.so")


def build(out=None, cc="gcc", shared=False) -> str:
    """The executable, or with shared=True the library form (no main)."""
    out = out or (LIB_OUT if shared else OUT)
    lib_dir = os.path.join(ROOT, "paper_2106_06601_amd")
    # the library is found next to the tree: relative to the client when it
    # sits in tests/c_client, else by the absolute path of this tree
    rel = os.path.relpath(lib_dir, os.path.dirname(os.path.abspath(out)))
    cmd = [cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           *(["-DCOSTA_CLIENT_NO_MAIN", "-shared", "-fPIC"] if shared else []),
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", out,
           "-L", lib_dir, "-l:libcosta_mi355x.so", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,$ORIGIN/{rel}", f"-Wl,-rpath,{lib_dir}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    print(build())
    print(build(shared=True))
