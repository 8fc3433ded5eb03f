"""Compile tests/c_abi/erc_example.c into tests/c_abi/liberc_example.so with gcc: plain
C99 against include/erc.h and the HIP runtime, linked to the package's liberc.so (found
next to it at run time through a relative rpath).  Called by __graft_entry__.build()
after the library is built; the GPU test loads the result with ctypes."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "liberc_example.so")


def build(verbose: bool = False) -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    pkg = os.path.join(ROOT, "paper_2609_27209_amd")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-shared", "-fPIC",
           "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(ROOT, 'include')}",
           f"-I{os.path.join(rocm, 'include')}", os.path.join(HERE, "erc_example.c"),
           f"-L{pkg}", "-lerc", "-Wl,-rpath,$ORIGIN/../../paper_2609_27209_amd",
           f"-L{os.path.join(rocm, 'lib')}", "-lamdhip64",
           f"-Wl,-rpath,{os.path.join(rocm, 'lib')}", "-lm", "-o", OUT + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("building the C example failed")
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
