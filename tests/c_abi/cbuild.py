"""Compile the plain-C caller of the C ABI (tests/c_abi/fbl_c_caller.c) with
gcc -std=c11 against include/fbl.h and the built libfbl.so.  Test
infrastructure: the GPU test runs the binary this writes."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "fbl_c_caller.c")
OUT = os.path.join(HERE, "build", "fbl_c_caller")


def command(out: str, rpath: str) -> list:
    return ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic", "-D__HIP_PLATFORM_AMD__",
            "-I", os.path.join(ROOT, "include"), "-isystem", "/opt/rocm/include", SRC, "-o", out,
            "-L", os.path.join(ROOT, "paper_2607_21624_amd"), "-l:libfbl.so", "-L", "/opt/rocm/lib", "-lamdhip64",
            f"-Wl,-rpath,{rpath}", "-Wl,-rpath,/opt/rocm/lib"]


def build(out: str = OUT, verbose: bool = False) -> str:
    os.makedirs(os.path.dirname(out), exist_ok=True)
    # the library is found next to the package, relative to the binary
    rel = os.path.relpath(os.path.join(ROOT, "paper_2607_21624_amd"), os.path.dirname(out))
    cmd = command(out, "$ORIGIN/" + rel)
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("gcc failed building the C caller")
    return out


if __name__ == "__main__":
    print(build(verbose=True))
