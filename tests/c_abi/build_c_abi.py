"""Builds the pure-C test program of the C ABI (cifar_quick_c) against the
in-tree libcnn.so and liboracle.so; rpaths are relative to the program, so the
tree can move."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
PROGRAM = os.path.join(HERE, "cifar_quick_c")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(ROOT, 'oracle')}", f"-I{ROCM}/include",
           os.path.join(HERE, "cifar_quick_c.c"), "-o", PROGRAM + ".tmp",
           f"-L{os.path.join(ROOT, 'paper_1511_07376_amd')}", "-l:libcnn.so",
           f"-L{os.path.join(ROOT, 'oracle')}", "-l:liboracle.so", f"-L{ROCM}/lib", "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_1511_07376_amd:$ORIGIN/../../oracle:" + f"{ROCM}/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(PROGRAM + ".tmp", PROGRAM)
    return PROGRAM


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
