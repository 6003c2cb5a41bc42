"""Builds tests/abi_c/layer_main, a plain-C caller of libomnimoe.so (host compiler only)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BIN = os.path.join(HERE, "layer_main")


def build(verbose: bool = False) -> str:
    lib_dir = os.path.join(ROOT, "paper_2602_05711_amd")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(rocm, "include"), os.path.join(HERE, "layer_main.c"),
           "-o", BIN, "-L", lib_dir, "-lomnimoe", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath," + lib_dir, "-Wl,-rpath," + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return BIN


if __name__ == "__main__":
    build(verbose=True)
