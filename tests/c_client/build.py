"""Compile the plain C client of libpda.so (a test program: it links the
oracle for its expected values).  The binary sits beside its source and finds
both libraries relative to itself, so the tree can move."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "pda_c_client.c")
BIN = os.path.join(HERE, "pda_c_client")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           "-o", BIN + ".tmp", SRC,
           "-L", os.path.join(ROOT, "paper_2405_11143_amd"), "-lpda",
           "-L", os.path.join(ROOT, "oracle"), "-lpda_oracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2405_11143_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    build(verbose=True)
