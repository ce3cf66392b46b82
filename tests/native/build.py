"""Build the native C-ABI driver (tests/native/step_driver): host C++ with g++, linked against the
in-tree libemb.so, the oracle's liboracle.so (the driver is a test) and the HIP runtime."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
BINARY = os.path.join(HERE, "step_driver")


def build(verbose=False):
    """Compile the driver every time (after libemb.so and liboracle.so are built); returns its path."""
    tmp = BINARY + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
           os.path.join(HERE, "step_driver.cpp"),
           "-L", os.path.join(ROOT, "paper_2110_09132_amd"), "-l:libemb.so",
           "-L", os.path.join(ROOT, "oracle"), "-l:liboracle.so",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2110_09132_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib"),
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, BINARY)
    return BINARY


if __name__ == "__main__":
    print("built", build(verbose=True))
