"""Build the C-ABI driver tests/capi/capi_check against the in-tree library."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2609_38198_amd")
CXX = os.environ.get("CXX_HOST", "g++")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "capi_check")


def build(verbose: bool = True) -> str:
    src = os.path.join(HERE, "capi_check.cpp")
    # host code only (the device work is all in libflashdiff.so): the host
    # compiler with the HIP runtime headers and library
    cmd = [CXX, "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), src,
           "-L", PKG, "-lflashdiff", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2609_38198_amd", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}",
           "-o", EXE + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"capi_check build failed:\n{res.stderr[-4000:]}")
    os.replace(EXE + ".tmp", EXE)
    if verbose:
        print(f"built {EXE}")
    return EXE


if __name__ == "__main__":
    build()
