"""Build the C-ABI driver tests/capi/capi_check and the internal checks
tests/capi/jacobi_check and tests/capi/gemm_check against the in-tree library."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2609_38198_amd")
CXX = os.environ.get("CXX_HOST", "g++")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "capi_check")


def _build_one(name: str, extra_includes=(), verbose: bool = True) -> str:
    src = os.path.join(HERE, name + ".cpp")
    exe = os.path.join(HERE, name)
    # host code only (the device work is all in libflashdiff.so): the host
    # compiler with the HIP runtime headers and library
    inc = []
    for d in (os.path.join(ROOT, "include"), *extra_includes, os.path.join(ROCM, "include")):
        inc += ["-I", d]
    cmd = [CXX, "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__", *inc, src,
           "-L", PKG, "-lflashdiff", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2609_38198_amd", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}",
           "-o", exe + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"{name} build failed:\n{res.stderr[-4000:]}")
    os.replace(exe + ".tmp", exe)
    if verbose:
        print(f"built {exe}")
    return exe


def build(verbose: bool = True) -> str:
    _build_one("jacobi_check", (os.path.join(PKG, "csrc"),), verbose)
    _build_one("gemm_check", (os.path.join(PKG, "csrc"),), verbose)
    return _build_one("capi_check", (), verbose)


if __name__ == "__main__":
    build()
