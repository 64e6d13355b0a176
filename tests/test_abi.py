"""The C ABI: the library builds for gfx950, loads, exports every declared
symbol, and validates arguments on the host (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2609_38198_amd import _lib as fd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashdiff.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fd_[a-z_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("fd_degree", "fd_kernel_matmul", "fd_block_lanczos", "fd_continuation"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = fd.load()
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert set(declared_functions()) <= set(fd.EXPORTS)


def test_status_strings_and_defaults():
    lib = fd.load()
    assert lib.fd_status_string(0) == b"FD_OK"
    assert lib.fd_status_string(5) == b"FD_ERR_NOT_CONVERGED"
    o = fd.default_opts()
    assert o.tol == 1e-5 and o.max_restarts > 0


def test_workspace_sizes():
    s1 = fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, 65536, 65536, 12, 16)
    s2 = fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, 65536, 65536, 12, 32)
    assert 0 < s1 < s2
    assert fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, 10, 10, 65, 4) == 0   # D > 64
    assert fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, 10, 10, 4, 65) == 0   # b > 64
    assert fd.fd_workspace_size(fd.FD_OP_DEGREE, 1 << 20, 1 << 20, 30) > 0
    # the dyadic ladder adds the squared-kernel partial sums to the degree workspace
    assert (fd.fd_workspace_size(fd.FD_OP_DEGREE_DYADIC, 65536, 65536, 12)
            > fd.fd_workspace_size(fd.FD_OP_DEGREE, 65536, 65536, 12) > 0)
    assert fd.fd_workspace_size(fd.FD_OP_BLOCK_LANCZOS, 2048, 2048, 4, 8, 16) > 0
    assert fd.fd_workspace_size(fd.FD_OP_BLOCK_LANCZOS, 10, 10, 4, 8, 11) == 0  # k > N


def test_host_validation_without_gpu():
    lib = fd.load()
    c = ctypes.c_void_p
    # NULL X
    assert lib.fd_kernel_matmul(None, 10, None, 10, 4, 4, 0, 1.0, None, None, None, 8, 8, None, 8,
                                None, 0, None) == 1
    fake = c(256)
    # bad b, bad ldx, negative beta, unknown dtype
    assert lib.fd_kernel_matmul(fake, 10, fake, 10, 4, 4, 0, 1.0, None, None, fake, 0, 8, fake, 8,
                                None, 0, None) == 1
    assert lib.fd_kernel_matmul(fake, 10, fake, 10, 4, 3, 0, 1.0, None, None, fake, 8, 8, fake, 8,
                                None, 0, None) == 1
    assert lib.fd_kernel_matmul(fake, 10, fake, 10, 4, 4, 0, -1.0, None, None, fake, 8, 8, fake, 8,
                                None, 0, None) == 1
    assert lib.fd_kernel_matmul(fake, 10, fake, 10, 4, 4, 7, 1.0, None, None, fake, 8, 8, fake, 8,
                                None, 0, None) == 1
    # missing workspace
    assert lib.fd_kernel_matmul(fake, 10, fake, 10, 4, 4, 0, 1.0, None, None, fake, 8, 8, fake, 8,
                                None, 0, None) == 3
    # empty and degenerate sizes: no rows, no columns, no features, D > 64
    for N, Nc, D in ((0, 10, 4), (10, 0, 4), (10, 10, 0)):
        assert lib.fd_kernel_matmul(fake, N, fake, Nc, D, 4, 0, 1.0, None, None, fake, 8, 8,
                                    fake, 8, None, 0, None) == 1
    assert lib.fd_kernel_matmul(fake, 10, None, 0, 65, 65, 0, 1.0, None, None, fake, 8, 8, fake,
                                8, None, 0, None) == 2
    assert b"D above 64" in lib.fd_last_error()
    assert lib.fd_degree(fake, 0, 0, 4, 4, 1.0, 0.5, None, None, None, None, None, 0, None) == 1
    assert lib.fd_degree(fake, 0, 10, 0, 4, 1.0, 0.5, None, None, None, None, None, 0, None) == 1
    # degree: alpha out of range, beta = 0
    assert lib.fd_degree(fake, 0, 10, 4, 4, 1.0, 1.5, None, None, None, None, None, 0, None) == 1
    assert lib.fd_degree(fake, 0, 10, 4, 4, 0.0, 0.5, None, None, None, None, None, 0, None) == 1
    assert b"alpha" in lib.fd_last_error() or b"beta" in lib.fd_last_error()
    # dyadic ladder: levels outside [1, 32], beta0 <= 0, beta0 2^(nbeta-1) not finite
    # in float, alpha out of range, missing workspace
    for beta0, nb, alpha in ((1.0, 0, 0.5), (1.0, 33, 0.5), (0.0, 2, 0.5), (3e38, 3, 0.5),
                             (1.0, 2, -0.1)):
        assert lib.fd_degree_dyadic(fake, 0, 10, 4, 4, beta0, nb, alpha, None, None, None, None,
                                    None, 0, None) == 1
    assert lib.fd_degree_dyadic(fake, 0, 10, 4, 4, 1.0, 3, 0.5, None, None, None, None, None, 0,
                                None) == 3


def test_struct_layouts_match_the_header(tmp_path):
    # the ctypes mirrors of the ABI structs against a C compiler's view of the header
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"fd_lanczos_opts": fd.LanczosOpts, "fd_lanczos_info": fd.LanczosInfo,
               "fd_flow_opts": fd.FlowOpts, "fd_flow_probe": fd.FlowProbe}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "flashdiff.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'printf("{name} size %zu\\n", sizeof({name}));')
        for field, _ in cls._fields_:
            lines.append(f'printf("{name} {field} %zu\\n", offsetof({name}, {field}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for name, cls in structs.items():
        assert got[(name, "size")] == ctypes.sizeof(cls), name
        for field, _ in cls._fields_:
            assert got[(name, field)] == getattr(cls, field).offset, (name, field)


def test_flow_workspace_and_validation_without_gpu():
    assert fd.fd_workspace_size(fd.FD_OP_BETA_FLOW, 2048, 2048, 4, 8, 16) > 0
    assert fd.fd_workspace_size(fd.FD_OP_BETA_FLOW, 2048, 2048, 4, 8, 1) == 0   # k < 2
    lib = fd.load()
    fake = ctypes.c_void_p(256)
    o = fd.flow_default_opts()
    assert o.kappa == 10.0 and o.p == 6.0 and o.max_probes == 24
    recs = (fd.FlowProbe * 26)()
    n, bx, why = ctypes.c_int64(), ctypes.c_double(), ctypes.c_int32()
    ev = (ctypes.c_double * 16)()
    args = lambda k, fo: (fake, 0, 2048, 4, 4, 0.5, 8, k, ctypes.byref(fo), None, recs,
                          ctypes.byref(n), ctypes.byref(bx), ctypes.byref(why), ev, fake, None,
                          None, 0, None)
    assert lib.fd_beta_flow(*args(1, o)) == 1  # k < 2
    bad = fd.flow_default_opts(max_probes=0)
    assert lib.fd_beta_flow(*args(16, bad)) == 1
    assert lib.fd_beta_flow(*args(16, o)) == 3  # no workspace
