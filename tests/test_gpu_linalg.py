"""The tall-skinny products of the eigensolver against float64 sums on the host.

C = A^T B (float64 sums of float32 products, on the float64 matrix unit) and
Z = beta Z + alpha Q C (float32) are internal to libflashdiff.so; the C++
driver tests/capi/gemm_check.cpp calls them on shapes that take every load
path (vector and scalar loads, one to four 16-column blocks per wave, partly
used blocks, several column tiles, 16, 32 and 64 rows per wave, ragged row
counts, offset and odd leading dimensions, up to 2^18 + 3 rows and a
1024-column basis) and compares each result with the host's float64 sum
within the bound of the two summation orders.  It also checks the block
Cholesky and inverse (fd::chol_rinv) on full-rank and rank-deficient Gram
matrices.
"""
import os
import subprocess

import pytest

from gpu_util import case

pytestmark = pytest.mark.gpu

GEMM_CHECK = os.path.join(os.path.dirname(os.path.abspath(__file__)), "capi", "gemm_check")


def test_tall_skinny_products_match_float64_sums():
    case("gemm_tn / gemm_nn edge shapes against host float64 sums")
    assert os.path.exists(GEMM_CHECK), "gemm_check is not built (run __graft_entry__.build())"
    res = subprocess.run([GEMM_CHECK], capture_output=True, text=True, timeout=110)
    print(res.stdout)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.count(": ok") == 31 and "all ok" in res.stdout, res.stdout
