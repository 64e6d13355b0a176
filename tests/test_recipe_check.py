"""The compile-time proof of the split-exponent layouts accepts the shipped
table and rejects planted mistakes.

The float32 path evaluates the Gram-form exponent (Sec. 2.2, eq. rbf_gram) as
a float16 matrix-core contraction over pieces of the coordinates; a table of
"recipes" says which piece sits in which slot, and a `constexpr` check in the
HIP source proves at compile time that each recipe contracts the intended sum
(every wanted piece product once per feature, every wanted offset piece once,
nothing else).  This test compiles that table and check as plain C++17 on the
host, then plants one mistake at a time (a wrong piece, a dropped instruction,
a wrong chunk pairing, a short split claiming to be exact, a shifted feature)
and requires each to fail the check.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2609_38198_amd", "csrc", "hx_kernels.hip")

MUTATIONS = [
    # x2 b2 in place of x1 b2 (D <= 8)
    ("{8, 1, 1, 1, 3, {0}, {0},\n     {{{{X(1, 0, 8), X(2, 8, 8), X(1, 16, 8)",
     "{8, 1, 1, 1, 3, {0}, {0},\n     {{{{X(1, 0, 8), X(2, 8, 8), X(2, 16, 8)"),
    # one instruction dropped (D <= 13)
    ("{13, 2, 2, 2, 3, {0, 1}, {0, 1}", "{13, 2, 2, 1, 3, {0, 1}, {0, 1}"),
    # wrong column chunk for an instruction (D <= 30)
    ("{30, 2, 2, 3, 3, {0, 1, 0}, {0, 0, 1}", "{30, 2, 2, 3, 3, {0, 1, 1}, {0, 0, 1}"),
    # a short split declared exact (D <= 32)
    ("{32, 3, 3, 4, 3, {0, 2, 1, 0}, {0, 2, 0, 1}", "{32, 3, 3, 4, 4, {0, 2, 1, 0}, {0, 2, 0, 1}"),
    # features of the second x1 chunk shifted by one (D <= 64, column side)
    ("{{{{X(1, 0, 32)}}, {{X(1, 0, 32, 32)}}, {{X(2, 0, 32)}}, {{X(2, 0, 32, 32)}},\n       {{ONES(0), AOF(3)}}}}",
     "{{{{X(1, 0, 32)}}, {{X(1, 0, 32, 31)}}, {{X(2, 0, 32)}}, {{X(2, 0, 32, 32)}},\n       {{ONES(0), AOF(3)}}}}"),
]


def _table_source():
    src = open(SRC).read()
    a = src.index("enum : int8_t { SEG_END")
    b = src.index("template <int RID>\nstruct Hx {")
    return "#include <cstdint>\n" + src[a:b] + "\nint main() { return 0; }\n"


def _compiles(code, tmp_path, name):
    path = tmp_path / f"{name}.cpp"
    path.write_text(code)
    res = subprocess.run([shutil.which("g++") or "g++", "-std=c++17", "-fsyntax-only", str(path)],
                         capture_output=True, text=True)
    return res.returncode == 0, res.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs a host C++ compiler")
def test_shipped_recipes_pass_and_planted_mistakes_fail(tmp_path):
    code = _table_source()
    ok, err = _compiles(code, tmp_path, "shipped")
    assert ok, err[-2000:]
    for k, (old, new) in enumerate(MUTATIONS):
        assert code.count(old) == 1, f"mutation {k} no longer matches the table"
        ok, _ = _compiles(code.replace(old, new), tmp_path, f"mut{k}")
        assert not ok, f"planted mistake {k} passed the recipe check"
