"""The boundary is a C ABI: both headers compile as pedantic C99 and as C++, and a C
program linked against libembx.so gets from the host-only calls what the Python binding
gets (same coefficients, byte-identical plan text), so the structs agree across
compilers. No GPU: these calls never touch the device."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INC = os.path.join(ROOT, "include")
PKG = os.path.join(ROOT, "paper_2507_01676_amd")

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")


@pytest.mark.parametrize("header", ["embx.h", "embx_fill.h"])
@pytest.mark.parametrize("lang", [["gcc", "-std=c99", "-pedantic", "-x", "c"], ["g++", "-std=c++17", "-x", "c++"]])
def test_header_compiles_alone(tmp_path, header, lang):
    src = tmp_path / "h.c"
    src.write_text(f'#include "{header}"\nint main(void) {{ return 0; }}\n')
    r = subprocess.run([lang[0], *lang[1:], "-Wall", "-Wextra", "-Werror", "-I", INC, "-fsyntax-only", str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_caller_matches_the_binding(tmp_path):
    import paper_2507_01676_amd as embx
    exe = tmp_path / "plan_from_c"
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", INC, os.path.join(ROOT, "tests", "c", "plan_from_c.c"),
                        "-L", PKG, "-lembx", f"-Wl,-rpath,{PKG}", "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stderr)
    first, rest = r.stdout.split("\n", 1)
    assert [float(x) for x in first.split()] == embx.default_beta(256)
    stats = [dict(mean_pooling=1.0, max_pooling=1, hot_rows=[], hot_freq=[], unique_frac=1.0),
             dict(mean_pooling=4.0, max_pooling=8, hot_rows=[3, 11], hot_freq=[0.5, 0.25], unique_frac=0.5),
             dict(mean_pooling=20.0, max_pooling=40, hot_rows=[], hot_freq=[], unique_frac=-1.0)]
    assert rest == embx.plan_text([1000, 50000, 7], 64, "f32", stats, 128, 4)
