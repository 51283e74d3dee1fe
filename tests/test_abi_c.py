"""The header as plain C: it compiles under -std=c99 -pedantic -Werror, its
struct layouts equal the Python binding's ctypes layouts field by field, and
a C program linked against libmassive.so gets the documented status codes
from argument errors (no GPU needed)."""
import ctypes
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "abi_from_c.c")

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")


def compile_and_run(tmp_path, link):
    from paper_2410_22697_amd import massive
    exe = str(tmp_path / "abi_from_c")
    cmd = ["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           SRC, "-o", exe]
    if link:
        libdir = os.path.dirname(massive.LIB_PATH)
        cmd += ["-L", libdir, "-l:libmassive.so", "-Wl,-rpath," + libdir]
    else:
        cmd += ["-Wl,--unresolved-symbols=ignore-all"]
    subprocess.check_call(cmd)
    out = subprocess.run([exe] + (["errors"] if link else []), capture_output=True, text=True, timeout=120,
                         check=True).stdout
    rows = {}
    for line in out.splitlines():
        a, b, *rest = line.split()
        rows[(a, b)] = tuple(int(x) for x in rest)
    return rows


def test_struct_layouts_match_the_binding(tmp_path):
    from paper_2410_22697_amd import massive
    rows = compile_and_run(tmp_path, link=False)
    for cname, py in (("massive_init_args", massive.InitArgs), ("massive_batch", massive.Batch)):
        assert rows[(cname, "sizeof")][0] == ctypes.sizeof(py), cname
        names = [f[0] for f in py._fields_]
        assert names == [b for (a, b) in rows if a == cname and b != "sizeof"], cname
        for f, t in py._fields_:
            assert rows[(cname, f)] == (getattr(py, f).offset, ctypes.sizeof(t)), (cname, f)


def test_error_codes_from_c(tmp_path):
    from paper_2410_22697_amd import massive
    if not os.path.exists(massive.LIB_PATH):
        pytest.skip("libmassive.so not built")
    rows = compile_and_run(tmp_path, link=True)
    assert rows[("err", "init_null_args")] == (massive.EINVAL, 1)  # and *out set to NULL
    assert rows[("err", "last_error_set")] == (1,)
    assert rows[("err", "sample_null_ctx")] == (massive.EINVAL,)
    assert rows[("err", "destroy_null_ctx")] == (massive.OK,)
