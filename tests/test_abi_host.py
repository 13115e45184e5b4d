"""The C-ABI library loads, exports every declared entry point, and rejects
invalid inputs on the host before any device call (no GPU needed)."""

import ctypes
import os
import re

import pytest

from paper_1905_11722_amd import rcdp

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "rc.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(rc_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    lib = rcdp.load_library()
    names = declared_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    for st in (0, 1, -1, -2, -3, -4, -5, -6, -7, -9):
        assert rcdp.status_str(st)


def _create(n, row_ptr, col_idx, T, M):
    lib = rcdp.load_library()
    h = ctypes.c_void_p()
    rp, ci, Ta, Ma = (rcdp._i32(x) for x in (row_ptr, col_idx, T, M))
    return lib.rc_graph_create(n, rp.ctypes.data, ci.ctypes.data, Ta.ctypes.data, Ma.ctypes.data,
                               rcdp.ALLOC_FN(), rcdp.FREE_FN(), None, None, ctypes.byref(h))


@pytest.mark.parametrize("args,expected", [
    ((-1, [0], [], [], []), rcdp.E_ARG),
    ((5000, [0] * 5001, [], [1] * 5000, [1] * 5000), rcdp.E_ARG),       # more than 4096 nodes
    ((3, [1, 1, 2, 2], [1, 2], [1] * 3, [1] * 3), rcdp.E_ARG),          # row_ptr[0] != 0
    ((3, [0, 2, 1, 2], [1, 2], [1] * 3, [1] * 3), rcdp.E_ARG),          # not monotone
    ((3, [0, 1, 2, 2], [1, 3], [1] * 3, [1] * 3), rcdp.E_ARG),          # index out of range
    ((3, [0, 1, 2, 2], [1, -1], [1] * 3, [1] * 3), rcdp.E_ARG),
    ((3, [0, 1, 2, 3], [1, 2, 0], [1] * 3, [1] * 3), rcdp.E_CYCLE),     # 0 -> 1 -> 2 -> 0
    ((2, [0, 1, 1], [0], [1] * 2, [1] * 2), rcdp.E_CYCLE),              # self-loop
    ((3, [0, 1, 2, 2], [1, 2], [1, 0, 1], [1] * 3), rcdp.E_COST),
    ((3, [0, 1, 2, 2], [1, 2], [1] * 3, [1, 1, -4], ), rcdp.E_COST),
    ((2, [0, 1, 1], [1], [2 ** 31 - 1, 5], [1, 1]), rcdp.E_OVERFLOW),   # T(V) too large
    ((2, [0, 1, 1], [1], [1, 1], [2 ** 28, 2 ** 28]), rcdp.E_OVERFLOW), # M(V) too large
])
def test_graph_validation(args, expected):
    assert _create(*args) == expected


def test_null_handles():
    lib = rcdp.load_library()
    h = ctypes.c_void_p()
    t = ctypes.c_int64()
    info = rcdp.FamilyInfo()
    assert lib.rc_build_family(None, 0, 10, None, ctypes.byref(h)) == rcdp.E_ARG
    assert lib.rc_family_stats(None, ctypes.byref(info)) == rcdp.E_ARG
    assert lib.rc_solve(None, 10, 0, None, ctypes.byref(h), ctypes.byref(t), ctypes.byref(t)) == rcdp.E_ARG
    assert lib.rc_reconstruct(None, None, None, None, None, None, None, None, None) == rcdp.E_ARG
    assert lib.rc_export_table(None, 0, 0, None, None, None) == rcdp.E_ARG
    assert lib.rc_family_sets(None, None, None) == rcdp.E_ARG
    path = ctypes.c_int32()
    assert lib.rc_solution_fill_path(None, ctypes.byref(path)) == rcdp.E_ARG
    assert lib.rc_solution_trace_path(None, ctypes.byref(path)) == rcdp.E_ARG
    lib.rc_graph_free(None)
    lib.rc_family_free(None)
    lib.rc_solution_free(None)


def test_header_is_plain_c(tmp_path):
    """include/rc.h is a C ABI: it compiles as strict C99 with every warning."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = tmp_path / "use_rc.c"
    src.write_text('#include "rc.h"\nint main(void) { return (int)sizeof(rc_family_info); }\n')
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                        "-fsyntax-only", "-I", os.path.join(root, "include"), str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
