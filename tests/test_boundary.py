"""CPU tests of the C-ABI boundary: the library builds, loads, exports every
symbol the header declares, the binding mirrors them by name, and the
oracle and the HIP path share no code.  No device work is issued."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "symtile.h")
PKG = os.path.join(ROOT, "paper_2511_12500_amd")
LIB = os.path.join(PKG, "libsymtile.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(symtile_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def libpath():
    if not os.path.exists(LIB):
        from paper_2511_12500_amd.build import build_library
        build_library()
    return LIB


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("symtile_heap_create", "symtile_heap_alloc", "symtile_translate",
                     "symtile_gemm_all_scatter", "symtile_tile_copy", "symtile_barrier",
                     "symtile_atomic_exercise", "symtile_heap_bases"):
        assert required in names


def test_library_exports_every_declared_symbol(libpath):
    lib = ctypes.CDLL(libpath)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, f"not exported: {missing}"


def test_host_only_entry_points(libpath):
    lib = ctypes.CDLL(libpath)
    lib.symtile_version.restype = ctypes.c_char_p
    lib.symtile_last_error.restype = ctypes.c_char_p
    assert b"gfx950" in lib.symtile_version()
    assert isinstance(lib.symtile_last_error(), bytes)
    # argument validation happens before any device call
    lib.symtile_heap_alloc.restype = ctypes.c_int
    assert lib.symtile_heap_alloc(None, 16, 0, None) == -1          # EINVAL: NULL heap
    assert b"NULL" in lib.symtile_last_error()
    lib.symtile_gemm_all_scatter.restype = ctypes.c_int
    assert lib.symtile_gemm_all_scatter(*([None] * 6 + [0] * 8 + [None, None])) == -1


def test_binding_mirrors_every_symbol(libpath):
    import paper_2511_12500_amd as pkg
    missing = [n for n in declared_functions() if not callable(getattr(pkg, n, None))]
    assert not missing, f"binding lacks: {missing}"


def test_oracle_and_hip_path_share_nothing():
    hip_files = []
    for d, _, files in os.walk(PKG):
        hip_files += [os.path.join(d, f) for f in files if f.endswith((".py", ".hip", ".h"))]
    for f in hip_files:
        text = open(f).read()
        assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), f
        assert "oracle.c" not in text and "oracle/" not in text, f
    odir = os.path.join(ROOT, "oracle")
    for f in os.listdir(odir):
        if f.endswith((".py", ".c", ".h")):
            text = open(os.path.join(odir, f)).read()
            assert "paper_2511_12500_amd" not in text and "symtile" not in text, f
            assert not re.search(r"#include\s+\"", text), f


def test_product_has_no_cpu_fallback():
    """The binding loads the HIP library when first used and raises if it is
    absent; the build module imports without it."""
    src = open(os.path.join(PKG, "_binding.py")).read()
    assert "raise ImportError" in src
    assert "lib = _load()" in src


def test_build_module_imports_without_the_library(tmp_path):
    import shutil
    import subprocess
    import sys
    dst = tmp_path / "paper_2511_12500_amd"
    shutil.copytree(PKG, dst, ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    code = ("import paper_2511_12500_amd as p, paper_2511_12500_amd.build as b; "
            "assert b.SOURCES\n"
            "try:\n    p.Heap\nexcept ImportError as e:\n    print('raised', e)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=tmp_path, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert "raised" in r.stdout and "not built" in r.stdout
