"""CPU tests of the C-ABI boundary: the library builds, loads, exports every
symbol the header declares, the binding mirrors them by name, and the
oracle and the HIP path share no code.  No device work is issued."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "symtile.h")
DEVICE_HEADER = os.path.join(ROOT, "include", "symtile_device.h")
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


def test_device_api_header_is_part_of_the_boundary():
    """The device-side API (Section 3.3 device API table) is the header-only
    include/symtile_device.h: translate, value load/store, tile put/get/copy,
    the eight atomics with ordering and scope, and the per-tile flag verbs;
    every kernel source of the library includes it from there (no private
    copy under the package)."""
    assert os.path.exists(DEVICE_HEADER)
    text = open(DEVICE_HEADER).read()
    for verb in ("translate", "load", "store", "put", "get", "copy", "atomic_add", "atomic_xchg",
                 "atomic_cas", "atomic_and", "atomic_or", "atomic_xor", "atomic_min",
                 "atomic_max", "flag_publish", "flag_wait"):
        assert re.search(r"__device__ __forceinline__ [\w:<>* ]+\b%s\(" % verb, text), verb
    csrc = os.path.join(PKG, "csrc")
    assert not os.path.exists(os.path.join(csrc, "symtile_device.h"))
    from paper_2511_12500_amd.build import SOURCES
    for src in SOURCES:
        assert '#include "symtile_device.h"' in open(os.path.join(csrc, src)).read(), src


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


def test_gas_config_mirror_matches_the_header(tmp_path):
    """The binding's GasConfig has the size and field offsets of
    symtile_gas_config as a C compiler lays it out from the header."""
    import shutil
    import subprocess
    from paper_2511_12500_amd._binding import GasConfig
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    names = [f[0] for f in GasConfig._fields_]
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "symtile.h"\nint main(void) {\n'
        '  printf("size %zu\\n", sizeof(symtile_gas_config));\n' +
        "".join(f'  printf("{n} %zu\\n", offsetof(symtile_gas_config, {n}));\n' for n in names) +
        "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    out = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                        check=True).stdout.splitlines())
    assert int(out["size"]) == ctypes.sizeof(GasConfig)
    for n in names:
        assert int(out[n]) == getattr(GasConfig, n).offset, n


def test_split_k_workspace_size_is_host_only(libpath):
    """Two uint32 counters per tile rounded up to 256 bytes, then split_k fp32
    partial tiles per tile; 0 without a split; argument errors."""
    import paper_2511_12500_amd as pkg
    ws = pkg.symtile_gas_workspace_bytes
    assert ws(8192, 1024, 256, 256, 2) == 1024 + 128 * 2 * 256 * 256 * 4
    assert ws(1024, 1024, 256, 256, 16) == 256 + 16 * 16 * 256 * 256 * 4
    assert ws(300, 136, 128, 128, 3) == 256 + 6 * 3 * 128 * 128 * 4
    assert ws(3000, 3000, 64, 64, 2) == (47 * 47 * 8 + 255) // 256 * 256 + 47 * 47 * 2 * 64 * 64 * 4
    assert ws(4096, 3584, 256, 224, 2) == 2048 + 256 * 2 * 256 * 224 * 4
    for split in (0, 1):
        assert ws(8192, 1024, 256, 256, split) == 0
    assert ws(0, 1024, 256, 256, 2) == 0                   # no tiles: nothing to keep
    for bad in ((8192, 1024, 256, 256, 65), (8192, 1024, 256, 256, -1),
                (8192, 1024, 32, 32, 2), (-1, 1024, 256, 256, 2)):
        with pytest.raises(pkg.SymtileError) as e:
            ws(*bad)
        assert e.value.name == "EINVAL", bad
