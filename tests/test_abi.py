"""The C-ABI library loads and exports every entry point include/ee.h declares
(CPU only: no compute calls). Also checks the binding mirrors the names."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ee.h")
LIB = os.path.join(ROOT, "paper_2609_14144_amd", "libee.so")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ee_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for s in ("ee_create", "ee_load_weights", "ee_prefill", "ee_decode_step", "ee_decode_n",
              "ee_calibrate_threshold", "ee_reset", "ee_last_error", "ee_destroy"):
        assert s in syms


@pytest.mark.skipif(not os.path.exists(LIB), reason="libee.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [s for s in declared_symbols() if not hasattr(lib, s)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="libee.so not built")
def test_binding_mirrors_abi_names():
    import paper_2609_14144_amd as pkg
    methods = set(dir(pkg.Engine))
    for s in declared_symbols():
        if s in ("ee_create", "ee_destroy"):
            continue
        assert s in methods, s


def test_header_compiles_as_c():
    import shutil
    import subprocess
    import tempfile
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("no gcc")
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "t.c")
        with open(src, "w") as f:
            f.write('#include "ee.h"\nint main(void){ee_config c; (void)c; return EE_OK;}\n')
        subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER), src,
                        "-o", os.path.join(d, "t")], check=True)
