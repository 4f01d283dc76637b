"""The C-ABI library loads on the CPU host and exports every function that
include/gbt.h declares (no GPU work is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gbt.h")
LIB = os.path.join(ROOT, "paper_2005_09148_amd", "libgbt.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gbt_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ["gbt_quantize", "gbt_gradients", "gbt_sample", "gbt_build_hist",
                 "gbt_eval_splits", "gbt_partition", "gbt_update_leaves", "gbt_train_tree",
                 "gbt_predict"]:
        assert want in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libgbt.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    lib.gbt_abi_version.restype = ctypes.c_int32
    assert lib.gbt_abi_version() == 3


@pytest.mark.skipif(not os.path.exists(LIB), reason="libgbt.so not built")
def test_binding_signatures_cover_the_header():
    from paper_2005_09148_amd import gbt
    assert set(gbt.SIGNATURES) == set(declared_functions())


def test_oracle_is_not_imported_by_the_product():
    pkg = os.path.join(ROOT, "paper_2005_09148_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "from oracle" not in text and "import oracle" not in text, f
                assert "gbt_oracle" not in text, f
