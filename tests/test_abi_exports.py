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
    assert lib.gbt_abi_version() == 7


@pytest.mark.skipif(not os.path.exists(LIB), reason="libgbt.so not built")
def test_binding_signatures_cover_the_header():
    from paper_2005_09148_amd import gbt
    assert set(gbt.SIGNATURES) == set(declared_functions())


def test_binding_fails_loudly_without_the_library(tmp_path):
    # a copy of the binding whose package holds no libgbt.so must refuse to
    # import (there is no fallback path that would run without the kernels)
    import shutil
    import subprocess
    import sys
    pkg = tmp_path / "gbtcopy"
    pkg.mkdir()
    (pkg / "__init__.py").write_text("")
    shutil.copy(os.path.join(ROOT, "paper_2005_09148_amd", "gbt.py"), pkg / "gbt.py")
    r = subprocess.run([sys.executable, "-c", "import gbtcopy.gbt"], cwd=tmp_path, capture_output=True, text=True)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "is not built" in r.stderr


def test_oracle_is_not_imported_by_the_product():
    pkg = os.path.join(ROOT, "paper_2005_09148_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "from oracle" not in text and "import oracle" not in text, f
                assert "gbt_oracle" not in text, f


def _c_layout(names):
    """sizeof and the #define/enum constants of include/gbt.h, from a C
    program compiled with the host compiler."""
    import subprocess
    import tempfile
    structs = [s for s, _ in names]
    consts = ["GBT_E_INVALID", "GBT_E_OOM", "GBT_E_BUDGET", "GBT_E_DEVICE", "GBT_E_UNSUPPORTED", "GBT_E_IO",
              "GBT_HOME_DEVICE", "GBT_HOME_PINNED_HOST", "GBT_HOME_DISK", "GBT_COMPACT_AUTO",
              "GBT_COMPACT_STREAM", "GBT_COMPACT_GATHER", "GBT_SAMPLE_MVS", "GBT_SAMPLE_SGB", "GBT_SAMPLE_GOSS",
              "GBT_HIST_AUTO", "GBT_HIST_PLAIN", "GBT_HIST_ROTATED"]
    body = "".join(f'printf("{s} %zu\\n", sizeof({s}));' for s in structs)
    body += "".join(f'printf("{k} %d\\n", (int)({k}));' for k in consts)
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "layout.c"), os.path.join(d, "layout")
        with open(src, "w") as fh:
            fh.write('#include <stdio.h>\n#include "gbt.h"\nint main(void){' + body + "return 0;}\n")
        subprocess.run(["gcc", "-std=c11", "-I", os.path.dirname(HEADER), src, "-o", exe], check=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    return dict((k, int(v)) for k, v in (line.split() for line in out.splitlines()))


def test_binding_layouts_and_constants_match_the_header():
    # the ctypes mirrors of the header's structs and constants (host logic:
    # a layout drift would pass garbage through the boundary)
    from paper_2005_09148_amd import gbt
    pairs = [("gbt_input", gbt.Input), ("gbt_quant_params", gbt.QuantParams),
             ("gbt_matrix_info", gbt.MatrixInfo), ("gbt_train_params", gbt.TrainParams),
             ("gbt_seg", gbt.Seg), ("gbt_sub", gbt.Sub), ("gbt_split", gbt.Split), ("gbt_tree", gbt.Tree),
             ("gbt_tree_stats", gbt.TreeStats), ("gbt_sample_params", gbt.SampleParams),
             ("gbt_sampled_info", gbt.SampledInfo)]
    c = _c_layout(pairs + [("gbt_node", None)])
    for name, cls in pairs:
        assert c[name] == ctypes.sizeof(cls), name
    assert c["gbt_node"] == gbt.NODE_DTYPE.itemsize and c["gbt_split"] == gbt.SPLIT_DTYPE.itemsize
    assert c["gbt_seg"] == gbt.SEG_DTYPE.itemsize
    # the numpy form of gbt_tree that gbt_train_trees passes as an array
    assert c["gbt_tree"] == gbt._TREE_DTYPE.itemsize
    for f, _ in gbt.Tree._fields_:
        assert gbt._TREE_DTYPE.fields[f][1] == getattr(gbt.Tree, f).offset, f
    py = {"GBT_E_INVALID": gbt.GBT_E_INVALID, "GBT_E_OOM": gbt.GBT_E_OOM, "GBT_E_BUDGET": gbt.GBT_E_BUDGET,
          "GBT_E_DEVICE": gbt.GBT_E_DEVICE, "GBT_E_UNSUPPORTED": gbt.GBT_E_UNSUPPORTED, "GBT_E_IO": gbt.GBT_E_IO,
          "GBT_HOME_DEVICE": gbt.HOME_DEVICE, "GBT_HOME_PINNED_HOST": gbt.HOME_PINNED_HOST,
          "GBT_HOME_DISK": gbt.HOME_DISK, "GBT_SAMPLE_MVS": gbt.SAMPLE_MVS, "GBT_SAMPLE_SGB": gbt.SAMPLE_SGB,
          "GBT_SAMPLE_GOSS": gbt.SAMPLE_GOSS, "GBT_COMPACT_AUTO": gbt.Context.COMPACT_AUTO,
          "GBT_COMPACT_STREAM": gbt.Context.COMPACT_STREAM, "GBT_COMPACT_GATHER": gbt.Context.COMPACT_GATHER,
          "GBT_HIST_AUTO": gbt.Context.HIST_AUTO, "GBT_HIST_PLAIN": gbt.Context.HIST_PLAIN,
          "GBT_HIST_ROTATED": gbt.Context.HIST_ROTATED}
    for k, v in py.items():
        assert c[k] == v, k
