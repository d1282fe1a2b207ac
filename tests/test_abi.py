"""The library builds, loads and exports every entry point its header declares
(no GPU needed: nothing is called)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wfstdec.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wd_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def libpath():
    from paper_1804_03243_amd import wfstdec
    if not os.path.exists(wfstdec.LIB_PATH):
        from paper_1804_03243_amd import build
        build.build()
    return wfstdec.LIB_PATH


def test_header_declares_the_documented_entry_points():
    names = declared()
    for n in ("wd_graph_bytes", "wd_graph_load", "wd_graph_free", "wd_workspace_bytes", "wd_decode",
              "wd_decode_batch", "wd_result_lattice", "wd_result_words", "wd_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(libpath):
    lib = ctypes.CDLL(libpath)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing
    out = subprocess.run(["nm", "-D", "--defined-only", libpath], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (wd_[a-z_]+)\b", out))
    assert set(declared()) <= exported


def test_binding_names_match_header():
    from paper_1804_03243_amd import wfstdec
    assert set(wfstdec.EXPORTS) == set(declared())
    for n in declared():
        if n.startswith(("wd_result_", "wd_clat_")) and n not in ("wd_result_free",):
            continue  # accessors, read by wd_result_read / wd_lattice_determinize
        if n == "wd_last_error":
            continue
        assert hasattr(wfstdec, n), n


def test_record_layouts():
    from paper_1804_03243_amd import wfstdec
    assert wfstdec.LINK_DTYPE.itemsize == 48
    assert wfstdec.NODE_DTYPE.itemsize == 16
    assert wfstdec.TOKEN_DTYPE.itemsize == 16
    assert ctypes.sizeof(wfstdec.wd_stats) == 8 + 7 * 8 + 8 + 6 * 8  # wd_caps: 6 x int64


def test_oracle_is_not_imported_by_the_library():
    """The product package neither imports nor links the CPU oracle."""
    pkg = os.path.join(ROOT, "paper_1804_03243_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in txt and "wfst_oracle" not in txt, f
                assert "wdo_" not in txt, f
