"""The C-ABI library loads and exports every function include/treekv.h declares (no GPU needed)."""
import os
import re

import paper_2609_39334_amd as tkv

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "treekv.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tkv_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("tkv_bm_create", "tkv_bm_extend", "tkv_prune", "tkv_bm_coalesce", "tkv_plan_create",
                 "tkv_plan_upload", "tkv_decode", "tkv_verify"):
        assert must in names


def test_library_exports_every_declared_symbol():
    L = tkv.lib()
    for name in _declared():
        assert hasattr(L, name), name


def test_binding_covers_every_declared_symbol():
    assert sorted(tkv.EXPORTED) == _declared()
    for name in _declared():
        assert callable(getattr(tkv, name)), name


def test_noalloc_limit_matches_header():
    src = open(HEADER).read()
    m = re.search(r"#define TKV_NOALLOC_MAX_BYTES \(\(size_t\)(\d+) << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == tkv.TKV_NOALLOC_MAX_BYTES
