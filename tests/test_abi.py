"""The C-ABI library loads and exports every function include/hotcold_kv.h
declares, and the Python binding covers them all (CPU only: no compute calls)."""

import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hotcold_kv.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("defined",)))


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("kv_pool_create", "kv_evict_session", "kv_resume_session",
                     "paged_decode_attention"):
        assert required in names
    assert len(names) >= 20


def test_library_exports_every_declared_symbol():
    from paper_2609_25782_amd import hotcold_kv as kv
    lib = ctypes.CDLL(kv.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    from paper_2609_25782_amd import hotcold_kv as kv
    assert sorted(_declared()) == kv.exported_names()
    for n in _declared():
        assert callable(getattr(kv, n))


def test_page_bytes_and_strerror():
    from paper_2609_25782_amd import hotcold_kv as kv
    d = kv.kv_pool_desc(48, 4, 128, 16, kv.KV_DTYPE_BF16, 1, 1, 0, 1, 1, 0, 0)
    assert kv.kv_page_bytes(d) == 1536 * 1024
    d.page_size = 8
    assert kv.kv_page_bytes(d) == 0
    assert kv.kv_strerror(kv.KV_ERR_NO_HOT_PAGES) == "hot pool exhausted"
