"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/pic.h declares, and rejects bad arguments before any
device work."""
import ctypes

import pytest

from paper_2602_01519_amd import pic


def test_library_exports_every_header_function():
    names = pic.header_functions()
    assert {"pic_store_create", "pic_store_put", "pic_link_attn", "pic_link_decode",
            "pic_debug_gather", "pic_status_str", "pic_last_error"} <= set(names)
    L = pic.lib()
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    L = pic.lib()
    for code, name in [(0, "PIC_OK"), (-1, "PIC_ERR_INVALID"), (-2, "PIC_ERR_NOT_FOUND"),
                       (-3, "PIC_ERR_EXISTS"), (-4, "PIC_ERR_OOM"), (-5, "PIC_ERR_HIP"),
                       (-6, "PIC_ERR_UNSUPPORTED")]:
        assert L.pic_status_str(code).decode() == name


@pytest.mark.parametrize("desc,status", [
    (dict(kind=2), pic.ERR_INVALID),
    (dict(dtype=7), pic.ERR_INVALID),
    (dict(n_kv_heads=0), pic.ERR_INVALID),
    (dict(d_k=0), pic.ERR_INVALID),
    (dict(capacity_tokens=0), pic.ERR_INVALID),
    (dict(n_layers=-1), pic.ERR_INVALID),
    (dict(n_layers=257), pic.ERR_INVALID),
    (dict(kind=pic.MLA, n_kv_heads=2), pic.ERR_INVALID),
    (dict(kind=pic.MLA, n_kv_heads=1, d_v=256, d_k=128), pic.ERR_INVALID),
    (dict(d_k=12), pic.ERR_UNSUPPORTED),
])
def test_store_create_rejects_bad_descriptors(desc, status):
    base = dict(kind=pic.GQA, dtype=pic.BF16, n_kv_heads=2, d_k=64, d_v=64, n_layers=0,
                capacity_tokens=1024)
    base.update(desc)
    d = pic.StoreDesc(**base)
    h = ctypes.c_void_p(123)
    assert pic.lib().pic_store_create(ctypes.byref(d), ctypes.byref(h)) == status
    assert not h.value            # *out cleared on error
    assert pic.last_error()


def test_null_arguments_are_rejected():
    L = pic.lib()
    assert L.pic_store_create(None, None) == pic.ERR_INVALID
    assert L.pic_store_destroy(None) == pic.OK
    assert L.pic_store_put(None, 1, 1, None, None, None) == pic.ERR_INVALID
    n = ctypes.c_int64()
    assert L.pic_store_lookup(None, 1, ctypes.byref(n)) == pic.ERR_INVALID
    assert L.pic_store_remove(None, 1, None) == pic.ERR_INVALID
    assert L.pic_store_usage(None, None, None, None) == pic.ERR_INVALID
    assert L.pic_link_attn(None, None, 8, None, None, None, 1.0, None, None, None) == pic.ERR_INVALID
    assert L.pic_link_decode(None, None, 8, None, None, None, 1.0, 0, None, None, None) == pic.ERR_INVALID
    assert L.pic_debug_gather(None, None, 0, 0, None, None, None) == pic.ERR_INVALID
    assert "NULL" in pic.last_error()
    h = ctypes.c_void_p(123)
    assert L.pic_link_plan_create(None, None, 8, pic.PREFILL, 0, ctypes.byref(h)) == pic.ERR_INVALID
    assert not h.value
    assert L.pic_link_plan_create(None, None, 8, pic.PREFILL, 0, None) == pic.ERR_INVALID
    assert L.pic_link_plan_run(None, 0, None, None, None, 1.0, None, None, None) == pic.ERR_INVALID
    assert L.pic_link_plan_destroy(None) == pic.OK


def test_import_rejects_what_export_did_not_write():
    """pic_store_import checks the description before any HIP call."""
    L = pic.lib()
    h = ctypes.c_void_p(123)
    assert L.pic_store_import(None, 0, ctypes.byref(h)) == pic.ERR_INVALID
    blob = bytes(64)
    assert L.pic_store_import(blob, len(blob), ctypes.byref(h)) == pic.ERR_INVALID
    assert not h.value
    junk = bytes(range(256)) * 4
    assert L.pic_store_import(junk, len(junk), ctypes.byref(h)) == pic.ERR_INVALID
    assert "exported store" in pic.last_error()
    n = ctypes.c_size_t()
    assert L.pic_store_export(None, None, 0, ctypes.byref(n)) == pic.ERR_INVALID
