"""Host-only checks of the C-ABI library: it loads without a GPU, exports
every entry point include/dualmap.h declares, and rejects bad arguments on
the host before touching a device."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    import paper_2602_06502_amd as pk
    if not os.path.exists(pk.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return pk, pk.load_library()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "dualmap.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dm_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("dm_build_rings", "dm_index_insert", "dm_route_batch", "dm_rebalance",
                     "dm_scale", "dm_create", "dm_sync"):
        assert required in names


def test_library_exports_every_declared_symbol():
    pk, lib = _lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(pk.EXPORTS) == set(declared_functions())


def test_library_is_not_linked_to_the_oracle():
    pk, _ = _lib()
    data = open(pk.LIB_PATH, "rb").read()
    assert b"or_route" not in data and b"liboracle" not in data


def test_config_validation_on_host():
    pk, lib = _lib()
    good = dict(block=16, key_blocks=4, seeds=(1, 2), vnodes=8, max_slots=8, index_log2_slots=10)
    bad = [dict(good, block=12), dict(good, block=2), dict(good, block=128),
           dict(good, key_blocks=0), dict(good, key_blocks=65), dict(good, vnodes=0),
           dict(good, max_slots=0), dict(good, max_slots=5000), dict(good, index_log2_slots=3),
           dict(good, index_log2_slots=31), dict(good, queue_div=3), dict(good, queue_div=0)]
    h = C.c_void_p()
    for cfg in bad:
        assert lib.dm_create(C.byref(pk.make_config(cfg)), None, C.byref(h)) == pk.DM_EINVAL, cfg
    assert lib.dm_create(None, None, C.byref(h)) == pk.DM_EINVAL
    c = pk.make_config(good)
    c.reserved = 1
    assert lib.dm_create(C.byref(c), None, C.byref(h)) == pk.DM_EINVAL


def test_null_context_is_rejected():
    pk, lib = _lib()
    assert lib.dm_sync(None) == pk.DM_EINVAL
    assert lib.dm_build_rings(None, None, 0) == pk.DM_EINVAL
    assert lib.dm_route_batch(None, None, 0, None, 0, None, None) == pk.DM_EINVAL
    assert lib.dm_rebalance(None, None, None, None, 0) == pk.DM_EINVAL
    assert lib.dm_scale(None, None, 0, None, 0, None, 0, None, None, None, None) == pk.DM_EINVAL
    assert lib.dm_index_insert(None, 0, None, 0) == pk.DM_EINVAL
    assert lib.dm_set_policy(None, 0) == pk.DM_EINVAL
    assert lib.dm_last_error(None) == b"null context"
    lib.dm_destroy(None)


def test_no_cpu_fallback_without_library(tmp_path):
    import paper_2602_06502_amd as pk
    saved = pk._lib
    try:
        pk._lib = None
        with pytest.raises(ImportError):
            pk.load_library(str(tmp_path / "missing.so"))
    finally:
        pk._lib = saved
