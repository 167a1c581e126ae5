"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/minima_kv.h declares, sizes pools, and rejects bad
arguments before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "minima_kv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:mkv_status|const char\*)\s+(\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def mk():
    import paper_2608_23834_amd as mk
    mk.lib()
    return mk


def test_exports_match_header(mk):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(mk.lib(), n), n
    assert set(mk.EXPORTS) == set(names)


def test_pool_bytes(mk):
    b8, bs, b3, bc = mk.pool_bytes(16, 24, 4, 256, 1000, 2000, 1024)
    assert b8 == 16 * 1000 * 4 * 2 * 16 * 256
    assert bs == 16 * 1000 * 4 * 2 * 4
    assert b3 == 16 * 2000 * 4 * 4128
    assert bc >= 4 * (64 + 1000 + 2000 + 4 * 1000) + 256


@pytest.mark.parametrize("geom,code", [
    ((1, 8, 1, 64, 10, 10, 16), 2),     # head_dim not compiled
    ((1, 34, 2, 128, 10, 10, 16), 2),   # group 17 > 16
    ((1, 6, 4, 128, 10, 10, 16), 1),    # heads not a multiple
    ((0, 8, 1, 128, 10, 10, 16), 1),    # no layers
    ((1, 8, 1, 128, 0, 10, 16), 1),     # no FP8 pages
    ((1, 8, 1, 128, 10, 10, 0), 1),     # W < 1
])
def test_pool_bytes_rejects(mk, geom, code):
    with pytest.raises(mk.MkvError) as e:
        mk.pool_bytes(*geom)
    assert e.value.code == code


def _desc(mk, **kw):
    d = mk.PoolDesc(1, 8, 1, 128, 16, 4, 4, 16)
    fake = 1 << 20  # aligned non-null placeholders; validation fails before any device access
    d.fp8_data = d.fp8_scales = d.tq3_data = d.ctrl = fake
    b8, bs, b3, bc = mk.pool_bytes(1, 8, 1, 128, 4, 4, 16)
    d.fp8_data_bytes, d.fp8_scales_bytes, d.tq3_data_bytes, d.ctrl_bytes = b8, bs, b3, bc
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def test_pool_create_validates_before_device(mk):
    L = mk.lib()
    sig = np.ones(128, np.int8)
    h = ctypes.c_void_p()
    d = _desc(mk, rot_signs=None)
    assert L.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == 1
    bad = sig.copy()
    bad[3] = 2
    d = _desc(mk, rot_signs=bad.ctypes.data)
    assert L.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == 1
    order = np.array([0, 1, 1, 2], np.int32)
    d = _desc(mk, rot_signs=sig.ctypes.data, fp8_order=order.ctypes.data)
    assert L.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == 1
    d = _desc(mk, rot_signs=sig.ctypes.data)
    d.tq3_data_bytes -= 1
    assert L.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == 3
    d = _desc(mk, rot_signs=sig.ctypes.data, fp8_data=(1 << 20) + 4)
    assert L.kv_pool_create(ctypes.byref(d), ctypes.byref(h)) == 1
    assert h.value is None


def test_calls_reject_null_handles(mk):
    L = mk.lib()
    assert L.paged_attn_decode(None, 0, 1, None, None, None, 1, None, None, None, None, 0, None) == 1
    assert L.kv_append_fp8(None, -1, 1, None, None, 1, None, None, 0, None, None, None) == 1
    assert L.kv_migrate_to_tq3(None, 1, None, None, 1, None, None, None) == 1
    assert L.paged_attn_chunk(None, 0, 1, None, None, 1, None, None, 1, None, None, None, 0, None) == 1
    assert L.kv_partition_pages(0, None, None, 1, None, None, None, None, None) == 1
    assert L.mkv_status_string(3) == b"buffer too small"


def test_stream_probe_rejects_bad_arguments(mk):
    L = mk.lib()
    sink = ctypes.c_void_p(64)  # never dereferenced: validation fails first
    assert L.mkv_stream_read(None, 16, sink, None) == 1
    assert L.mkv_stream_read(ctypes.c_void_p(16), 16, None, None) == 1
    assert L.mkv_stream_read(ctypes.c_void_p(8), 16, sink, None) == 1      # misaligned
    assert L.mkv_stream_read(ctypes.c_void_p(16), 24, sink, None) == 1     # not whole 16-byte words
