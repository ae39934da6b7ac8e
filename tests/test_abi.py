"""The C-ABI library loads and exports every entry point include/m2c.h
declares; host-side argument checks fail cleanly without touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2410_14740_amd import m2c

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "m2c.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(m2c_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(m2c.LIB_PATH):
        from paper_2410_14740_amd import build
        build.build()
    return m2c.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 16
    raw = ctypes.CDLL(m2c.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_record_bytes(lib):
    assert m2c.m2c_record_bytes(8192, 3) == 49152
    assert m2c.m2c_record_bytes(8192, 2) == 24960
    assert m2c.m2c_record_bytes(8192, 1) == 12672
    assert m2c.m2c_record_bytes(4096, 1) == 6336
    assert m2c.m2c_record_bytes(100, 1) == -1
    assert m2c.m2c_record_bytes(1024, 0) == -1


@pytest.mark.parametrize("field,value,needle", [
    ("d_model", 100, "d_model"), ("d_ff", 0, "d_ff"), ("pred_rank", 12, "pred_rank"),
    ("group", 64, "group"), ("k_max", 5000, "k_max"), ("max_batch", 33, "max_batch"),
    ("cache_slots", -1, "cache_slots"), ("staging_slots", 3, "staging_slots"),
])
def test_create_rejects_bad_descriptors(lib, field, value, needle):
    desc = m2c.make_desc(1024, 2752, 128, 688, 100)
    setattr(desc, field, value)
    z = np.zeros(8, np.uint16)
    with pytest.raises(m2c.M2CError) as ei:
        m2c.m2c_layer_create(desc, z, z, z, z, z)
    assert ei.value.status == m2c.M2C_ERR_INVALID_ARG
    assert needle in str(ei.value)


def test_null_arguments(lib):
    P = ctypes.c_void_p
    out = P()
    desc = m2c.make_desc(1024, 2752, 128, 688, 1376)
    rc = lib.m2c_layer_create(ctypes.byref(desc), None, None, None, None, None, None, ctypes.byref(out))
    assert rc == m2c.M2C_ERR_INVALID_ARG and out.value is None
    assert lib.m2c_predict_rank(None, None, 1, 1, 0, 0, None, None, None) == m2c.M2C_ERR_INVALID_ARG
    assert lib.m2c_cache_plan(None, None, 1, 0, None, None) == m2c.M2C_ERR_INVALID_ARG
    assert lib.m2c_cache_fill(None, None, None) == m2c.M2C_ERR_INVALID_ARG
    assert lib.m2c_sparse_ffn(None, None, 1, None, None, None) == m2c.M2C_ERR_INVALID_ARG
    assert lib.m2c_layer_destroy(None) == m2c.M2C_OK
    assert "NULL" in m2c.m2c_last_error()
