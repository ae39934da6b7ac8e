"""The library's SSD -> DRAM tier (m2c_dram_*) on the CPU: plain host memory,
a file of synthetic layers, acquires in decode order. Every acquire returns
the layer's bytes, and the library's load decisions are the oracle's
(oracle/preload.py) one for one, whatever the loader thread's timing."""
import os

import numpy as np
import pytest

from oracle.preload import TwoLevelDram
from paper_2410_14740_amd import m2c


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(m2c.LIB_PATH):
        from paper_2410_14740_amd import build
        build.build()
    return m2c.load()


def _file(tmp_path, n_layers, layer_bytes, direct_pad=True):
    """Layer l is bytes (l * 37 + j) % 251, padded to 4096 per layer."""
    pad = (layer_bytes + 4095) // 4096 * 4096
    path = str(tmp_path / "layers.bin")
    with open(path, "wb") as f:
        for l in range(n_layers):
            b = ((l * 37 + np.arange(pad)) % 251).astype(np.uint8)
            b[layer_bytes:] = 0
            f.write(b.tobytes())
    return path, [l * pad for l in range(n_layers)]


def _expect(l, n):
    return ((l * 37 + np.arange(n)) % 251).astype(np.uint8)


@pytest.mark.parametrize("L,fixed,slots,a,flags", [
    (12, 3, 4, 2, 0), (10, 0, 3, 2, 0), (9, 2, 7, 1, 0), (8, 8, 2, 1, 0),
    (16, 4, 6, 3, m2c.DRAM_DIRECT_IO), (7, 1, 6, 2, 0)])
def test_decisions_and_bytes_match_oracle(lib, tmp_path, L, fixed, slots, a, flags):
    layer_bytes = 10000 + 123 * L
    path, offs = _file(tmp_path, L, layer_bytes)
    desc = m2c.DramDesc(L, fixed, slots, a, layer_bytes, m2c.DRAM_HOST_MEMORY | flags, 0)
    D = m2c.m2c_dram_create(desc, path, offs)
    ref = TwoLevelDram(L, fixed, slots, a)
    tokens = 4
    for t in range(tokens):
        for l in range(L):
            got = m2c.m2c_dram_acquire(D, l, layer_bytes)
            assert np.array_equal(got, _expect(l, layer_bytes)), f"token {t} layer {l}: bytes"
            m2c.m2c_dram_release(D, l)
            ref.use(l)
    log = m2c.m2c_dram_get_log(D)
    assert log == [(m, old) for (_, m, _, old) in ref.log]
    st = m2c.m2c_dram_get_stats(D)
    assert st.acquires == tokens * L
    assert st.loads == len(ref.log) and st.bytes_read == len(ref.log) * layer_bytes
    assert st.fixed_bytes == fixed * layer_bytes
    assert st.evictions == sum(1 for e in ref.log if e[3] >= 0)
    m2c.m2c_dram_destroy(D)


def test_errors(lib, tmp_path):
    path, offs = _file(tmp_path, 4, 5000)
    bad = m2c.DramDesc(4, 1, 1, 2, 5000, m2c.DRAM_HOST_MEMORY, 0)  # slots < lookahead + 1
    with pytest.raises(m2c.M2CError) as e:
        m2c.m2c_dram_create(bad, path, offs)
    assert e.value.status == m2c.M2C_ERR_INVALID_ARG and "lookahead" in str(e.value)
    with pytest.raises(m2c.M2CError):
        m2c.m2c_dram_create(m2c.DramDesc(4, 1, 3, 1, 5000, m2c.DRAM_HOST_MEMORY, 0), path,
                            [0, 4096, 8193, 12288])  # unaligned offset
    with pytest.raises(m2c.M2CError):
        m2c.m2c_dram_create(m2c.DramDesc(4, 1, 3, 1, 5000, m2c.DRAM_HOST_MEMORY, 0),
                            str(tmp_path / "missing.bin"), offs)
    D = m2c.m2c_dram_create(m2c.DramDesc(4, 1, 3, 1, 5000, m2c.DRAM_HOST_MEMORY, 0), path, offs)
    with pytest.raises(m2c.M2CError) as e:
        m2c.m2c_dram_release(D, 2)  # not held
    assert e.value.status == m2c.M2C_ERR_STATE
    with pytest.raises(m2c.M2CError):
        m2c.m2c_dram_acquire(D, 4, 10)
    # a layer past the end of the file: the read fails and the acquire reports it
    D2 = m2c.m2c_dram_create(m2c.DramDesc(5, 0, 3, 1, 5000, m2c.DRAM_HOST_MEMORY, 0), path,
                             offs + [4 * 8192])
    with pytest.raises(m2c.M2CError) as e:
        for l in range(5):
            m2c.m2c_dram_acquire(D2, l, 10)
            m2c.m2c_dram_release(D2, l)
    assert "file" in str(e.value)
    m2c.m2c_dram_destroy(D2)
    m2c.m2c_dram_destroy(D)
