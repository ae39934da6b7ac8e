"""m2c_ratio_search (Algorithm 1 on the FFN-error proxy, every FFN through the
layer's kernels) against the oracle's search: the same candidate ratios, the
same scores within the tolerance the FFN's fp32 accumulation allows, and
the same choice (or, on a near tie, a choice whose oracle score is within
that tolerance of the minimum)."""
import numpy as np
import pytest

from oracle import ratio_search as RS
from paper_2410_14740_amd import m2c
from paper_2410_14740_amd import workloads as W

from helpers import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

UQ_RTOL = 1e-3


@pytest.mark.parametrize("d,d_ff,r,n_low0,step,bit_ratio", [
    (1024, 2752, 128, 688, 16, 4),
    (1024, 2752, 128, 688, 32, 2),
    (384, 700, 48, 175, 5, 4),
])
def test_ratio_search_matches_oracle(d, d_ff, r, n_low0, step, bit_ratio):
    T = 4
    ld = W.make_layer(W.WORKLOADS["tiny"].seed + d_ff, 9, d, d_ff, r, T, rhos=(0.9,))
    say(f"ratio search d={d} d_ff={d_ff} n_low0={n_low0} step={step} n={bit_ratio}")
    L = m2c.Layer(m2c.make_desc(d, d_ff, r, d_ff, d_ff // 3), ld)
    x = torch.from_numpy(np.ascontiguousarray(ld.x[:, 0].view(np.uint16))).cuda()
    cands, uqs, best = m2c.m2c_ratio_search(L.handle, x, T, n_low0, step, bit_ratio)
    ocands, ouqs, obest = RS.search(ld, ld.x[:, 0], n_low0, step, bit_ratio)
    assert cands == ocands
    for i, (u, ou) in enumerate(zip(uqs, ouqs)):
        assert abs(u - ou) <= UQ_RTOL * ou, f"candidate {i} {cands[i]}: uq {u:.6e} vs {ou:.6e}"
    m = min(ouqs)
    assert ouqs[best] <= m * (1 + 2 * UQ_RTOL)
    if sorted(ouqs)[1] > m * (1 + 2 * UQ_RTOL):  # a clear minimum: the same choice
        assert best == obest
    say(f"ratio search: chose {cands[best]} (oracle {ocands[obest]}), uq {uqs[best]:.4e}")
    # the layer is left cold (counters cleared by the reset) and usable
    st = L.stats()
    assert st.plans == 0 and st.req == 0
    tiers = torch.zeros((1, d_ff), dtype=torch.uint8, device="cuda")
    tiers[0, :10] = 3
    L.cache_plan(tiers, 1, 0)
    torch.cuda.synchronize()
    assert L.read_plan()["counts"][m2c.CNT_NEW] == 10
    L.close()


def test_ratio_search_arguments():
    ld = W.make_layer(5, 0, 256, 300, 16, 1)
    L = m2c.Layer(m2c.make_desc(256, 300, 16, 100, 100), ld)  # k_max < d_ff
    x = torch.from_numpy(np.ascontiguousarray(ld.x[:, 0].view(np.uint16))).cuda()
    with pytest.raises(m2c.M2CError) as e:
        m2c.m2c_ratio_search(L.handle, x, 1, 100, 4, 4)
    assert e.value.status == m2c.M2C_ERR_CAPACITY
    L.close()
    L = m2c.Layer(m2c.make_desc(256, 300, 16, 300, 100), ld)
    with pytest.raises(m2c.M2CError):
        m2c.m2c_ratio_search(L.handle, x, 1, 100, 4, 3)  # bit ratio 3
    cands, uqs, best = m2c.m2c_ratio_search(L.handle, x, 1, 3, 4, 4)  # no candidate
    assert cands == [] and best == -1
    L.close()
