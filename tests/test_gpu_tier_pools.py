"""The per-tier record arena (M2C_FLAG_TIER_POOLS) against the oracle's
TierPoolCache: tiers, every plan field (slots in tier blocks), each pool's
tables, the counters and the FFN outputs over several steps, with pools
smaller than their tier's demand (evictions and bypasses in every pool),
larger (hits), an empty pool, the 70B shape at the HBM budget of C = k
FP16-sized slots, and the overflow report; with exact-tier hits and with
dominance hits across the pools (M2C_FLAG_DOMINANT_HITS)."""
import numpy as np
import pytest

import oracle
from paper_2410_14740_amd import m2c
from paper_2410_14740_amd import workloads as W

from helpers import FFN_TOL, oracle_ffn, r8_errors, say, work_order

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _x16(ld, t):
    return torch.from_numpy(np.ascontiguousarray(ld.x[t].view(np.uint16))).cuda().view(torch.float16)


def _run(ld, steps, k, n16, n8, tier_slots, label, dominance=False):
    d, d_ff = ld.d_model, ld.d_ff
    flags = m2c.FLAG_DOMINANT_HITS if dominance else 0
    L = m2c.Layer(m2c.make_desc(d, d_ff, ld.pred_rank, k, 0, flags=flags, tier_slots=tier_slots), ld)
    info = L.info
    C = {t: tier_slots[t] for t in (1, 2, 3)}
    S = {t: info.pool_slots[t] - C[t] for t in (1, 2, 3)}
    assert all(S[t] == max(0, k - C[t]) for t in (1, 2, 3))
    cache = oracle.TierPoolCache(d_ff, C, S,
                                 oracle.POLICY_DOMINANCE if dominance else oracle.POLICY_EXACT)
    assert [info.pool_first[t] for t in (3, 2, 1)] == [cache.first[t] for t in (3, 2, 1)]
    assert all(info.pool_stride[t] == info.record_stride[t] for t in (1, 2, 3))
    tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.empty((1, d), dtype=torch.float32, device="cuda")
    tot = np.zeros(16, np.int64)
    worst = 0.0
    for t in range(steps):
        say(f"{label} step {t}")
        x = _x16(ld, t)
        L.predict_rank(x, 1, k, n16, n8, None, tiers)
        L.cache_plan(tiers, 1, t)
        L.cache_fill()
        y.zero_()
        L.sparse_ffn(x, 1, y)
        torch.cuda.synchronize()
        _, s = oracle.predict(ld.pred_a, ld.pred_b, ld.bias, ld.x[t, 0])
        tm, _ = oracle.select_tiers(s, k, n16, n8)
        assert np.array_equal(tiers.cpu().numpy()[0], tm)
        o = cache.plan(tm, t)
        g = L.read_plan()
        for key in ("req_ids", "req_tier", "req_hit", "req_slot", "req_mask", "fill_ids",
                    "fill_tier", "fill_slot", "fill_from", "evicted_ids"):
            assert np.array_equal(g[key], o[key]), f"step {t}: plan field {key} differs"
        assert np.array_equal(g["counts"][:14], np.concatenate([o["counts"][:13], [0]]))
        ws, wm = work_order(o)
        assert np.array_equal(g["work_slot"], ws) and np.array_equal(g["work_mask"], wm)
        tot += o["counts"]
        for tr in (1, 2, 3):
            so, key, last = m2c.m2c_debug_read_pool_tables(L.handle, tr, d_ff, C[tr])
            pc = cache.pools[tr]
            assert np.array_equal(so, pc.slot_of), f"step {t} pool {tr}: slot_of"
            assert np.array_equal(key, pc.slot_key[:C[tr]]), f"step {t} pool {tr}: slot_key"
            assert np.array_equal(last, pc.slot_last[:C[tr]]), f"step {t} pool {tr}: slot_last"
        y_ref = oracle_ffn(ld, ld.x[t], o["req_ids"], o["req_tier"])[0]
        err = r8_errors(y.cpu().numpy()[0], y_ref).max()
        worst = max(worst, err)
        assert err <= FFN_TOL, f"step {t}: FFN error {err:.3e}"
    st = L.stats()
    assert (st.plans, st.req, st.hit, st.refill, st.new_, st.bypass, st.evict) == (
        steps, tot[0], tot[1], tot[2], tot[3], tot[4], tot[5])
    assert (st.fill[3], st.fill[2], st.fill[1]) == (tot[10], tot[11], tot[12])
    L.close()
    return worst, tot


@pytest.mark.parametrize("dominance", [False, True])
@pytest.mark.parametrize("tier_slots", [{3: 60, 2: 150, 1: 250}, {3: 400, 2: 500, 1: 700},
                                        {3: 0, 2: 300, 1: 300}])
def test_tier_pools_tiny(tier_slots, dominance):
    ld = W.make_layer(W.WORKLOADS["tiny"].seed, 11, 1024, 2752, 128, 10, rhos=(0.85,))
    k, n16, n8 = 688, 229, 229
    worst, tot = _run(ld, 10, k, n16, n8, tier_slots, f"pools {tier_slots} dom {dominance}",
                      dominance)
    assert tot[1] > 0  # hits happened
    say(f"pools {tier_slots} dominance {dominance}: worst FFN error {worst:.2e}, hits {tot[1]}, "
        f"bypass {tot[4]}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("dominance", [False, True])
def test_tier_pools_llama70b_layer_at_the_same_budget(dominance):
    """The 70B shape with the HBM of C = k = 2867 FP16-sized slots split into
    pools that each hold the same multiple of their tier's demand."""
    wl = W.WORKLOADS["llama2-70b"]
    say("70B pools: drawing weights")
    ld = W.workload_layer(wl, 0, steps=8)
    k, n16, n8 = wl.counts()
    budget = wl.cache_slots() * 6 * wl.d_model
    ts = m2c.pool_slots_for_budget(wl.d_model, {3: n16, 2: n8, 1: k - n16 - n8}, budget)
    worst, tot = _run(ld, 8, k, n16, n8, ts, f"70B pools dom {dominance}", dominance)
    say(f"70B pools {ts} dominance {dominance}: worst FFN error {worst:.2e}, "
        f"hit rate {tot[1] / tot[0]:.3f}")


@pytest.mark.parametrize("dominance", [False, True])
def test_tier_pools_lists_longer_than_the_merge_staging(dominance):
    """k = 5000: the merged required and fill lists are longer than the 4096
    ids the merge kernel stages in LDS, so it searches the pools' lists in
    global memory instead."""
    ld = W.make_layer(19, 0, 256, 12000, 16, 4, rhos=(0.7,))
    k, n16, n8 = 5000, 500, 2000
    worst, tot = _run(ld, 4, k, n16, n8, {3: 800, 2: 1500, 1: 2000},
                      f"long lists dom {dominance}", dominance)
    assert tot[0] == 4 * k and tot[1] > 0
    say(f"long merge lists dominance {dominance}: worst FFN error {worst:.2e}")


def test_tier_pools_overflow_leaves_everything_unchanged():
    ld = W.make_layer(17, 0, 256, 300, 16, 2)
    L = m2c.Layer(m2c.make_desc(256, 300, 16, 20, 0, tier_slots={3: 5, 2: 5, 1: 5}), ld)
    tiers = torch.zeros((1, 300), dtype=torch.uint8, device="cuda")
    tiers[0, :10] = 3
    L.cache_plan(tiers, 1, 0)  # fits: 10 FP16 neurons, 5 resident + 5 bypass
    torch.cuda.synchronize()
    before = [m2c.m2c_debug_read_pool_tables(L.handle, t, 300, 5) for t in (1, 2, 3)]
    tiers[0, :] = 1
    tiers[0, :30] = 2
    L.cache_plan(tiers, 1, 1)  # 300 active > capacity 20
    torch.cuda.synchronize()
    assert L.read_plan()["counts"][m2c.CNT_REQ] == 0
    with pytest.raises(m2c.M2CError) as e:
        L.stats()
    assert e.value.status == m2c.M2C_ERR_CAPACITY
    after = [m2c.m2c_debug_read_pool_tables(L.handle, t, 300, 5) for t in (1, 2, 3)]
    for b, a in zip(before, after):
        assert all(np.array_equal(x, y) for x, y in zip(b, a))
    L.close()


def test_tier_pool_descriptor_checks():
    ld = W.make_layer(18, 0, 256, 300, 16, 1)
    for kw in ({"flags": m2c.FLAG_DETERMINISTIC_FFN}, {"max_batch": 2}, {"staging_slots": 10}):
        with pytest.raises(m2c.M2CError) as e:
            m2c.Layer(m2c.make_desc(256, 300, 16, 20, 0, tier_slots={3: 5, 2: 5, 1: 5}, **kw), ld)
        assert e.value.status == m2c.M2C_ERR_INVALID_ARG
    d = m2c.make_desc(256, 300, 16, 20, 0, tier_slots={3: 5, 2: 5, 1: 5})
    d.cache_slots = 16  # not the sum of the pools
    with pytest.raises(m2c.M2CError):
        m2c.Layer(d, ld)
