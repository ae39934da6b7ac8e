"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

Integer outputs (records, scores bits, tiers, plans, slot tables) must match
bit for bit; FFN outputs within 2e-3 of the oracle under the floored
relative error of helpers.r8_errors.
"""
import numpy as np
import pytest

import oracle
from paper_2410_14740_amd import m2c
from paper_2410_14740_amd import workloads as W

from helpers import (FFN_TOL, derived_fills, oracle_ffn, r8_errors, say, subset_records,
                     work_order)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# (name, d_model, d_ff, pred_rank, seed): a ragged shape (d/8 = 48 chunks,
# r/8 = 6 chunks, d_ff not a multiple of 64) and the tiny workload's shape.
SHAPES = [("ragged", 384, 700, 48, 101), ("tiny", 1024, 2752, 128, W.WORKLOADS["tiny"].seed)]


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _x16(ld, t):
    return _dev(ld.x[t].view(np.uint16)).view(torch.float16)


def _layer(ld, k_max, C, max_batch=1, staging=-1, flags=0):
    desc = m2c.make_desc(ld.d_model, ld.d_ff, ld.pred_rank, k_max, C, max_batch, staging,
                         flags=flags)
    return m2c.Layer(desc, ld)


def _counts(k, frac16=(1, 3), frac8=(1, 3)):
    n16 = k * frac16[0] // frac16[1]
    n8 = k * (frac16[0] * frac8[1] + frac8[0] * frac16[1]) // (frac16[1] * frac8[1]) - n16
    return n16, n8


@pytest.mark.parametrize("name,d,d_ff,r,seed", SHAPES)
def test_records_bit_exact(name, d, d_ff, r, seed):
    ld = W.make_layer(seed, 0, d, d_ff, r, 1)
    say(f"records {name} d={d} d_ff={d_ff}")
    L = _layer(ld, d_ff // 4, d_ff // 2)
    for t in (1, 2, 3):
        ref = oracle.build_records(ld.w_gate, ld.w_up, ld.w_down, t)
        nb = L.info.record_stride[t]
        assert ref.shape[1] == nb
        got = np.stack([m2c.m2c_debug_read_record(L.handle, t, i, nb) for i in range(d_ff)])
        assert np.array_equal(got, ref), f"tier {t}: {np.argwhere((got != ref).any(1))[:5].ravel()}"
    L.close()


@pytest.mark.parametrize("batch", [1, 3])
@pytest.mark.parametrize("name,d,d_ff,r,seed", SHAPES)
def test_predict_and_tiers_bit_exact(name, d, d_ff, r, seed, batch):
    rhos = tuple([0.9, 0.5, 0.95][:batch])
    ld = W.make_layer(seed, 1, d, d_ff, r, 4, rhos=rhos, zipf_bias=(batch == 3))
    k = d_ff // 4
    n16, n8 = _counts(k)
    say(f"predict {name} batch={batch}")
    L = _layer(ld, k, d_ff // 2, max_batch=batch)
    scores = torch.empty((batch, d_ff), dtype=torch.float32, device="cuda")
    tiers = torch.empty((batch, d_ff), dtype=torch.uint8, device="cuda")
    for t in range(4):
        L.predict_rank(_x16(ld, t), batch, k, n16, n8, scores, tiers)
        torch.cuda.synchronize()
        s_gpu, t_gpu = scores.cpu().numpy(), tiers.cpu().numpy()
        for b in range(batch):
            _, s_ref = oracle.predict(ld.pred_a, ld.pred_b, ld.bias, ld.x[t, b])
            assert np.array_equal(s_gpu[b].view(np.uint32), s_ref.view(np.uint32)), \
                f"step {t} row {b}: {np.count_nonzero(s_gpu[b] != s_ref)} scores differ"
            t_ref, _ = oracle.select_tiers(s_ref, k, n16, n8)
            assert np.array_equal(t_gpu[b], t_ref)
    L.close()


def _compare_plan(g, o, step):
    """Every field of the library's plan against the oracle's: the method's
    lists and counts, plus the FFN work order and the derived-fill count the
    library adds (both follow from the oracle's lists)."""
    for key in ("req_ids", "req_tier", "req_hit", "req_slot", "req_mask", "fill_ids",
                "fill_tier", "fill_slot", "fill_from", "evicted_ids"):
        assert np.array_equal(g[key], o[key]), f"step {step}: plan field {key} differs"
    assert np.array_equal(g["counts"][:13], o["counts"][:13]), f"step {step}: counts differ"
    ws, wm = work_order(o)
    assert np.array_equal(g["work_slot"], ws), f"step {step}: FFN work order differs"
    assert np.array_equal(g["work_mask"], wm), f"step {step}: FFN work masks differ"
    assert g["counts"][m2c.CNT_FILL_DERIVED] == derived_fills(o), f"step {step}: derived count"


def _run_steps(ld, steps, k, n16, n8, C, batch=1, check_ffn=True, label="", flags=0):
    """predict -> plan -> fill -> FFN on the GPU and in the oracle, step by
    step, comparing every stage."""
    d_ff = ld.d_ff
    L = _layer(ld, k, C, max_batch=batch, flags=flags)
    policy = (oracle.POLICY_DOMINANCE if flags & m2c.FLAG_DOMINANT_HITS
              else oracle.POLICY_EXACT)
    cache = oracle.LRUCache(d_ff, C, L.info.staging_slots, policy)
    tiers = torch.empty((batch, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.empty((batch, ld.d_model), dtype=torch.float32, device="cuda")
    stats = np.zeros(16, np.int64)
    worst = 0.0
    for t in range(steps):
        say(f"{label} step {t}")
        x = _x16(ld, t)
        L.predict_rank(x, batch, k, n16, n8, None, tiers)
        L.cache_plan(tiers, batch, t)
        L.cache_fill()
        if check_ffn:
            y.zero_()
            L.sparse_ffn(x, batch, y)
        torch.cuda.synchronize()
        tm_ref = np.stack([oracle.select_tiers(oracle.predict(ld.pred_a, ld.pred_b, ld.bias,
                                                              ld.x[t, b])[1], k, n16, n8)[0]
                           for b in range(batch)])
        assert np.array_equal(tiers.cpu().numpy(), tm_ref), f"step {t}: tier maps differ"
        o = cache.plan(tm_ref, t)
        g = L.read_plan()
        _compare_plan(g, o, t)
        stats += o["counts"]
        stats[13] += derived_fills(o)
        slot_of, key, stier, last = m2c.m2c_debug_read_tables(L.handle, d_ff, C)
        assert np.array_equal(slot_of, cache.slot_of)
        assert np.array_equal(key, cache.slot_key[:C])
        assert np.array_equal(stier, cache.slot_tier[:C])
        assert np.array_equal(last, cache.slot_last[:C])
        # fills made on the GPU from the resident FP16 record: the store's bytes
        der = [(int(i), int(tr), int(sl)) for i, tr, sl, fr in
               zip(o["fill_ids"], o["fill_tier"], o["fill_slot"], o["fill_from"])
               if fr == 3 and tr < 3]
        if der:
            recs, row = subset_records(ld, [i for i, _, _ in der])
            for i, tr, sl in der:
                nb = L.info.record_bytes[tr]
                got = m2c.m2c_debug_read_slot(L.handle, sl, nb)
                assert np.array_equal(got, recs[tr][row[i]][:nb]), \
                    f"step {t}: derived tier-{tr} record of neuron {i} differs"
        if check_ffn:
            y_ref = oracle_ffn(ld, ld.x[t], o["req_ids"], o["req_tier"],
                               o["req_mask"] if batch > 1 else None)
            yg = y.cpu().numpy()
            for b in range(batch):
                err = r8_errors(yg[b], y_ref[b]).max()
                worst = max(worst, err)
                assert err <= FFN_TOL, f"step {t} row {b}: FFN error {err:.3e}"
    st = L.stats()
    assert (st.plans, st.req, st.hit, st.refill, st.new_, st.bypass, st.evict) == (
        steps, stats[0], stats[1], stats[2], stats[3], stats[4], stats[5])
    assert (st.fill[3], st.fill[2], st.fill[1]) == (stats[10], stats[11], stats[12])
    assert (st.req_tier[3], st.req_tier[2], st.req_tier[1]) == (stats[7], stats[8], stats[9])
    assert st.derived[1] + st.derived[2] == stats[13] and st.derived[3] == 0
    rb = L.info.record_bytes
    assert st.host_bytes == st.fill_bytes - st.derived[1] * rb[1] - st.derived[2] * rb[2]
    L.close()
    return worst, int(stats[13])


@pytest.mark.parametrize("flags", [0, m2c.FLAG_DETERMINISTIC_FFN])
@pytest.mark.parametrize("name,d,d_ff,r,seed", SHAPES)
def test_end_to_end_steps(name, d, d_ff, r, seed, flags):
    ld = W.make_layer(seed, 2, d, d_ff, r, 10, rhos=(0.8,))
    k = d_ff // 4
    n16, n8 = _counts(k)
    # C < k forces evictions and bypasses every step
    _, derived = _run_steps(ld, 10, k, n16, n8, C=(2 * k) // 3, label=f"e2e {name} flags={flags}",
                            flags=flags)
    assert derived > 0  # FP16 -> lower-tier refills were made on the GPU and checked


def test_tiny_workload_all_steps():
    wl = W.WORKLOADS["tiny"]
    ld = W.workload_layer(wl, 0)
    k, n16, n8 = wl.counts()
    worst, _ = _run_steps(ld, wl.steps, k, n16, n8, wl.cache_slots(), label="tiny workload")
    say(f"tiny workload worst FFN error {worst:.2e}")


def test_batched_plan_union_and_bypass():
    """Batch 4 on a ragged layer: union plans with bypasses, and the batched
    (MFMA) FFN against the oracle's masked FFN, row by row."""
    ld = W.make_layer(77, 0, 384, 700, 48, 6, rhos=(0.5, 0.95, 0.9, 0.7), zipf_bias=True)
    k = 120
    n16, n8 = _counts(k, (1, 10), (2, 5))
    _run_steps(ld, 6, k, n16, n8, C=200, batch=4, label="batched plan")


@pytest.mark.parametrize("batch,d,d_ff,r", [(2, 1024, 1000, 64), (16, 256, 600, 32),
                                             (17, 256, 600, 32), (20, 512, 900, 32),
                                             (32, 384, 700, 48)])
def test_batched_ffn_shapes(batch, d, d_ff, r):
    """Batch 2 and 16 (one 16-row MFMA batch tile), 17, 20 and 32 (two tiles;
    32 is the largest batch), an odd number of quantization groups (d 384),
    mixed tiers, C below the union."""
    rhos = tuple(0.5 + 0.45 * (b % 2) for b in range(batch))
    ld = W.make_layer(300 + batch, 0, d, d_ff, r, 3, rhos=rhos, zipf_bias=True)
    k = d_ff // 6
    n16, n8 = _counts(k, (1, 5), (3, 10))
    worst, _ = _run_steps(ld, 3, k, n16, n8, C=k, batch=batch, label=f"batched B={batch}")
    say(f"batched B={batch} worst FFN error {worst:.2e}")


@pytest.mark.parametrize("scale_exp", [-8, 6])
def test_batched_ffn_input_scale(scale_exp):
    """x scaled by 2^-8 (h about 2^-16 of its usual size) and by 2^6: the
    batched down projection normalises h s per wave before splitting it into
    fp16 parts, so the error stays within tolerance at any magnitude."""
    ld = W.make_layer(410, 0, 512, 900, 32, 3, rhos=(0.5, 0.95, 0.9, 0.7, 0.6, 0.8, 0.95, 0.5),
                      zipf_bias=True)
    ld.x = (ld.x.astype(np.float32) * np.float32(2.0 ** scale_exp)).astype(np.float16)
    k = 150
    n16, n8 = _counts(k, (1, 5), (3, 10))
    worst, _ = _run_steps(ld, 2, k, n16, n8, C=k, batch=8, label=f"batched x*2^{scale_exp}")
    say(f"batched x*2^{scale_exp} worst FFN error {worst:.2e}")


def test_batched_all_fp16_equals_single_token():
    """All-FP16: row b of the batched FFN equals the single-token FFN of x_b
    over row b's own selection (the union only adds neurons masked out of b)."""
    d, d_ff, r, B = 512, 800, 32, 4
    ld = W.make_layer(91, 0, d, d_ff, r, 1, rhos=(0.9, 0.5, 0.95, 0.7))
    k = 100
    Lb = _layer(ld, k, d_ff, max_batch=B)
    tiers = torch.empty((B, d_ff), dtype=torch.uint8, device="cuda")
    x = _x16(ld, 0)
    Lb.predict_rank(x, B, k, k, 0, None, tiers)
    Lb.cache_plan(tiers, B, 0)
    Lb.cache_fill()
    yb = torch.zeros((B, d), dtype=torch.float32, device="cuda")
    Lb.sparse_ffn(x, B, yb)
    torch.cuda.synchronize()
    tm = tiers.cpu().numpy()
    for b in range(B):
        L1 = _layer(ld, k, d_ff)
        t1 = torch.from_numpy(np.ascontiguousarray(tm[b:b + 1])).cuda()
        L1.cache_plan(t1, 1, 0)
        L1.cache_fill()
        y1 = torch.zeros((1, d), dtype=torch.float32, device="cuda")
        L1.sparse_ffn(x[b:b + 1], 1, y1)
        torch.cuda.synchronize()
        err = r8_errors(yb.cpu().numpy()[b], y1.cpu().numpy()[0].astype(np.float64)).max()
        assert err <= 1e-4, f"row {b}: batched vs single {err:.2e}"
        L1.close()
    Lb.close()


def test_batched_llama7b_b8_workload():
    """The batch-8 decode workload on the 7B-shaped layer (d 4096, d_ff 11008,
    rank 256, k 2201 per row with tiers 220/880/1101, log-Zipf popularity,
    rho 0.5 / 0.95 rows, C = 30% of d_ff): plans bit-exact and every row of
    the batched FFN within tolerance, two steps."""
    wl = W.WORKLOADS["llama2-7b-b8"]
    say("7B batch-8 layer: drawing weights")
    ld = W.workload_layer(wl, 0, steps=2)
    k, n16, n8 = wl.counts()
    worst, _ = _run_steps(ld, 2, k, n16, n8, wl.cache_slots(), batch=wl.batch, label="7B b8")
    say(f"7B batch-8 worst FFN error {worst:.2e}")


def test_dense_equivalence_all_fp16():
    """k = d_ff, every neuron FP16, every neuron cached: the sparse FFN is the
    dense SwiGLU FFN."""
    d, d_ff = 512, 640
    ld = W.make_layer(55, 0, d, d_ff, 32, 2)
    L = _layer(ld, d_ff, d_ff)
    tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.empty((1, d), dtype=torch.float32, device="cuda")
    for t in range(2):
        x = _x16(ld, t)
        L.predict_rank(x, 1, d_ff, d_ff, 0, None, tiers)
        L.cache_plan(tiers, 1, t)
        L.cache_fill()
        y.zero_()
        L.sparse_ffn(x, 1, y)
        torch.cuda.synchronize()
        assert (tiers.cpu().numpy() == 3).all()
        y_ref = oracle.dense_ffn(ld.w_gate, ld.w_up, ld.w_down, ld.x[t, 0])
        assert r8_errors(y.cpu().numpy()[0], y_ref).max() <= FFN_TOL
    g = L.read_plan()
    assert g["counts"][m2c.CNT_HIT] == d_ff  # second step: everything hits
    L.close()


def test_k_zero_and_all_equal_scores():
    d, d_ff, r = 256, 300, 16
    ld = W.make_layer(9, 0, d, d_ff, r, 2)
    ld.pred_a[:] = 0  # every score is exactly +0.0: ties resolve by id
    L = _layer(ld, 40, 100)
    tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.empty((1, d), dtype=torch.float32, device="cuda")
    x = _x16(ld, 0)
    L.predict_rank(x, 1, 40, 10, 10, None, tiers)
    torch.cuda.synchronize()
    tm = tiers.cpu().numpy()[0]
    assert list(tm[:40]) == [3] * 10 + [2] * 10 + [1] * 20 and not tm[40:].any()
    L.predict_rank(x, 1, 0, 0, 0, None, tiers)
    L.cache_plan(tiers, 1, 0)
    L.cache_fill()
    y.zero_()
    L.sparse_ffn(x, 1, y)
    torch.cuda.synchronize()
    assert not tiers.cpu().numpy().any()
    assert L.read_plan()["counts"][m2c.CNT_REQ] == 0
    assert not y.cpu().numpy().any()
    L.close()


def test_fill_twice_and_cache_reset_keep_derived_records_exact():
    """A fill derived on the GPU quantizes the FP16 bytes in the slot. Running
    the fill of a plan a second time must not quantize the INT8 / INT4 bytes
    again (it copies from the store instead), and after a cache reset no slot
    counts as holding an FP16 record."""
    ld = W.make_layer(41, 0, 512, 900, 32, 8, rhos=(0.7,))
    k = 300
    n16, n8 = _counts(k)
    L = _layer(ld, k, 250)
    tiers = torch.empty((1, 900), dtype=torch.uint8, device="cuda")
    y = torch.empty((1, 512), dtype=torch.float32, device="cuda")
    checked = 0
    for rnd in range(2):
        for t in range(8):
            say(f"fill twice: round {rnd} step {t}")
            x = _x16(ld, t)
            L.predict_rank(x, 1, k, n16, n8, None, tiers)
            L.cache_plan(tiers, 1, 8 * rnd + t)
            L.cache_fill()
            L.cache_fill()  # again, on the same plan
            y.zero_()
            L.sparse_ffn(x, 1, y)
            torch.cuda.synchronize()
            g = L.read_plan()
            der = [(int(i), int(tr), int(sl)) for i, tr, sl, fr in
                   zip(g["fill_ids"], g["fill_tier"], g["fill_slot"], g["fill_from"])
                   if fr == 3 and tr < 3]
            if der:
                recs, row = subset_records(ld, [i for i, _, _ in der])
                for i, tr, sl in der:
                    nb = L.info.record_bytes[tr]
                    got = m2c.m2c_debug_read_slot(L.handle, sl, nb)
                    assert np.array_equal(got, recs[tr][row[i]][:nb]), \
                        f"round {rnd} step {t}: tier-{tr} record of neuron {i} differs"
                checked += len(der)
            y_ref = oracle_ffn(ld, ld.x[t], g["req_ids"], g["req_tier"])
            err = r8_errors(y.cpu().numpy()[0], y_ref[0]).max()
            assert err <= FFN_TOL, f"round {rnd} step {t}: FFN error {err:.3e}"
        L.reset_cache()
        torch.cuda.synchronize()
    assert checked > 0
    L.close()


def test_host_errors_leave_layer_usable():
    ld = W.make_layer(3, 0, 256, 200, 16, 3)
    L = _layer(ld, 50, 60)
    tiers = torch.zeros((1, 200), dtype=torch.uint8, device="cuda")
    L.cache_plan(tiers, 1, 5)
    with pytest.raises(m2c.M2CError) as e:
        L.cache_plan(tiers, 1, 5)
    assert e.value.status == m2c.M2C_ERR_STATE
    with pytest.raises(m2c.M2CError) as e:
        L.predict_rank(_x16(ld, 0), 1, 51, 0, 0, None, tiers)
    assert e.value.status == m2c.M2C_ERR_CAPACITY
    with pytest.raises(m2c.M2CError) as e:
        L.predict_rank(_x16(ld, 0), 2, 10, 0, 0, None, tiers)
    assert e.value.status == m2c.M2C_ERR_CAPACITY
    with pytest.raises(m2c.M2CError) as e:
        L.predict_rank(_x16(ld, 0), 1, 10, 6, 6, None, tiers)
    assert e.value.status == m2c.M2C_ERR_INVALID_ARG
    L.predict_rank(_x16(ld, 0), 1, 10, 2, 3, None, tiers)
    L.cache_plan(tiers, 1, 6)
    torch.cuda.synchronize()
    assert L.read_plan()["counts"][m2c.CNT_REQ] == 10
    L.reset_cache()
    L.cache_plan(tiers, 1, 0)  # history cleared by the reset
    torch.cuda.synchronize()
    assert L.read_plan()["counts"][m2c.CNT_NEW] == 10
    L.close()


def test_shared_store_layers():
    ld0 = W.make_layer(13, 0, 256, 300, 16, 2)
    ld1 = W.make_layer(13, 1, 256, 300, 16, 2, weight_layer=0)
    L0 = _layer(ld0, 60, 60)
    desc = m2c.make_desc(256, 300, 16, 60, 60)
    L1 = m2c.Layer(desc, ld1, weights_of=L0)
    nb = L0.info.record_stride[2]
    assert np.array_equal(m2c.m2c_debug_read_record(L1.handle, 2, 7, nb),
                          m2c.m2c_debug_read_record(L0.handle, 2, 7, nb))
    L0.close()  # the store stays alive for L1
    ref = oracle.build_records(ld0.w_gate, ld0.w_up, ld0.w_down, 2)
    assert np.array_equal(m2c.m2c_debug_read_record(L1.handle, 2, 7, nb), ref[7])
    L1.close()


@pytest.mark.timeout(900)
def test_llama70b_layer_shape():
    """One layer at the 70B shape (d 8192, d_ff 28672, rank 512, k 2867,
    tiers 286/860/1721, C = k): scores, tiers, plans and tables bit-exact,
    every FFN output within tolerance, over eight steps (C = k: every step
    evicts what the previous token used and the new one does not)."""
    wl = W.WORKLOADS["llama2-70b"]
    say("70B layer: drawing weights")
    ld = W.workload_layer(wl, 0, steps=8)
    k, n16, n8 = wl.counts()
    worst, _ = _run_steps(ld, 8, k, n16, n8, wl.cache_slots(), label="70B layer")
    say(f"70B layer worst FFN error {worst:.2e}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama2-7b", "llama2-13b"])
def test_llama7b_13b_layer_shapes(name):
    """One layer at the 7B shape (d 4096, d_ff 11008, rank 256, k 2201 =
    220/880/1101, C 3302) and at the 13B shape (d 5120 -- not a power of two:
    padded lanes in every gate/up unit -- d_ff 13824, k 2073 = 414/622/1037,
    C 2764), batch 1, over sixteen steps (the LRU reaches steady-state
    eviction): scores, tiers, plans, slot tables and derived records
    bit-exact, every FFN output within tolerance."""
    wl = W.WORKLOADS[name]
    say(f"{name} layer: drawing weights")
    ld = W.workload_layer(wl, 0, steps=16)
    k, n16, n8 = wl.counts()
    worst, _ = _run_steps(ld, 16, k, n16, n8, wl.cache_slots(), label=f"{name} layer")
    say(f"{name} layer worst FFN error {worst:.2e}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cap,mix", [((1, 10), "10/40/50"), ((1, 10), "fp16"), ((3, 5), "fp16")])
def test_batched_llama7b_b8_sweep_points(cap, mix):
    """More points of the batch-8 sweep at full shape: C = 10% of d_ff (most
    of the union bypasses through staging slots) with mixed tiers and all
    FP16, and C = 60% all FP16; two steps each."""
    wl = W.WORKLOADS["llama2-7b-b8"]
    say(f"7B batch-8 C={cap} {mix}: drawing weights")
    ld = W.workload_layer(wl, 0, steps=2)
    k, n16, n8 = wl.counts()
    if mix == "fp16":
        n16, n8 = k, 0
    C = wl.d_ff * cap[0] // cap[1]
    worst, _ = _run_steps(ld, 2, k, n16, n8, C, batch=wl.batch, label=f"7B b8 C={C} {mix}")
    say(f"7B batch-8 C={C} {mix} worst FFN error {worst:.2e}")


@pytest.mark.parametrize("batch", [1, 4])
def test_no_cache_slots_everything_bypasses(batch):
    """C = 0: every active neuron is a BYPASS filled into a staging slot each
    step, nothing is retained."""
    ld = W.make_layer(71, 0, 512, 900, 32, 4, rhos=(0.8, 0.5, 0.95, 0.7)[:batch])
    k = 150
    n16, n8 = _counts(k, (1, 5), (3, 10))
    worst, _ = _run_steps(ld, 4, k, n16, n8, C=0, batch=batch, label=f"C=0 B={batch}")
    say(f"C=0 batch {batch} worst FFN error {worst:.2e}")


def test_wide_d_ff_general_kernels():
    """d_ff above 32768 runs the general select and plan kernels (the
    register select and the ballot plan take d_ff <= 32768): tiers, plans and
    tables bit-exact, FFN within tolerance, over four steps with evictions."""
    ld = W.make_layer(83, 0, 256, 40000, 16, 4, rhos=(0.7,))
    k = 3000
    n16, n8 = _counts(k, (1, 10), (3, 10))
    worst, _ = _run_steps(ld, 4, k, n16, n8, C=2500, label="d_ff=40000")
    say(f"d_ff=40000 worst FFN error {worst:.2e}")


def test_wide_d_ff_general_kernels_batched_dominance():
    ld = W.make_layer(84, 0, 256, 36000, 16, 3, rhos=(0.7, 0.9))
    k = 1200
    n16, n8 = _counts(k, (1, 5), (3, 10))
    _run_steps(ld, 3, k, n16, n8, C=1500, batch=2, flags=m2c.FLAG_DOMINANT_HITS,
               label="d_ff=36000 B=2 dominance")


@pytest.mark.parametrize("batch,C", [(1, 200), (4, 200), (1, 2752)])
def test_dominant_hits_policy(batch, C):
    """Dominance hits (a neuron resident at a tier at or above the requested
    one is a hit at its resident tier): plans, step tiers, tables and the FFN
    over the resident records against the oracle's dominance policy, with
    evictions and bypasses (C = 200) and with everything resident."""
    ld = W.make_layer(W.WORKLOADS["tiny"].seed, 5, 1024, 2752, 128, 10,
                      rhos=(0.8, 0.5, 0.95, 0.7)[:batch])
    k = 688
    n16, n8 = _counts(k)
    worst, _ = _run_steps(ld, 10, k, n16, n8, C=C, batch=batch, flags=m2c.FLAG_DOMINANT_HITS,
                          label=f"dominance B={batch} C={C}")
    say(f"dominance B={batch} C={C} worst FFN error {worst:.2e}")


@pytest.mark.timeout(900)
def test_dominant_hits_llama7b_layer():
    """Dominance hits on the 7B-shaped layer (C = 30%) over eight steps."""
    wl = W.WORKLOADS["llama2-7b"]
    say("7B layer, dominance: drawing weights")
    ld = W.workload_layer(wl, 1, steps=8)
    k, n16, n8 = wl.counts()
    worst, _ = _run_steps(ld, 8, k, n16, n8, wl.cache_slots(), flags=m2c.FLAG_DOMINANT_HITS,
                          label="7B layer dominance")
    say(f"7B dominance worst FFN error {worst:.2e}")


def test_ffn_wait_give_up_is_reported():
    """The one-launch FFN's bounded wait: with its h values withheld (test
    support), every down task gives up after a few polls and exits, the call's
    output misses the down projection, m2c_layer_stats reports M2C_ERR_STATE
    once and clears it, and the next normal call is correct again."""
    ld = W.make_layer(44, 0, 1024, 2752, 128, 3)
    k = 688
    n16, n8 = _counts(k)
    L = _layer(ld, k, 1376)
    tiers = torch.empty((1, ld.d_ff), dtype=torch.uint8, device="cuda")
    x = _x16(ld, 0)
    L.predict_rank(x, 1, k, n16, n8, None, tiers)
    L.cache_plan(tiers, 1, 0)
    L.cache_fill()
    y = torch.zeros((1, ld.d_model), dtype=torch.float32, device="cuda")
    say("give-up: withheld h values")
    m2c.m2c_debug_ffn_withhold_h(L.handle, 16)
    L.sparse_ffn(x, 1, y)
    torch.cuda.synchronize()
    assert not y.cpu().numpy().any()  # every down task took h = 0
    with pytest.raises(m2c.M2CError) as e:
        L.stats()
    assert e.value.status == m2c.M2C_ERR_STATE
    L.stats()  # reported once, then cleared
    m2c.m2c_debug_ffn_withhold_h(L.handle, 0)
    plan = L.read_plan()
    y_ref = oracle_ffn(ld, ld.x[0], plan["req_ids"], plan["req_tier"])[0]
    for t in range(2):
        say(f"give-up: normal call {t}")
        y.zero_()
        L.sparse_ffn(x, 1, y)
        torch.cuda.synchronize()
        assert r8_errors(y.cpu().numpy()[0], y_ref).max() <= FFN_TOL
    L.stats()
    L.close()


@pytest.mark.parametrize("d,d_ff", [(1024, 2752), (1536, 2000), (2048, 2000), (3072, 2000),
                                    (4096, 3000), (5120, 2000), (8192, 3000)])
def test_ffn_modes_accumulate_and_determinism(d, d_ff):
    """Both FFN paths add into y; the deterministic path repeats bit for bit
    and the fused path agrees with it to fp32 rounding. (Each of the fused
    path's per-workgroup atomic adds rounds at the magnitude of what y already
    holds, so the cross-mode check starts from y = 0; a column's sum is one
    fp32 partial per down task that covers it, and their number follows the
    task geometry, so the cross-mode bound is a quarter of the oracle
    tolerance rather than a fixed multiple of one rounding.) The widths cover
    every fused kernel instance: K = 1, 2, 4 and 8 sixteen-byte loads per
    lane and unit, each with d = 1024 K (K > 1) and with another d."""
    ld = W.make_layer(61, 0, d, d_ff, 64, 1)
    k = d_ff // 5
    n16, n8 = _counts(k, (1, 10), (2, 5))
    outs = {}
    for flags in (0, m2c.FLAG_DETERMINISTIC_FFN):
        say(f"ffn modes d={d} flags={flags}")
        L = _layer(ld, k, k, flags=flags)
        tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
        x = _x16(ld, 0)
        L.predict_rank(x, 1, k, n16, n8, None, tiers)
        L.cache_plan(tiers, 1, 0)
        L.cache_fill()
        ys = []
        for _ in range(3):
            y = torch.zeros((1, d), dtype=torch.float32, device="cuda")
            L.sparse_ffn(x, 1, y)
            ys.append(y)
        base = torch.linspace(-1.0, 1.0, d, device="cuda").reshape(1, d)
        yb = base.clone()
        L.sparse_ffn(x, 1, yb)
        torch.cuda.synchronize()
        ys = [yy.cpu().numpy()[0] for yy in ys]
        if flags:
            assert all(np.array_equal(ys[0], yy) for yy in ys[1:])
        plan = L.read_plan()
        y_ref = oracle_ffn(ld, ld.x[0], plan["req_ids"], plan["req_tier"])[0]
        for yy in ys:
            assert r8_errors(yy, y_ref).max() <= FFN_TOL
        acc = (yb - base).cpu().numpy()[0].astype(np.float64)
        assert r8_errors(acc, y_ref).max() <= FFN_TOL  # accumulated into y
        outs[flags] = ys[0]
        L.close()
    assert r8_errors(outs[0], outs[m2c.FLAG_DETERMINISTIC_FFN]).max() <= FFN_TOL / 4


def test_plan_overflow_is_reported():
    """A tier map with more active neurons than the plan capacity leaves the
    plan empty and the cache unchanged; m2c_layer_stats reports it once."""
    ld = W.make_layer(17, 0, 256, 200, 16, 2)
    L = _layer(ld, 20, 30)  # capacity min(d_ff, 1 * 20) = 20
    tiers = torch.full((1, 200), 1, dtype=torch.uint8, device="cuda")  # 200 active
    say("plan overflow")
    L.cache_plan(tiers, 1, 0)
    torch.cuda.synchronize()
    assert L.read_plan()["counts"][m2c.CNT_REQ] == 0
    with pytest.raises(m2c.M2CError) as e:
        L.stats()
    assert e.value.status == m2c.M2C_ERR_CAPACITY
    st = L.stats()  # reported once, then cleared
    assert st.req == 0 and st.plans == 0
    slot_of, key, _, _ = m2c.m2c_debug_read_tables(L.handle, 200, 30)
    assert (slot_of == -1).all() and (key == -1).all()
    L.close()


def test_one_launch_ffn_call_tags_and_graph_replay():
    """The batch-1 FFN tags its h values with a per-call count kept on the
    device: calls that reuse one plan with different x never read an h of an
    earlier call, and a graph that captured the launch is correct on every
    replay (the count advances without any host argument)."""
    ld = W.make_layer(W.WORKLOADS["tiny"].seed, 3, 1024, 2752, 128, 6)
    k = 688
    n16, n8 = _counts(k)
    L = _layer(ld, k, 1376)
    tiers = torch.empty((1, ld.d_ff), dtype=torch.uint8, device="cuda")
    say("call tags: plan")
    L.predict_rank(_x16(ld, 0), 1, k, n16, n8, None, tiers)
    L.cache_plan(tiers, 1, 0)
    L.cache_fill()
    torch.cuda.synchronize()
    plan = L.read_plan()

    def ref(t):
        return oracle_ffn(ld, ld.x[t], plan["req_ids"], plan["req_tier"])[0]

    # eager calls on one plan, x changing every call
    for t in (1, 2, 1, 3):
        say(f"call tags: eager x[{t}]")
        y = torch.zeros((1, ld.d_model), dtype=torch.float32, device="cuda")
        L.sparse_ffn(_x16(ld, t), 1, y)
        torch.cuda.synchronize()
        assert r8_errors(y.cpu().numpy()[0], ref(t)).max() <= FFN_TOL, f"eager call with x[{t}]"
    # graph: zero y (a kernel, not a memset) and the FFN on a fixed x buffer
    xg = _x16(ld, 0).clone()
    yg = torch.zeros((1, ld.d_model), dtype=torch.float32, device="cuda")
    ye = torch.zeros((1, ld.d_model), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    say("call tags: capture")
    with torch.cuda.graph(g, stream=s):
        yg.zero_()
        L.sparse_ffn(xg, 1, yg)
    torch.cuda.synchronize()
    for t in (4, 5, 4):
        say(f"call tags: replay with x[{t}]")
        xg.copy_(_x16(ld, t))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert r8_errors(yg.cpu().numpy()[0], ref(t)).max() <= FFN_TOL, f"replay with x[{t}]"
        # eager work between replays advances the same counters
        ye.zero_()
        L.sparse_ffn(_x16(ld, 2), 1, ye)
        torch.cuda.synchronize()
        assert r8_errors(ye.cpu().numpy()[0], ref(2)).max() <= FFN_TOL
    del g
    L.stats()  # no wait was given up
    L.close()


def test_widest_layer_uses_two_kernel_ffn():
    """d_model = 16384, the widest layer the library takes: the batch-1 FFN
    runs as two kernels there (the one-launch kernel stages x for d <= 8192);
    every stage against the oracle over two steps."""
    ld = W.make_layer(29, 0, 16384, 600, 32, 2)
    k = 150
    n16, n8 = _counts(k)
    worst, _ = _run_steps(ld, 2, k, n16, n8, 300, label="d=16384")
    say(f"d=16384 worst FFN error {worst:.2e}")
