"""Pins of the CPU oracle against what the definitions and the mathematics fix.

Each test checks the oracle against something other than itself: a library
routine (numpy's fp16 conversion, fp64 matmul, lexsort), a brute force over
every candidate, a closed form (the Adjacent Token Update hit count), or a
value worked out by hand from the definition.
"""
import numpy as np
import pytest

import oracle
from paper_2410_14740_amd import workloads as W


# --------------------------------------------------------------------------
# fp16 conversions (the format every weight, activation and scale uses)

def test_f16_to_f32_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.f16_to_f32(bits)
    ref = bits.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_f32_to_f16_rne_matches_numpy():
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(0.02),
        (rng.standard_normal(50000) * 1e-6).astype(np.float32),   # subnormal range
        (rng.standard_normal(50000) * 3e4).astype(np.float32),    # near overflow
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 65536.0, 1e9, -1e9,
                  2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -14, np.inf, -np.inf],
                 np.float32),
    ])
    # exact ties between two fp16 neighbours: midpoints of random fp16 pairs
    h = rng.integers(0, 0x7bff, 20000).astype(np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    vals = np.concatenate([vals, ((lo + hi) / 2).astype(np.float32)])
    ours = oracle.f32_to_f16(vals)
    with np.errstate(over="ignore"):
        ref = vals.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)


# --------------------------------------------------------------------------
# quantization and records

def _tiny_weights(d=256, d_ff=6, seed=3):
    lw = W.make_layer(seed, 0, d, d_ff, 8, 1)
    return lw.w_gate, lw.w_up, lw.w_down


def _vectors(wg, wu, wd, i):
    return [wg[i].astype(np.float64), wu[i].astype(np.float64), wd[:, i].astype(np.float64)]


def _decode_int(rec, d, tier):
    """Independent numpy decode of an INT8 / INT4 record -> (codes [3][d], scales [3][G])."""
    G = d // 128
    cb = d if tier == 2 else d // 2
    codes = []
    for v in range(3):
        raw = rec[v * cb:(v + 1) * cb]
        if tier == 2:
            codes.append(raw.view(np.int8).astype(np.int64))
        else:
            lo = (raw & 0xF).astype(np.int64)
            hi = (raw >> 4).astype(np.int64)
            q = np.empty(d, np.int64)
            q[0::2], q[1::2] = lo, hi
            codes.append(np.where(q >= 8, q - 16, q))
    sc = rec[3 * cb:3 * cb + 6 * G].view(np.float16).astype(np.float64).reshape(3, G)
    return np.stack(codes), sc


@pytest.mark.parametrize("tier,qmax", [(2, 127), (1, 7)])
def test_quant_brute_force_argmin(tier, qmax):
    d = 256
    wg, wu, wd = _tiny_weights(d)
    recs = oracle.build_records(wg, wu, wd, tier)
    assert recs.shape[1] == oracle.record_stride(d, tier)
    cand = np.arange(-qmax, qmax + 1, dtype=np.float64)
    for i in range(wg.shape[0]):
        codes, sc = _decode_int(recs[i], d, tier)
        for v, vec in enumerate(_vectors(wg, wu, wd, i)):
            for g in range(d // 128):
                w = vec[g * 128:(g + 1) * 128]
                s = sc[v, g]
                # scale: fp16(fp32(amax) / qmax), via numpy's IEEE fp32 and fp16 rounding
                amax = np.float32(np.max(np.abs(w)))
                assert s == np.float64(np.float16(amax / np.float32(qmax)))
                # code: argmin_q |w - q s| over every candidate, ties to the even code
                err = np.abs(w[:, None] - cand[None, :] * s)
                best = err.min(axis=1, keepdims=True)
                tie = err == best
                n_win = tie.sum(axis=1)
                # one winner, or two adjacent codes tied: take the even one
                even_win = tie & (np.abs(cand[None, :]) % 2 == 0)
                pick = np.where(n_win == 1, cand[np.argmax(tie, axis=1)],
                                cand[np.argmax(even_win, axis=1)])
                assert np.all((n_win == 1) | (even_win.sum(axis=1) == 1))
                assert np.array_equal(codes[v, g * 128:(g + 1) * 128], pick.astype(np.int64))
                # in-range error bound of round to nearest
                assert np.all(np.abs(w - codes[v, g * 128:(g + 1) * 128] * s) <= s / 2 + 0.0)


def test_quant_hand_worked_ties_and_zero_group():
    """Hand-worked groups: INT8 with amax = 127 * 2^-10 gives s = 2^-10, so
    w = 2.5 s -> 2, 3.5 s -> 4, -2.5 s -> -2 (half to even); an all-zero group
    has s = 0 and codes 0. INT4 with amax = 7 * 2^-6 gives s = 2^-6."""
    d, d_ff = 128, 1
    wg = np.zeros((d_ff, d), np.float16)
    wu = np.zeros((d_ff, d), np.float16)
    wd = np.zeros((d, d_ff), np.float16)
    s8 = 2.0 ** -10
    wg[0, :5] = np.array([127 * s8, 2.5 * s8, 3.5 * s8, -2.5 * s8, 0.5 * s8])
    s4 = 2.0 ** -6
    wu[0, :5] = np.array([7 * s4, 2.5 * s4, 1.5 * s4, -0.5 * s4, -7 * s4])
    r8 = oracle.build_records(wg, wu, wd, 2)[0]
    c8, sc8 = _decode_int(r8, d, 2)
    assert sc8[0, 0] == s8 and list(c8[0, :5]) == [127, 2, 4, -2, 0]
    assert sc8[2, 0] == 0.0 and not c8[2].any()          # zero group
    r4 = oracle.build_records(wg, wu, wd, 1)[0]
    c4, sc4 = _decode_int(r4, d, 1)
    assert sc4[1, 0] == s4 and list(c4[1, :5]) == [7, 2, 2, 0, -7]
    # nibble order: element 0 in the low nibble of byte 0 of the up vector
    up_codes = r4[d // 2:d]
    assert up_codes[0] == ((2 & 0xF) << 4 | (7 & 0xF))


def test_fp16_record_is_exact_copy():
    wg, wu, wd = _tiny_weights(256, 4)
    r = oracle.build_records(wg, wu, wd, 3)
    assert r.shape[1] == 6 * 256
    for i in range(4):
        got = r[i].view(np.float16)
        assert np.array_equal(got[:256], wg[i])
        assert np.array_equal(got[256:512], wu[i])
        assert np.array_equal(got[512:], wd[:, i])
        g, u, dn = oracle.dequant_record(r[i], 256, 3)
        assert np.array_equal(g, wg[i].astype(np.float64))
        assert np.array_equal(dn, wd[:, i].astype(np.float64))


def test_record_sizes():
    for d in (128, 1024, 4096, 5120, 8192):
        G = d // 128
        assert oracle.record_bytes(d, 3) == 6 * d
        assert oracle.record_bytes(d, 2) == 3 * d + 6 * G
        assert oracle.record_bytes(d, 1) == 3 * d // 2 + 6 * G
    # the record sizes of the 70B-shaped layer
    assert [oracle.record_bytes(8192, t) for t in (3, 2, 1)] == [49152, 24960, 12672]


# --------------------------------------------------------------------------
# predictor

def test_predict_within_fp32_bound_of_fp64():
    lw = W.make_layer(11, 0, 1024, 700, 48, 2)
    x = lw.x[1, 0]
    z, s = oracle.predict(lw.pred_a, lw.pred_b, None, x)
    A = lw.pred_a.astype(np.float64)
    xd = x.astype(np.float64)
    z64 = A @ xd
    gam = lambda n: n * 2.0 ** -24 / (1 - n * 2.0 ** -24)
    assert np.all(np.abs(z - z64) <= gam(1024) * (np.abs(A) @ np.abs(xd)))
    Bm = lw.pred_b.astype(np.float64)
    zd = z.astype(np.float64)
    s64 = Bm @ zd
    assert np.all(np.abs(s - s64) <= gam(48) * (np.abs(Bm) @ np.abs(zd)))
    assert np.max(np.abs(z - z64) / (np.abs(z64) + 1e-3)) < 1e-5


def test_predict_basis_vector_and_bias():
    d, d_ff, r = 256, 50, 16
    lw = W.make_layer(5, 0, d, d_ff, r, 1)
    x = np.zeros(d, np.float16)
    x[37] = 1.0
    z, s = oracle.predict(lw.pred_a, lw.pred_b, None, x)
    assert np.array_equal(z, lw.pred_a[:, 37].astype(np.float32))
    bias = np.random.default_rng(0).standard_normal(d_ff).astype(np.float32)
    _, sb = oracle.predict(lw.pred_a, lw.pred_b, bias, x)
    assert np.array_equal(sb, s + bias)  # one fp32 addition after the dot product


def test_predict_hand_worked_order():
    """n = 16 gives L = 2 partial sums: chunk 0 -> partial 0, chunk 1 -> partial 1.
    Partial 0 = 256*256 = 65536. Partial 1 = fma(-256, 256, fma(2^-4, 2^-4, 0))
    = -65536 + 2^-8 (exact, the fp32 spacing there is 2^-8). Sum = 2^-8. A plain
    left-to-right sum would give (65536 + 2^-8) -> 65536 (tie to even), then 0."""
    A = np.zeros((8, 16), np.float16)  # rank 8; only row 0 is non-zero
    x = np.zeros(16, np.float16)
    A[0, 0], x[0] = 256.0, 256.0
    A[0, 8], x[8] = 2.0 ** -4, 2.0 ** -4
    A[0, 9], x[9] = -256.0, 256.0
    Bm = np.ones((1, 8), np.float16)
    z, _ = oracle.predict(A, Bm, None, x)
    assert z[0] == np.float32(2.0 ** -8)


# --------------------------------------------------------------------------
# top-k and tiers

def _lexsort_tiers(s, k, n16, n8):
    order = np.lexsort((np.arange(s.size), -s.astype(np.float64)))
    tier = np.zeros(s.size, np.uint8)
    tier[order[:n16]] = 3
    tier[order[n16:n16 + n8]] = 2
    tier[order[n16 + n8:k]] = 1
    return tier, order[:k]


@pytest.mark.parametrize("d_ff,k,n16,n8", [(2752, 688, 229, 229), (1000, 1000, 100, 400),
                                           (1000, 0, 0, 0), (777, 13, 13, 0), (64, 63, 0, 0)])
def test_select_matches_lexsort(d_ff, k, n16, n8):
    s = np.random.default_rng(d_ff + k).standard_normal(d_ff).astype(np.float32)
    s[5:9] = s[4]  # some exact ties, broken by id
    tier, ranked = oracle.select_tiers(s, k, n16, n8)
    rt, ro = _lexsort_tiers(s, k, n16, n8)
    assert np.array_equal(tier, rt)
    assert np.array_equal(ranked, ro)


def test_select_all_equal_and_signed_zero():
    s = np.full(100, 0.25, np.float32)
    tier, _ = oracle.select_tiers(s, 10, 3, 3)
    assert list(tier[:10]) == [3, 3, 3, 2, 2, 2, 1, 1, 1, 1] and not tier[10:].any()
    s = np.array([-0.0, 0.0, -1.0], np.float32)
    tier, ranked = oracle.select_tiers(s, 1, 1, 0)
    assert list(ranked) == [1]  # +0.0 ranks above -0.0


# --------------------------------------------------------------------------
# LRU slot cache

def _brute_lru_step(state, tiers, step, C, dominance=False):
    """Brute force of one atomic step: sort every untouched slot by
    (last use, slot) and hand them out in that order. dominance: a neuron
    resident at a tier at or above the requested one is a hit at its resident
    tier (tiers[i] is updated to the tier the step uses)."""
    slot_of, key, stier, last = state
    req = [i for i in sorted(tiers) if tiers[i] > 0]
    touched = set()
    res = {}
    for i in req:
        if i in slot_of:
            s = slot_of[i]
            touched.add(s)
            hit = stier[s] == tiers[i] or (dominance and stier[s] > tiers[i])
            res[i] = ("HIT" if hit else "REFILL", s, stier[s])
            if hit:
                tiers[i] = stier[s]
            stier[s] = tiers[i]
    free = sorted((last[s], s) for s in range(C) if s not in touched)
    new = [i for i in req if i not in slot_of]
    evicted, nb = [], 0
    for j, i in enumerate(new):
        if j < len(free):
            s = free[j][1]
            if key[s] is not None:
                evicted.append(key[s])
                del slot_of[key[s]]
            key[s], stier[s], slot_of[i] = i, tiers[i], s
            res[i] = ("NEW", s)
        else:
            res[i] = ("BYPASS", C + nb)
            nb += 1
    for i in req:
        if res[i][0] != "BYPASS":
            last[res[i][1]] = step
    return req, res, evicted


@pytest.mark.parametrize("policy", [oracle.POLICY_EXACT, oracle.POLICY_DOMINANCE])
@pytest.mark.parametrize("d_ff,C,B", [(40, 7, 1), (40, 12, 3), (25, 25, 2), (30, 0, 1)])
def test_lru_matches_brute_force(d_ff, C, B, policy):
    rng = np.random.default_rng(d_ff * 100 + C)
    S = d_ff
    dom = policy == oracle.POLICY_DOMINANCE
    cache = oracle.LRUCache(d_ff, C, S, policy)
    st = ({}, [None] * C, [0] * C, [-1] * C)
    code = {"NEW": 0, "HIT": 1, "REFILL": 2, "BYPASS": 3}
    derived = tier_hits = 0
    for step in range(30):
        tm = np.zeros((B, d_ff), np.uint8)
        for b in range(B):
            ids = rng.choice(d_ff, size=rng.integers(0, 10), replace=False)
            tm[b, ids] = rng.integers(1, 4, size=ids.size)
        p = cache.plan(tm, step)
        tiers = {i: int(tm[:, i].max()) for i in range(d_ff)}
        asked = dict(tiers)
        req, res, ev = _brute_lru_step(st, tiers, step, C, dominance=dom)
        assert list(p["req_ids"]) == req
        assert [code[res[i][0]] for i in req] == list(p["req_hit"])
        assert [res[i][1] for i in req] == list(p["req_slot"])
        assert list(p["req_tier"]) == [tiers[i] for i in req]
        assert list(p["evicted_ids"]) == ev
        assert list(p["fill_ids"]) == [i for i in req if res[i][0] != "HIT"]
        # the tier a REFILL's slot held before the step (0 for NEW / BYPASS)
        frm = [res[i][2] if res[i][0] == "REFILL" else 0 for i in req if res[i][0] != "HIT"]
        assert list(p["fill_from"]) == frm
        # an FP16 record refilled to INT8 / INT4 happens only under exact tiers
        derived += sum(1 for f, i in zip(frm, p["fill_ids"]) if f == 3 and tiers[i] < 3)
        tier_hits += sum(1 for i in req if res[i][0] == "HIT" and tiers[i] != asked[i])
        c = p["counts"]
        assert c[0] == c[1] + c[2] + c[3] + c[4] == len(req)
        assert c[6] == c[2] + c[3] + c[4] == c[10] + c[11] + c[12]
        assert [c[7], c[8], c[9]] == [sum(1 for i in req if tiers[i] == t) for t in (3, 2, 1)]
        assert not c[13:].any()
        # masks: bit b set iff row b selected the neuron
        for n_, i in enumerate(req):
            assert p["req_mask"][n_] == sum(1 << b for b in range(B) if tm[b, i] > 0)
        # tables: the same as the brute force's, and inverse maps of each other
        assert {i: int(cache.slot_of[i]) for i in range(d_ff) if cache.slot_of[i] >= 0} == st[0]
        for s_ in range(C):
            k_ = cache.slot_key[s_]
            assert (k_ if k_ >= 0 else None) == st[1][s_]
            assert cache.slot_last[s_] == st[3][s_]
            if k_ >= 0:
                assert cache.slot_of[k_] == s_ and cache.slot_tier[s_] == st[2][s_]
    if dom:
        assert derived == 0 and (C == 0 or tier_hits > 0)  # hits above the requested tier
    else:
        assert tier_hits == 0 and (C == 0 or derived > 0)  # FP16 -> lower-tier refills


def test_lru_dominance_closed_form_when_everything_fits():
    """Dominance hits with C >= d_ff: nothing is ever evicted, a resident
    tier only rises, so neuron i is resident at the highest tier requested so
    far; a request at tier t is a hit iff i was requested before at some
    tier >= t, and the step then uses that highest tier."""
    d_ff = 50
    cache = oracle.LRUCache(d_ff, d_ff, 0, oracle.POLICY_DOMINANCE)
    rng = np.random.default_rng(5)
    best = np.zeros(d_ff, np.int64)
    for t in range(40):
        tm = np.zeros(d_ff, np.uint8)
        ids = rng.choice(d_ff, 12, replace=False)
        tm[ids] = rng.integers(1, 4, size=ids.size)
        p = cache.plan(tm, t)
        req = np.nonzero(tm)[0]
        hit = best[req] >= tm[req]
        assert list(p["req_ids"]) == list(req)
        assert list(p["req_hit"] == 1) == list(hit)
        assert list(p["req_tier"]) == list(np.where(hit, best[req], tm[req]))
        assert int(p["counts"][1]) == int(hit.sum()) and int(p["counts"][5]) == 0
        best[req] = np.maximum(best[req], tm[req])


def test_lru_dominance_equals_exact_with_one_tier():
    """With every active neuron at one tier the two policies are the same
    cache (no resident tier differs from a requested one)."""
    d_ff, C = 120, 30
    a = oracle.LRUCache(d_ff, C, d_ff, oracle.POLICY_EXACT)
    b = oracle.LRUCache(d_ff, C, d_ff, oracle.POLICY_DOMINANCE)
    rng = np.random.default_rng(8)
    for t in range(30):
        tm = np.zeros((2, d_ff), np.uint8)
        for r in range(2):
            tm[r, rng.choice(d_ff, 20, replace=False)] = 2
        pa, pb = a.plan(tm, t), b.plan(tm, t)
        for key in pa:
            assert np.array_equal(pa[key], pb[key]), key


def test_lru_atu_closed_form():
    """C = k, one tier, batch 1: every slot holds the previous token's active
    set, so the hits of step t are exactly |S_t & S_{t-1}| (the Adjacent Token
    Update policy of Sec. 5.3)."""
    d_ff, k = 500, 60
    lw = W.make_layer(21, 0, 256, d_ff, 32, 20, rhos=(0.9,))
    cache = oracle.LRUCache(d_ff, k, 0)
    prev = None
    for t in range(20):
        _, s = oracle.predict(lw.pred_a, lw.pred_b, None, lw.x[t, 0])
        tier, _ = oracle.select_tiers(s, k, k, 0)
        cur = set(np.nonzero(tier)[0])
        p = cache.plan(tier, t)
        hits = int(p["counts"][1])
        assert hits == (len(cur & prev) if prev is not None else 0)
        assert int(p["counts"][6]) == k - hits and int(p["counts"][4]) == 0
        prev = cur


def test_lru_never_evicts_when_everything_fits():
    d_ff = 64
    cache = oracle.LRUCache(d_ff, d_ff, 0)
    rng = np.random.default_rng(2)
    seen = set()
    for t in range(40):
        tm = np.zeros(d_ff, np.uint8)
        ids = rng.choice(d_ff, 10, replace=False)
        tm[ids] = 3
        p = cache.plan(tm, t)
        assert p["counts"][5] == 0 and p["counts"][4] == 0
        assert p["counts"][3] == len(set(ids) - seen)
        seen |= set(ids)


def test_lru_evicts_least_recent_first():
    """LRU property, with independent bookkeeping of every neuron's last use:
    no evicted neuron was used more recently than a neuron left resident."""
    d_ff, C = 80, 20
    cache = oracle.LRUCache(d_ff, C, d_ff)
    last_use = {}
    rng = np.random.default_rng(9)
    for t in range(60):
        tm = np.zeros(d_ff, np.uint8)
        ids = rng.choice(d_ff, rng.integers(1, 12), replace=False)
        tm[ids] = 3
        resident_before = {i for i in range(d_ff) if cache.slot_of[i] >= 0}
        p = cache.plan(tm, t)
        ev = set(p["evicted_ids"].tolist())
        kept = {i for i in range(d_ff) if cache.slot_of[i] >= 0} - set(ids.tolist())
        assert ev <= resident_before
        if ev and kept:
            assert max(last_use[i] for i in ev) <= min(last_use[i] for i in kept)
        for i in ids:
            last_use[int(i)] = t


# --------------------------------------------------------------------------
# sparse FFN

def _silu(a):
    return a / (1.0 + np.exp(-a))


def test_sparse_all_fp16_equals_dense():
    d, d_ff = 256, 300
    lw = W.make_layer(31, 0, d, d_ff, 16, 1)
    x = lw.x[0, 0]
    rec = oracle.build_records(lw.w_gate, lw.w_up, lw.w_down, 3)
    ids = np.arange(d_ff, dtype=np.int32)
    y = oracle.sparse_ffn(x, ids, np.full(d_ff, 3, np.uint8), {3: rec})[0]
    yd = oracle.dense_ffn(lw.w_gate, lw.w_up, lw.w_down, x)
    xd = x.astype(np.float64)
    ref = lw.w_down.astype(np.float64) @ (_silu(lw.w_gate.astype(np.float64) @ xd)
                                          * (lw.w_up.astype(np.float64) @ xd))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-15)
    assert np.allclose(yd, ref, rtol=1e-12, atol=1e-15)


def test_sparse_mixed_tiers_matches_numpy_decode():
    d, d_ff = 384, 90
    lw = W.make_layer(41, 0, d, d_ff, 16, 2, rhos=(0.9, 0.5))
    recs = {t: oracle.build_records(lw.w_gate, lw.w_up, lw.w_down, t) for t in (1, 2, 3)}
    rng = np.random.default_rng(4)
    ids = np.sort(rng.choice(d_ff, 40, replace=False)).astype(np.int32)
    tiers = rng.integers(1, 4, 40).astype(np.uint8)
    masks = rng.integers(1, 4, 40).astype(np.uint32)
    x = lw.x[1]
    y = oracle.sparse_ffn(x, ids, tiers, recs, masks)
    for b in range(2):
        xd = x[b].astype(np.float64)
        ref = np.zeros(d)
        for i, t, m in zip(ids, tiers, masks):
            if not (m >> b) & 1:
                continue
            if t == 3:
                g, u, dn = (lw.w_gate[i].astype(np.float64), lw.w_up[i].astype(np.float64),
                            lw.w_down[:, i].astype(np.float64))
            else:
                codes, sc = _decode_int(recs[t][i], d, t)
                deq = codes * np.repeat(sc, 128, axis=1)
                g, u, dn = deq
            ref += _silu(g @ xd) * (u @ xd) * dn
        assert np.allclose(y[b], ref, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# workload count rules

def test_workload_counts():
    got = {n: (w.counts(), w.cache_slots()) for n, w in W.WORKLOADS.items()}
    assert got["tiny"] == ((688, 229, 229), 1376)
    assert got["llama2-7b"] == ((2201, 220, 880), 3302)
    assert got["llama2-13b"] == ((2073, 414, 622), 2764)
    assert got["llama2-70b"] == ((2867, 286, 860), 2867)
    assert W.tier_counts(11008, W.F(1, 5), 1, 0) == (2201, 2201, 0)


def test_inputs_are_ar1_with_unit_marginals():
    x = W.layer_inputs(7, 0, 4096, 64, (0.9,)).astype(np.float64)[:, 0]
    assert abs(x.std() - 1.0) < 0.05
    c = np.mean([np.corrcoef(x[t], x[t + 1])[0, 1] for t in range(63)])
    assert abs(c - 0.9) < 0.02


def test_oracle_results_do_not_depend_on_threads():
    """Threads only split independent sums: records, scores and the FFN are
    the same bits at one thread and at several."""
    lw = W.make_layer(31, 0, 512, 300, 32, 2, rhos=(0.9, 0.5, 0.7))
    ids = np.arange(0, 300, 3, dtype=np.int32)
    tiers = (ids % 3 + 1).astype(np.uint8)
    masks = (ids % 7 + 1).astype(np.uint32)
    outs = []
    for n in (1, 4):
        oracle.set_threads(n)
        recs = {t: oracle.build_records(lw.w_gate, lw.w_up, lw.w_down, t) for t in (1, 2, 3)}
        _, sc = oracle.predict(lw.pred_a, lw.pred_b, None, lw.x[1, 0])
        y = oracle.sparse_ffn(lw.x[0], ids, tiers, recs, masks)
        outs.append((recs, sc, y))
    oracle.set_threads(1)
    (r1, s1, y1), (r4, s4, y4) = outs
    assert all(np.array_equal(r1[t], r4[t]) for t in (1, 2, 3))
    assert np.array_equal(s1.view(np.uint32), s4.view(np.uint32))
    assert np.array_equal(y1.view(np.uint64), y4.view(np.uint64))


@pytest.mark.parametrize("policy,d_ff,C", [
    (oracle.POLICY_EXACT, 60, {3: 3, 2: 5, 1: 8}),
    (oracle.POLICY_DOMINANCE, 60, {3: 3, 2: 5, 1: 8}),
    (oracle.POLICY_DOMINANCE, 30, {3: 10, 2: 10, 1: 6})])
def test_tier_pools_are_independent_lru_caches(policy, d_ff, C):
    """The per-tier arena: each pool is the step-atomic LRU brute force over
    the requests of its tier alone, slots numbered in tier blocks; the merged
    lists are the pools' lists in ascending id; no REFILL ever happens.
    Dominance: a neuron not resident in its own tier's pool but resident (at
    the step's start, in the brute force's own tables) in a pool of higher
    precision is that lowest such pool's request, a HIT at its tier."""
    B = 2
    S = {3: 20, 2: 20, 1: 20}
    cache = oracle.TierPoolCache(d_ff, C, S, policy)
    first = {3: 0, 2: C[3] + S[3], 1: C[3] + S[3] + C[2] + S[2]}
    states = {t: ({}, [None] * C[t], [0] * C[t], [-1] * C[t]) for t in (3, 2, 1)}
    rng = np.random.default_rng(12)
    code = {"NEW": 0, "HIT": 1, "REFILL": 2, "BYPASS": 3}
    dominance_hits = 0
    for step in range(40):
        tm = np.zeros((B, d_ff), np.uint8)
        for b in range(B):
            ids = rng.choice(d_ff, size=rng.integers(0, 12), replace=False)
            tm[b, ids] = rng.integers(1, 4, size=ids.size)
        p = cache.plan(tm, step)
        st = tm.max(axis=0)
        if policy == oracle.POLICY_DOMINANCE:
            for i in range(d_ff):
                t = int(st[i])
                if t and i not in states[t][0]:
                    up = [u for u in (1, 2, 3) if u > t and i in states[u][0]]
                    if up:
                        st[i] = min(up)
                        dominance_hits += 1
        want = {}
        evicted = []
        for t in (3, 2, 1):
            tiers = {i: (t if st[i] == t else 0) for i in range(d_ff)}
            req, res, ev = _brute_lru_step(states[t], tiers, step, C[t])
            for i in req:
                want[i] = (t, code[res[i][0]], first[t] + res[i][1])
            evicted += ev
        req = sorted(want)
        assert list(p["req_ids"]) == req
        assert list(p["req_tier"]) == [want[i][0] for i in req]
        assert list(p["req_hit"]) == [want[i][1] for i in req]
        assert list(p["req_slot"]) == [want[i][2] for i in req]
        assert 2 not in p["req_hit"]
        assert list(p["fill_ids"]) == [i for i in req if want[i][1] != 1]
        assert list(p["evicted_ids"]) == evicted
        assert not p["fill_from"].any()
    if policy == oracle.POLICY_DOMINANCE:
        assert dominance_hits > 10
