"""The decode schedule the benchmark times (paper_2410_14740_amd.pipeline:
predict + plan on an aux stream, fills on a copy stream, the FFN on the main
stream, cross-stream events with a look-ahead lag) against the oracle.

Every layer-step's plan (as the FFN saw it: copied on the main stream right
after the FFN), FFN output, the final slot tables and the layer counters are
compared with the oracle. The race variants make ordering mistakes visible:

  * each stream is held by a spin kernel of a seeded random length before its
    stage, so the stages of different layer-steps are pushed against each
    other in many orders;
  * every slot a fill writes is overwritten with 0xFF bytes on the copy
    stream right before the fill: an FFN that read a slot before its fill
    completed would read NaN, and a fill (or its poison) that started while
    an earlier FFN still read the slot would corrupt that FFN's output.
"""
import numpy as np
import pytest

import oracle
from paper_2410_14740_amd import m2c
from paper_2410_14740_amd import pipeline
from paper_2410_14740_amd import workloads as W

from helpers import FFN_TOL, derived_fills, oracle_ffn, r8_errors, say, work_order

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


class _Hooks:
    """Held streams, poisoned fill slots and the plan archive."""

    def __init__(self, layers, archive, hold, poison, seed):
        self.layers = layers
        self.archive = archive
        self.hold = hold
        self.poison = poison
        self.rng = np.random.default_rng(seed)

    def _spin(self, s):
        if self.hold:
            cycles = int(self.rng.integers(20_000, 400_000))  # about 10 to 200 us
            with torch.cuda.stream(s):
                torch.cuda._sleep(cycles)

    def before_predict(self, l, t, s):
        self._spin(s)

    def before_fill(self, l, t, s):
        self._spin(s)
        if self.poison:
            L = self.layers[l]
            m2c.m2c_debug_poison_fill_slots(L.handle, L.plan, s)

    def before_ffn(self, l, t, s):
        self._spin(s)

    def after_ffn(self, l, t, s):
        with torch.cuda.stream(s):
            self.archive[t, l].copy_(self.layers[l].plan)


def _check_plan(L, raw, o, where):
    g = L.read_plan(plan=raw)
    for key in ("req_ids", "req_tier", "req_hit", "req_slot", "req_mask", "fill_ids", "fill_tier",
                "fill_slot", "fill_from", "evicted_ids"):
        assert np.array_equal(g[key], o[key]), f"{where}: plan field {key} differs"
    assert np.array_equal(g["counts"][:13], o["counts"][:13]), f"{where}: counts differ"
    ws, wm = work_order(o)
    assert np.array_equal(g["work_slot"], ws) and np.array_equal(g["work_mask"], wm), \
        f"{where}: FFN work order differs"
    assert g["counts"][m2c.CNT_FILL_DERIVED] == derived_fills(o), f"{where}: derived count"


POOLS = {3: 20, 2: 80, 1: 120}  # below each tier's demand (35 / 140 / 175)


@pytest.mark.parametrize("n_layers,lag,hold,poison,flags,batch", [
    (4, 2, False, False, 0, 1),
    (4, 2, True, True, 0, 1),
    (2, 1, True, True, 0, 1),
    (3, 2, True, True, m2c.FLAG_DOMINANT_HITS, 1),
    (3, 2, True, True, m2c.FLAG_TIER_POOLS, 1),
    (3, 2, True, True, m2c.FLAG_TIER_POOLS | m2c.FLAG_DOMINANT_HITS, 1),
    (3, 2, True, True, 0, 4),
    (3, 2, True, True, m2c.FLAG_DOMINANT_HITS, 4),
])
def test_three_stream_schedule(n_layers, lag, hold, poison, flags, batch):
    d, d_ff, r, steps = 512, 1400, 32, 12
    k = 350
    n16, n8 = k // 10, (k // 2) - k // 10
    C = 250  # below k: evictions and bypasses through staging slots every step
    pools = bool(flags & m2c.FLAG_TIER_POOLS)
    desc = (m2c.make_desc(d, d_ff, r, k, 0, flags=flags & ~m2c.FLAG_TIER_POOLS, tier_slots=POOLS)
            if pools else m2c.make_desc(d, d_ff, r, k, C, max_batch=batch, flags=flags))
    policy = oracle.POLICY_DOMINANCE if flags & m2c.FLAG_DOMINANT_HITS else oracle.POLICY_EXACT
    rhos = (0.8, 0.5, 0.9, 0.7)[:batch]
    lds = [W.make_layer(900 + n_layers, l, d, d_ff, r, steps, rhos=rhos) for l in range(n_layers)]
    layers = [m2c.Layer(desc, ld) for ld in lds]
    x = torch.stack([torch.from_numpy(ld.x[:, :batch].view(np.uint16)).view(torch.float16)
                     for ld in lds]).cuda()  # [layer][step][row][d]
    y = torch.zeros((steps, n_layers, batch, d), dtype=torch.float32, device="cuda")
    tiers = torch.empty((n_layers, batch, d_ff), dtype=torch.uint8, device="cuda")
    archive = torch.empty((steps, n_layers, layers[0].info.plan_bytes), dtype=torch.uint8,
                          device="cuda")
    sched = pipeline.StackSchedule(torch, layers, k, n16, n8, tiers, lag=lag, batch=batch)
    hooks = _Hooks(layers, archive, hold, poison, seed=n_layers * 10 + lag + batch)
    torch.cuda.synchronize()
    say(f"pipeline layers={n_layers} lag={lag} hold={hold} poison={poison} flags={flags} "
        f"batch={batch}: enqueue")
    for t in range(steps):
        sched.step(t, lambda l: x[l, t], lambda l: y[t, l], hooks=hooks)
    torch.cuda.synchronize()
    say("pipeline: compare with the oracle")
    yg = y.cpu().numpy()
    arch = archive.cpu()
    worst = 0.0
    for l, (L, ld) in enumerate(zip(layers, lds)):
        if pools:
            cache = oracle.TierPoolCache(d_ff, POOLS, {t: max(0, k - POOLS[t]) for t in (1, 2, 3)},
                                         policy)
        else:
            cache = oracle.LRUCache(d_ff, C, L.info.staging_slots, policy)
        tot = np.zeros(16, np.int64)
        for t in range(steps):
            tm = np.stack([oracle.select_tiers(oracle.predict(ld.pred_a, ld.pred_b, ld.bias,
                                                              ld.x[t, b])[1], k, n16, n8)[0]
                           for b in range(batch)])
            o = cache.plan(tm if batch > 1 else tm[0], t)
            tot += o["counts"]
            _check_plan(L, arch[t, l], o, f"layer {l} step {t}")
            y_ref = oracle_ffn(ld, ld.x[t], o["req_ids"], o["req_tier"],
                               o["req_mask"] if batch > 1 else None)
            for b in range(batch):
                err = r8_errors(yg[t, l, b], y_ref[b]).max()
                worst = max(worst, err)
                assert err <= FFN_TOL, f"layer {l} step {t} row {b}: FFN error {err:.3e}"
        if pools:
            for tr in (1, 2, 3):
                so, key, last = m2c.m2c_debug_read_pool_tables(L.handle, tr, d_ff, POOLS[tr])
                pc = cache.pools[tr]
                assert np.array_equal(so, pc.slot_of) and np.array_equal(key, pc.slot_key[:POOLS[tr]])
                assert np.array_equal(last, pc.slot_last[:POOLS[tr]])
        else:
            slot_of, key, stier, last = m2c.m2c_debug_read_tables(L.handle, d_ff, C)
            assert np.array_equal(slot_of, cache.slot_of) and np.array_equal(key, cache.slot_key[:C])
            assert np.array_equal(stier, cache.slot_tier[:C])
            assert np.array_equal(last, cache.slot_last[:C])
        st = L.stats()  # raises if a plan overflowed or an FFN gave up waiting
        assert (st.plans, st.req, st.hit, st.refill, st.new_, st.bypass) == (
            steps, tot[0], tot[1], tot[2], tot[3], tot[4])
        assert st.bypass > 0 and st.evict > 0
    say(f"pipeline worst FFN error {worst:.2e}")
    for L in layers:
        L.close()


def test_schedule_with_layers_read_from_dram_cache(tmp_path):
    """The SSD -> DRAM tier under the same schedule: four layers' stores
    written to a file, a pinned two-level DRAM cache with one fixed layer and
    two dynamic slots (look-ahead 1), so every token reloads layers while the
    GPU fills still read others; held streams and poisoned slots as above.
    Outputs and plans match the oracle, every fill read the right bytes (the
    FFN would be wrong otherwise), and the cache's load decisions are the
    preloader oracle's."""
    from oracle.preload import TwoLevelDram
    n_layers, d, d_ff, r, steps = 4, 512, 1400, 32, 8
    k = 350
    n16, n8 = k // 10, (k // 2) - k // 10
    C = 250
    desc = m2c.make_desc(d, d_ff, r, k, C)
    lds = [W.make_layer(950, l, d, d_ff, r, steps, rhos=(0.8,)) for l in range(n_layers)]
    path = str(tmp_path / "stores.bin")
    offs, off = [], 0
    owners = []
    for ld in lds:
        o = m2c.Layer(desc, ld)
        offs.append(off)
        off += m2c.m2c_layer_write_store(o.handle, path, off)
        owners.append(o)
    layer_bytes = sum(d_ff * owners[0].info.record_stride[t] for t in (1, 2, 3))
    for o in owners:
        o.close()
    dram = m2c.m2c_dram_create(m2c.DramDesc(n_layers, 1, 2, 1, layer_bytes, 0, 0), path, offs)
    layers = [m2c.Layer(desc, ld, dram=dram, dram_index=l) for l, ld in enumerate(lds)]
    # a record read through the cache is the oracle's record
    rec = m2c.m2c_debug_read_record(layers[2].handle, 1, 17, layers[2].info.record_stride[1])
    ref = oracle.build_records(lds[2].w_gate[17:18], lds[2].w_up[17:18],
                               np.ascontiguousarray(lds[2].w_down[:, 17:18]), 1)[0]
    assert np.array_equal(rec, ref)
    x = torch.stack([torch.from_numpy(ld.x[:, 0].view(np.uint16)).view(torch.float16)
                     for ld in lds]).cuda()
    y = torch.zeros((steps, n_layers, d), dtype=torch.float32, device="cuda")
    tiers = torch.empty((n_layers, d_ff), dtype=torch.uint8, device="cuda")
    archive = torch.empty((steps, n_layers, layers[0].info.plan_bytes), dtype=torch.uint8,
                          device="cuda")
    sched = pipeline.StackSchedule(torch, layers, k, n16, n8, tiers, lag=2)
    hooks = _Hooks(layers, archive, True, True, seed=77)
    say("pipeline from the DRAM cache: enqueue")
    for t in range(steps):
        sched.step(t, lambda l: x[l, t], lambda l: y[t, l], hooks=hooks)
    torch.cuda.synchronize()
    yg = y.cpu().numpy()
    arch = archive.cpu()
    for l, (L, ld) in enumerate(zip(layers, lds)):
        cache = oracle.LRUCache(d_ff, C, L.info.staging_slots)
        for t in range(steps):
            _, s = oracle.predict(ld.pred_a, ld.pred_b, ld.bias, ld.x[t, 0])
            tm, _ = oracle.select_tiers(s, k, n16, n8)
            o = cache.plan(tm, t)
            _check_plan(L, arch[t, l], o, f"layer {l} step {t}")
            y_ref = oracle_ffn(ld, ld.x[t], o["req_ids"], o["req_tier"])[0]
            err = r8_errors(yg[t, l], y_ref).max()
            assert err <= FFN_TOL, f"layer {l} step {t}: FFN error {err:.3e}"
        L.stats()
    ref = TwoLevelDram(n_layers, 1, 2, 1)
    ref.use(2)  # the record read above acquired layer 2 first
    for t in range(steps):
        for l in range(n_layers):
            ref.use(l)
    assert m2c.m2c_dram_get_log(dram) == [(m, old) for (_, m, _, old) in ref.log]
    st = m2c.m2c_dram_get_stats(dram)
    assert st.loads == len(ref.log) > n_layers  # layers were reloaded while fills ran
    for L in layers:
        L.close()
    m2c.m2c_dram_destroy(dram)
