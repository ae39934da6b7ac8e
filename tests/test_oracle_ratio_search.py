"""Pins of the neuron-ratio search oracle (oracle/ratio_search.py): the
candidate ratios keep the active neurons' bytes fixed, the proxy score
equals an independent numpy evaluation (numpy decode of the records, numpy
SwiGLU, numpy dense FFN), and the chosen ratio is the last minimum."""
import numpy as np
import pytest

from oracle import ratio_search as RS
from paper_2410_14740_amd import workloads as W


@pytest.mark.parametrize("n_low0,step,n", [(688, 16, 4), (688, 32, 2), (100, 7, 4), (8, 8, 2)])
def test_candidates_keep_the_budget(n_low0, step, n):
    c = RS.candidates(n_low0, step, n)
    bits_low = 16 // n
    for i, (nh, nl) in enumerate(c, start=1):
        assert nh == i * step and nl >= 0
        assert nh * 16 + nl * bits_low == n_low0 * bits_low  # same bytes of codes
    # the next ratio would need a negative low count
    assert n_low0 - (len(c) + 1) * step * n < 0


def _numpy_ffn(ld, x, ids, tiers):
    """Independent evaluation: quantize with numpy from the definition, then
    the SwiGLU sum in fp64."""
    def quant(v, qmax):
        g = v.reshape(-1, 128).astype(np.float32)
        s = (np.abs(g).max(axis=1) / np.float32(qmax)).astype(np.float16).astype(np.float32)
        q = np.where(s[:, None] > 0, np.clip(np.rint(g / np.where(s > 0, s, 1)[:, None]), -qmax, qmax), 0)
        return (q * s[:, None]).reshape(-1).astype(np.float64)
    xd = x.astype(np.float64)
    y = np.zeros(ld.d_model)
    for i, t in zip(ids, tiers):
        vs = [ld.w_gate[i], ld.w_up[i], ld.w_down[:, i]]
        if t == 3:
            g, u, dn = (v.astype(np.float64) for v in vs)
        else:
            g, u, dn = (quant(v, 127 if t == 2 else 7) for v in vs)
        a, b = g @ xd, u @ xd
        y += a / (1 + np.exp(-a)) * b * dn
    return y


def test_uq_matches_numpy():
    import oracle
    ld = W.make_layer(401, 0, 256, 300, 16, 3)
    recs = {t: oracle.build_records(ld.w_gate, ld.w_up, ld.w_down, t) for t in (1, 2, 3)}
    xs = ld.x[:, 0]
    yd = np.stack([ld.w_down.astype(np.float64) @ (
        (lambda a, b: a / (1 + np.exp(-a)) * b)(ld.w_gate.astype(np.float64) @ xs[t].astype(np.float64),
                                                ld.w_up.astype(np.float64) @ xs[t].astype(np.float64)))
        for t in range(3)])
    for nh, nl, n in ((10, 60, 4), (20, 40, 2)):
        got = RS.uq_est(ld, recs, xs, nh, nl, n, yd)
        num = den = 0.0
        for t in range(3):
            _, s = oracle.predict(ld.pred_a, ld.pred_b, ld.bias, xs[t])
            order = np.lexsort((np.arange(300), -s.astype(np.float64)))[:nh + nl]
            tiers = np.where(np.arange(nh + nl) < nh, 3, 1 if n == 4 else 2)
            y = _numpy_ffn(ld, xs[t], order, tiers)
            num += np.sum((y - yd[t]) ** 2)
            den += np.sum(yd[t] ** 2)
        assert abs(got - num / den) <= 1e-9 * (num / den)


def test_search_keeps_the_last_minimum():
    ld = W.make_layer(402, 0, 256, 400, 16, 2)
    cands, uqs, best = RS.search(ld, ld.x[:, 0], 200, 8, 4)
    assert len(cands) == len(uqs) == 6
    m = min(uqs)
    assert best == max(i for i, u in enumerate(uqs) if u == m)
