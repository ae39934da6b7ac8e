"""Oracle of the offline neuron-ratio search (Sec. 5.2 "Offline Neuron Ratio
Search", Algorithm 1) on a synthetic proxy.

TEST INFRASTRUCTURE ONLY (tests/ use it; the library never does). It takes
the algorithm's steps in the paper's order and notation, on top of the CPU
oracle's predictor, top-k and fp64 sparse FFN (oracle/oracle.c):

  start with no high-precision neurons and r_low low-precision ones; each
  iteration adds s high-precision neurons and removes s * n low-precision
  ones, n = bits(high) / bits(low), so the memory the active neurons take
  stays the same; score each ratio with UQEst and keep the best (a later
  ratio wins ties, the paper's comparison is UQ_best >= UQ_score).

Readings where the paper cannot be followed literally (the library follows
the same ones):
  * UQEst is the entropy of a language model's next-token distributions on
    wikitext; there is no trained model here, so the proxy is the FFN's own
    output error against the full-precision FFN over calibration tokens:
    UQ = sum_t ||y_t - y*_t||^2 / sum_t ||y*_t||^2, where y_t is the sparse
    mixed-precision FFN of token t at the ratio and y*_t the dense FFN with
    every neuron at FP16 (both fp64 from the exact dequantized weights).
  * Ratios are neuron counts: n_high = i * s, n_low = n_low0 - i * s * n for
    iterations i = 1, 2, ...; the top (n_high + n_low) neurons by predictor
    score are active, the n_high best at FP16 and the rest at the low tier
    (INT4 for n = 4, INT8 for n = 2), the score-rank split of Sec. 5.2.
  * The loop as printed tests r_low >= 0 before it decrements, so its last
    ratio can have a negative low count; only ratios with n_low >= 0 are
    evaluated here.
"""
from __future__ import annotations

import numpy as np

import oracle


def candidates(n_low0: int, step: int, bit_ratio: int):
    """[(n_high, n_low)] in the order the search evaluates them."""
    out = []
    i = 1
    while n_low0 - i * step * bit_ratio >= 0:
        out.append((i * step, n_low0 - i * step * bit_ratio))
        i += 1
    return out


def uq_est(ld, records, xs, n_high: int, n_low: int, bit_ratio: int, y_dense) -> float:
    """The proxy UQEst of one ratio over the calibration tokens xs [T][d]."""
    num = den = 0.0
    k = n_high + n_low
    for t in range(xs.shape[0]):
        _, s = oracle.predict(ld.pred_a, ld.pred_b, ld.bias, xs[t])
        if bit_ratio == 4:
            tm, _ = oracle.select_tiers(s, k, n_high, 0)  # FP16 then INT4
        else:
            tm, _ = oracle.select_tiers(s, k, n_high, n_low)  # FP16 then INT8
        ids = np.nonzero(tm)[0].astype(np.int32)
        y = oracle.sparse_ffn(xs[t], ids, tm[ids], records)[0]
        num += float(np.sum((y - y_dense[t]) ** 2))
        den += float(np.sum(y_dense[t] ** 2))
    return num / den


def search(ld, xs, n_low0: int, step: int, bit_ratio: int):
    """Algorithm 1 on the proxy. Returns (candidates, uq per candidate, index
    of the chosen ratio)."""
    records = {t: oracle.build_records(ld.w_gate, ld.w_up, ld.w_down, t) for t in (1, 2, 3)}
    y_dense = np.stack([oracle.dense_ffn(ld.w_gate, ld.w_up, ld.w_down, xs[t])
                        for t in range(xs.shape[0])])
    cands = candidates(n_low0, step, bit_ratio)
    uq_best, best = float("inf"), -1
    uqs = []
    for i, (nh, nl) in enumerate(cands):
        uq = uq_est(ld, records, xs, nh, nl, bit_ratio, y_dense)
        uqs.append(uq)
        if uq_best >= uq:
            uq_best, best = uq, i
    return cands, uqs, best
