"""Shared helpers of the GPU parity tests (oracle side and comparisons)."""
import sys

import numpy as np

import oracle


def say(msg: str):
    """Progress line that names the case, flushed before a GPU step."""
    print(f"[m2c-test] {msg}", file=sys.stderr, flush=True)


def r8_errors(y, y_ref):
    """|y - y*| / max(|y*|, 1e-2 * rms(y*)) per element (the FFN tolerance
    reading: relative error, floored at 1% of the output's rms)."""
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    rms = np.sqrt(np.mean(y_ref * y_ref)) if y_ref.size else 0.0
    den = np.maximum(np.abs(y_ref), 1e-2 * rms)
    den = np.where(den > 0, den, 1.0)
    return np.abs(y - y_ref) / den


FFN_TOL = 2e-3


def work_order(plan):
    """The library's FFN work list of a plan, from the oracle's required
    list: slots and row masks tier-major (FP16, INT8, INT4), ascending id
    inside a tier (the layout the plan's work_slot / work_mask document)."""
    order = [p for t in (3, 2, 1) for p in range(len(plan["req_ids"])) if plan["req_tier"][p] == t]
    return (np.asarray([plan["req_slot"][p] for p in order], np.int32),
            np.asarray([plan["req_mask"][p] for p in order], np.uint32))


def derived_fills(plan):
    """Fills to INT8 / INT4 of a neuron whose slot held its FP16 record
    (fill_from == 3): the library makes them on the GPU from that record."""
    return int(np.count_nonzero((plan["fill_from"] == 3) & (plan["fill_tier"] < 3)))


def subset_records(ld, ids):
    """Oracle records (all three tiers) for the neurons `ids` only, indexed by
    position in `ids`; returns ({tier: records}, {neuron id: row})."""
    ids = np.asarray(ids, np.int64)
    wg = np.ascontiguousarray(ld.w_gate[ids])
    wu = np.ascontiguousarray(ld.w_up[ids])
    wd = np.ascontiguousarray(ld.w_down[:, ids])
    recs = {t: oracle.build_records(wg, wu, wd, t) for t in (1, 2, 3)}
    return recs, {int(i): r for r, i in enumerate(ids)}


def oracle_ffn(ld, x, req_ids, req_tier, req_mask=None, recs=None):
    """Oracle FFN over the listed neurons; builds records on demand."""
    if recs is None:
        recs, row = subset_records(ld, req_ids)
        ids = np.array([row[int(i)] for i in req_ids], np.int32)
    else:
        ids = np.asarray(req_ids, np.int32)
    return oracle.sparse_ffn(x, ids, req_tier, recs, req_mask)
