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
