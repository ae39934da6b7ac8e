"""CPU oracle of the M2Cache decode hot path (arXiv 2410.14740).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``, never by the product package. It is
a ctypes wrapper over ``oracle.c`` (plain C, loops, fp64 where floating point
is not fixed by the definition) and shares no code with the HIP library.

Functions and the passages of the paper they follow:
  build_records / dequant_record  Sec. 1 footnote, Sec. 5.2 (neurons stored at
                                  FP16 / INT8 / INT4; symmetric group-128
                                  quantization with fp16 scales)
  predict                         Sec. 1 "Active Neuron Identification"
                                  (low-rank predictor), Sec. 5.2
  select_tiers                    Sec. 5.2 (top-k active; higher score,
                                  higher precision)
  LRUCache.plan                   Sec. 5.3 (isolated per-layer cache unit),
                                  Sec. 1 / Sec. 6.4 (LRU neuron cache)
  sparse_ffn / dense_ffn          Sec. 1, Sec. 5.2 (FFN over active neurons)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

NCOUNTS = 16


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(
            ["gcc", "-O2", "-std=c99", "-Wall", "-ffp-contract=off", "-fno-fast-math",
             "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        I64 = ctypes.c_int64
        sig = {
            "orc_f16_to_f32_n": (None, [P, P, I64]),
            "orc_f32_to_f16_n": (None, [P, P, I64]),
            "orc_record_bytes": (I64, [I, I]),
            "orc_build_records": (I, [I, I, P, P, P, I, P, I64]),
            "orc_dequant_record": (I, [I, I, P, P, P, P]),
            "orc_predict": (I, [I, I, I, P, P, P, P, P, P]),
            "orc_select_tiers": (I, [I, P, I, I, I, P, P]),
            "orc_lru_plan": (I, [I, I, I, I, P, I, I] + [P] * 4 + [P] * 11),
            "orc_sparse_ffn": (I, [I, I, I, P, P, P, P, I64, P, I64, P, I64, P, P]),
            "orc_dense_ffn": (I, [I, I, P, P, P, P, P]),
            "orc_set_threads": (None, [I]),
            "orc_get_threads": (I, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def set_threads(n: int):
    """Threads the oracle's loops may use (1 = the serial program). Results
    do not depend on it: threads only split independent sums."""
    _load().orc_set_threads(int(n))


def get_threads() -> int:
    return int(_load().orc_get_threads())


def _p(a):
    return None if a is None else a.ctypes.data


def _h(a) -> np.ndarray:
    """fp16 array -> contiguous uint16 bit view."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    assert a.dtype == np.uint16
    return a


def f16_to_f32(bits) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(bits.shape, np.float32)
    _load().orc_f16_to_f32_n(_p(bits), _p(out), bits.size)
    return out


def f32_to_f16(vals) -> np.ndarray:
    vals = np.ascontiguousarray(vals, dtype=np.float32)
    out = np.empty(vals.shape, np.uint16)
    _load().orc_f32_to_f16_n(_p(vals), _p(out), vals.size)
    return out


def record_bytes(d: int, tier: int) -> int:
    return int(_load().orc_record_bytes(d, tier))


def record_stride(d: int, tier: int) -> int:
    return (record_bytes(d, tier) + 15) // 16 * 16


def build_records(w_gate, w_up, w_down, tier: int) -> np.ndarray:
    """All neuron records of one tier: uint8 [d_ff][record_stride]."""
    w_gate, w_up, w_down = _h(w_gate), _h(w_up), _h(w_down)
    d_ff, d = w_gate.shape
    assert w_up.shape == (d_ff, d) and w_down.shape == (d, d_ff)
    stride = record_stride(d, tier)
    out = np.zeros((d_ff, stride), np.uint8)
    rc = _load().orc_build_records(d, d_ff, _p(w_gate), _p(w_up), _p(w_down), tier, _p(out), stride)
    if rc != 0:
        raise ValueError("orc_build_records failed")
    return out


def dequant_record(rec, d: int, tier: int):
    """(gate, up, down) fp64 [d] each, the exact dequantized values."""
    rec = np.ascontiguousarray(rec, dtype=np.uint8)
    g, u, dn = (np.empty(d, np.float64) for _ in range(3))
    if _load().orc_dequant_record(d, tier, _p(rec), _p(g), _p(u), _p(dn)) != 0:
        raise ValueError("orc_dequant_record failed")
    return g, u, dn


def predict(A, B, bias, x):
    """(z fp32 [r], s fp32 [d_ff]) for one token x fp16 [d]."""
    A, B, x = _h(A), _h(B), _h(x)
    r, d = A.shape
    d_ff = B.shape[0]
    assert B.shape == (d_ff, r) and x.shape == (d,)
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.float32)
    z = np.empty(r, np.float32)
    s = np.empty(d_ff, np.float32)
    if _load().orc_predict(d, d_ff, r, _p(A), _p(B), _p(bias), _p(x), _p(z), _p(s)) != 0:
        raise ValueError("orc_predict failed")
    return z, s


def select_tiers(s, k: int, n16: int, n8: int):
    """(tier uint8 [d_ff], ranked ids int32 [k])."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    tier = np.empty(s.shape[0], np.uint8)
    ranked = np.empty(max(k, 1), np.int32)
    if _load().orc_select_tiers(s.shape[0], _p(s), k, n16, n8, _p(tier), _p(ranked)) != 0:
        raise ValueError("orc_select_tiers failed")
    return tier, ranked[:k]


POLICY_EXACT = 0      # a hit needs the resident tier to equal the requested one
POLICY_DOMINANCE = 1  # a resident tier at or above the requested one is a hit


class LRUCache:
    """Step-atomic LRU slot cache of one layer (C resident + S staging slots).
    policy: POLICY_EXACT or POLICY_DOMINANCE (how a resident neuron at
    another tier than the requested one is treated)."""

    def __init__(self, d_ff: int, C: int, S: int, policy: int = POLICY_EXACT):
        self.d_ff, self.C, self.S, self.policy = d_ff, C, S, policy
        self.slot_of = np.full(d_ff, -1, np.int32)
        self.slot_key = np.full(max(C, 1), -1, np.int32)
        self.slot_tier = np.zeros(max(C, 1), np.uint8)
        self.slot_last = np.full(max(C, 1), -1, np.int32)

    def plan(self, tier_map, step: int) -> dict:
        tm = np.ascontiguousarray(tier_map, dtype=np.uint8)
        if tm.ndim == 1:
            tm = tm[None, :]
        B, d_ff = tm.shape
        assert d_ff == self.d_ff
        n = d_ff
        counts = np.zeros(NCOUNTS, np.int32)
        out = dict(
            req_ids=np.zeros(n, np.int32), req_tier=np.zeros(n, np.uint8),
            req_hit=np.zeros(n, np.uint8), req_slot=np.zeros(n, np.int32),
            req_mask=np.zeros(n, np.uint32), fill_ids=np.zeros(n, np.int32),
            fill_tier=np.zeros(n, np.uint8), fill_slot=np.zeros(n, np.int32),
            fill_from=np.zeros(n, np.uint8), evicted_ids=np.zeros(n, np.int32),
        )
        rc = _load().orc_lru_plan(
            d_ff, self.C, self.S, B, _p(tm), int(step), int(self.policy),
            _p(self.slot_of), _p(self.slot_key), _p(self.slot_tier), _p(self.slot_last),
            _p(counts), _p(out["req_ids"]), _p(out["req_tier"]), _p(out["req_hit"]),
            _p(out["req_slot"]), _p(out["req_mask"]), _p(out["fill_ids"]), _p(out["fill_tier"]),
            _p(out["fill_slot"]), _p(out["fill_from"]), _p(out["evicted_ids"]),
        )
        if rc != 0:
            raise RuntimeError(f"orc_lru_plan failed ({rc})")
        nreq, nfill, nev = int(counts[0]), int(counts[6]), int(counts[5])
        res = {"counts": counts}
        for key in ("req_ids", "req_tier", "req_hit", "req_slot", "req_mask"):
            res[key] = out[key][:nreq].copy()
        for key in ("fill_ids", "fill_tier", "fill_slot", "fill_from"):
            res[key] = out[key][:nfill].copy()
        res["evicted_ids"] = out["evicted_ids"][:nev].copy()
        return res


def sparse_ffn(x, ids, tiers, records: dict, masks=None) -> np.ndarray:
    """y fp64 [B][d]: x fp16 [B][d]; records {tier: uint8 [d_ff][stride]}."""
    x = _h(x)
    if x.ndim == 1:
        x = x[None, :]
    B, d = x.shape
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    tiers = np.ascontiguousarray(tiers, dtype=np.uint8)
    if masks is not None:
        masks = np.ascontiguousarray(masks, dtype=np.uint32)
    y = np.empty((B, d), np.float64)
    r3, r2, r1 = records.get(3), records.get(2), records.get(1)
    st = lambda r: 0 if r is None else r.shape[1]
    rc = _load().orc_sparse_ffn(
        d, B, ids.size, _p(ids), _p(tiers), _p(masks),
        _p(r3), st(r3), _p(r2), st(r2), _p(r1), st(r1), _p(x), _p(y))
    if rc != 0:
        raise ValueError("orc_sparse_ffn failed")
    return y


def dense_ffn(w_gate, w_up, w_down, x) -> np.ndarray:
    w_gate, w_up, w_down, x = _h(w_gate), _h(w_up), _h(w_down), _h(x)
    d_ff, d = w_gate.shape
    y = np.empty(d, np.float64)
    if _load().orc_dense_ffn(d, d_ff, _p(w_gate), _p(w_up), _p(w_down), _p(x), _p(y)) != 0:
        raise ValueError("orc_dense_ffn failed")
    return y


class TierPoolCache:
    """Per-tier record arena: one step-atomic LRU slot cache per tier, each
    with slots of that tier's record size (Sec. 5.3's isolated cache unit,
    split by precision so that an INT4 neuron does not take an FP16-sized
    slot). A neuron required at step tier t (the highest tier any batch row
    asks for) is looked up in tier t's cache only: HIT if resident there,
    else NEW there (LRU victim, or BYPASS into that pool's staging slots).
    A neuron can be resident in several pools at once, each pool holding its
    own tier's record, so there are no REFILLs and the FFN output stays a
    function of the step's selection alone.

    C, S: {tier: resident slots}, {tier: staging slots}. Global slot ids are
    numbered in tier blocks, FP16 first: block t holds pool t's resident
    slots then its staging slots. The merged plan lists R in ascending id,
    the fills (every non-HIT) in ascending id, and the evictions of pool
    FP16, then INT8, then INT4, each in its victim order.

    policy POLICY_DOMINANCE (dominance hits across the pools): before the
    pools plan, a neuron required at tier t that is not resident in pool t
    but is resident in a pool of higher precision is served by the lowest
    such pool, as a HIT at that pool's tier (its record holds more bits of
    the same weights); residency is taken at the start of the step. Every
    other neuron stays with its own tier's pool."""

    TIERS = (3, 2, 1)

    def __init__(self, d_ff: int, C: dict, S: dict, policy: int = POLICY_EXACT):
        self.d_ff = d_ff
        self.policy = policy
        self.pools = {t: LRUCache(d_ff, C[t], S[t]) for t in self.TIERS}
        self.first, off = {}, 0
        for t in self.TIERS:
            self.first[t] = off
            off += C[t] + S[t]

    def resolve(self, step_tier) -> np.ndarray:
        """The pool tier each neuron is served from this step (0 = not
        required), as the dominance policy picks it; the step tier itself
        under POLICY_EXACT."""
        res = np.array(step_tier, dtype=np.uint8, copy=True)
        if self.policy != POLICY_DOMINANCE:
            return res
        for n in np.nonzero(res)[0]:
            t = int(res[n])
            if self.pools[t].slot_of[n] >= 0:
                continue
            for hi in range(t + 1, 4):
                if self.pools[hi].slot_of[n] >= 0:
                    res[n] = hi
                    break
        return res

    def plan(self, tier_map, step: int) -> dict:
        tm = np.ascontiguousarray(tier_map, dtype=np.uint8)
        if tm.ndim == 1:
            tm = tm[None, :]
        step_tier = self.resolve(tm.max(axis=0))
        parts = {}
        for t in self.TIERS:
            sub = np.where((tm > 0) & (step_tier == t)[None, :], t, 0).astype(np.uint8)
            p = self.pools[t].plan(sub, step)
            p["req_slot"] = p["req_slot"] + self.first[t]
            p["fill_slot"] = p["fill_slot"] + self.first[t]
            parts[t] = p
        res = {}
        order = np.argsort(np.concatenate([parts[t]["req_ids"] for t in self.TIERS]), kind="stable")
        for key in ("req_ids", "req_tier", "req_hit", "req_slot", "req_mask"):
            res[key] = np.concatenate([parts[t][key] for t in self.TIERS])[order]
        order = np.argsort(np.concatenate([parts[t]["fill_ids"] for t in self.TIERS]), kind="stable")
        for key in ("fill_ids", "fill_tier", "fill_slot", "fill_from"):
            res[key] = np.concatenate([parts[t][key] for t in self.TIERS])[order]
        res["evicted_ids"] = np.concatenate([parts[t]["evicted_ids"] for t in self.TIERS])
        res["counts"] = sum(parts[t]["counts"] for t in self.TIERS).astype(np.int32)
        return res
