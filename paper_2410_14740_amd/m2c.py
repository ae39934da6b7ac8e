"""ctypes binding of libm2c.so (include/m2c.h). Marshalling only: every step
of the hot path runs in the library's HIP kernels.

Functions keep the C names. Device buffers may be passed as torch tensors
(their data_ptr() is used) or as raw integer addresses; streams as
torch.cuda.Stream, raw hipStream_t integers, or None for torch's current
stream. Host arrays for m2c_layer_create are numpy arrays. A non-OK status
raises M2CError with the library's message.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libm2c.so")

M2C_OK, M2C_ERR_INVALID_ARG, M2C_ERR_OUT_OF_MEMORY, M2C_ERR_HIP, M2C_ERR_CAPACITY, M2C_ERR_STATE = range(6)
STATUS_NAMES = ["OK", "INVALID_ARG", "OUT_OF_MEMORY", "HIP", "CAPACITY", "STATE"]
TIER_NONE, TIER_INT4, TIER_INT8, TIER_FP16 = range(4)

# plan count indices (m2c.h)
CNT_REQ, CNT_HIT, CNT_REFILL, CNT_NEW, CNT_BYPASS, CNT_EVICT, CNT_FILL = range(7)
CNT_REQ_FP16, CNT_REQ_INT8, CNT_REQ_INT4, CNT_FILL_FP16, CNT_FILL_INT8, CNT_FILL_INT4 = range(7, 13)
CNT_FILL_DERIVED = 13
NCOUNTS = 16


class M2CError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"m2c {name}: {msg}")


FLAG_DETERMINISTIC_FFN = 1
FLAG_DOMINANT_HITS = 2
FLAG_TIER_POOLS = 4


class LayerDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d_model", "d_ff", "pred_rank", "group", "k_max", "max_batch", "cache_slots",
        "staging_slots", "device", "flags")] + [("tier_slots", ctypes.c_int32 * 4)]


class LayerInfo(ctypes.Structure):
    _fields_ = [
        ("record_bytes", ctypes.c_int32 * 4), ("record_stride", ctypes.c_int32 * 4),
        ("slot_bytes", ctypes.c_int32), ("cache_slots", ctypes.c_int32),
        ("staging_slots", ctypes.c_int32), ("plan_capacity", ctypes.c_int32),
        ("plan_bytes", ctypes.c_int64), ("host_store_bytes", ctypes.c_int64),
        ("device_bytes", ctypes.c_int64), ("pool_first", ctypes.c_int32 * 4),
        ("pool_slots", ctypes.c_int32 * 4), ("pool_resident", ctypes.c_int32 * 4),
        ("pool_stride", ctypes.c_int32 * 4), ("slot_arena_bytes", ctypes.c_int64)]


PLAN_FIELDS = ("counts", "req_ids", "req_tier", "req_hit", "req_slot", "req_mask", "fill_ids",
               "fill_tier", "fill_slot", "fill_from", "evicted_ids", "work_slot", "work_mask",
               "ffn_tasks", "total_bytes")


class PlanLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in PLAN_FIELDS]


DRAM_HOST_MEMORY = 1
DRAM_DIRECT_IO = 2


class DramDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("fixed_layers", ctypes.c_int32),
                ("dynamic_slots", ctypes.c_int32), ("lookahead", ctypes.c_int32),
                ("layer_bytes", ctypes.c_int64), ("flags", ctypes.c_int32),
                ("device", ctypes.c_int32)]


class DramStats(ctypes.Structure):
    _fields_ = [("acquires", ctypes.c_int64), ("hits", ctypes.c_int64), ("loads", ctypes.c_int64),
                ("evictions", ctypes.c_int64), ("bytes_read", ctypes.c_int64),
                ("fixed_bytes", ctypes.c_int64), ("read_seconds", ctypes.c_double),
                ("wait_seconds", ctypes.c_double), ("direct_io", ctypes.c_int32)]


class Stats(ctypes.Structure):
    _fields_ = [("plans", ctypes.c_int64), ("req", ctypes.c_int64), ("hit", ctypes.c_int64),
                ("refill", ctypes.c_int64), ("new_", ctypes.c_int64), ("bypass", ctypes.c_int64),
                ("evict", ctypes.c_int64), ("fill", ctypes.c_int64 * 4),
                ("fill_bytes", ctypes.c_int64), ("derived", ctypes.c_int64 * 4),
                ("host_bytes", ctypes.c_int64), ("req_tier", ctypes.c_int64 * 4),
                ("req_bytes", ctypes.c_int64)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libm2c.so. There is no fallback: a missing library, or one built
    from other sources than the ones in the tree, is an error."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2410_14740_amd.build`")
    # torch wheels bundle their own HIP runtime; load it first so that the
    # library binds to the same runtime instance as the device memory and
    # streams torch hands it (two runtimes in one process do not share them)
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P, I32, I64, S = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "m2c_record_bytes": (I64, [I32, I32]),
        "m2c_layer_create": (I32, [ctypes.POINTER(LayerDesc), P, P, P, P, P, P, ctypes.POINTER(P)]),
        "m2c_layer_create_shared": (I32, [ctypes.POINTER(LayerDesc), P, P, P, P, ctypes.POINTER(P)]),
        "m2c_layer_destroy": (I32, [P]),
        "m2c_layer_get_info": (I32, [P, ctypes.POINTER(LayerInfo)]),
        "m2c_plan_get_layout": (I32, [P, ctypes.POINTER(PlanLayout)]),
        "m2c_predict_rank": (I32, [P, P, I32, I32, I32, I32, P, P, P]),
        "m2c_predict_rank_noalloc": (I32, [P, P, I32, I32, I32, I32, P, P, P]),
        "m2c_cache_plan": (I32, [P, P, I32, I64, P, P]),
        "m2c_cache_fill": (I32, [P, P, P]),
        "m2c_sparse_ffn": (I32, [P, P, I32, P, P, P]),
        "m2c_layer_reset_cache": (I32, [P, P]),
        "m2c_layer_stats": (I32, [P, ctypes.POINTER(Stats)]),
        "m2c_debug_read_record": (I32, [P, I32, I32, P, S]),
        "m2c_debug_read_slot": (I32, [P, I32, P, S]),
        "m2c_debug_read_tables": (I32, [P, P, P, P, P]),
        "m2c_debug_read_pool_tables": (I32, [P, I32, P, P, P]),
        "m2c_debug_poison_fill_slots": (I32, [P, P, P]),
        "m2c_debug_ffn_withhold_h": (I32, [P, I32]),
        "m2c_layer_write_store": (I32, [P, ctypes.c_char_p, I64, ctypes.POINTER(I64)]),
        "m2c_dram_create": (I32, [ctypes.POINTER(DramDesc), ctypes.c_char_p, P, ctypes.POINTER(P)]),
        "m2c_dram_destroy": (I32, [P]),
        "m2c_dram_acquire": (I32, [P, I32, ctypes.POINTER(P)]),
        "m2c_dram_release": (I32, [P, I32]),
        "m2c_dram_get_stats": (I32, [P, ctypes.POINTER(DramStats)]),
        "m2c_dram_get_log": (I32, [P, P, P, I32, ctypes.POINTER(I32)]),
        "m2c_layer_create_from_dram": (I32, [ctypes.POINTER(LayerDesc), P, I32, P, P, P,
                                             ctypes.POINTER(P)]),
        "m2c_ratio_search": (I32, [P, P, I32, I32, I32, I32, I32, P, P, P,
                                   ctypes.POINTER(I32), ctypes.POINTER(I32), P]),
        "m2c_last_error": (ctypes.c_char_p, []),
        "m2c_build_id": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    from . import build as _build
    want, got = _build.source_id(), lib.m2c_build_id().decode()
    if got != want:
        raise ImportError(f"{path} was built from other sources (build id {got}, sources {want}); "
                          "run `python -m paper_2410_14740_amd.build`")
    _lib = lib
    return lib


def is_current(path: str = LIB_PATH) -> bool:
    """True when the library exists and was built from the sources in the tree
    (checked without loading it: the build id string is in the file)."""
    if not os.path.exists(path):
        return False
    from . import build as _build
    with open(path, "rb") as f:
        return _build.source_id().encode() in f.read()


def _check(status: int):
    if status != M2C_OK:
        raise M2CError(status, load().m2c_last_error().decode())


def _ptr(a):
    if a is None:
        return None
    if isinstance(a, int):
        return a
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    raise TypeError(f"cannot pass {type(a)} as a pointer")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _host16(a):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError("fp16 host arrays expected")
    return a


def m2c_record_bytes(d_model: int, tier: int) -> int:
    return int(load().m2c_record_bytes(d_model, tier))


def m2c_layer_create(desc: LayerDesc, w_gate, w_up, w_down, pred_a, pred_b, score_bias=None):
    w_gate, w_up, w_down, pred_a, pred_b = map(_host16, (w_gate, w_up, w_down, pred_a, pred_b))
    if score_bias is not None:
        score_bias = np.ascontiguousarray(score_bias, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(load().m2c_layer_create(ctypes.byref(desc), _ptr(w_gate), _ptr(w_up), _ptr(w_down),
                                   _ptr(pred_a), _ptr(pred_b), _ptr(score_bias), ctypes.byref(out)))
    return out.value


def m2c_layer_create_shared(desc: LayerDesc, weights_of: int, pred_a, pred_b, score_bias=None):
    pred_a, pred_b = _host16(pred_a), _host16(pred_b)
    if score_bias is not None:
        score_bias = np.ascontiguousarray(score_bias, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(load().m2c_layer_create_shared(ctypes.byref(desc), weights_of, _ptr(pred_a),
                                          _ptr(pred_b), _ptr(score_bias), ctypes.byref(out)))
    return out.value


def m2c_layer_destroy(layer: int):
    _check(load().m2c_layer_destroy(layer))


def m2c_layer_get_info(layer: int) -> LayerInfo:
    info = LayerInfo()
    _check(load().m2c_layer_get_info(layer, ctypes.byref(info)))
    return info


def m2c_plan_get_layout(layer: int) -> PlanLayout:
    lay = PlanLayout()
    _check(load().m2c_plan_get_layout(layer, ctypes.byref(lay)))
    return lay


def m2c_predict_rank(layer, x, batch, k, n_fp16, n_int8, scores, tier_map, stream=None):
    _check(load().m2c_predict_rank(layer, _ptr(x), batch, k, n_fp16, n_int8, _ptr(scores),
                                   _ptr(tier_map), _stream(stream)))


def m2c_predict_rank_noalloc(layer, x, batch, k, n_fp16, n_int8, scores, tier_map, stream=None):
    _check(load().m2c_predict_rank_noalloc(layer, _ptr(x), batch, k, n_fp16, n_int8, _ptr(scores),
                                           _ptr(tier_map), _stream(stream)))


def m2c_cache_plan(layer, tier_map, batch, step, plan, stream=None):
    _check(load().m2c_cache_plan(layer, _ptr(tier_map), batch, step, _ptr(plan), _stream(stream)))


def m2c_cache_fill(layer, plan, stream=None):
    _check(load().m2c_cache_fill(layer, _ptr(plan), _stream(stream)))


def m2c_sparse_ffn(layer, x, batch, plan, y, stream=None):
    _check(load().m2c_sparse_ffn(layer, _ptr(x), batch, _ptr(plan), _ptr(y), _stream(stream)))


def m2c_layer_reset_cache(layer, stream=None):
    _check(load().m2c_layer_reset_cache(layer, _stream(stream)))


def m2c_layer_stats(layer) -> Stats:
    st = Stats()
    _check(load().m2c_layer_stats(layer, ctypes.byref(st)))
    return st


def m2c_debug_read_record(layer, tier: int, neuron: int, nbytes: int) -> np.ndarray:
    out = np.empty(nbytes, np.uint8)
    _check(load().m2c_debug_read_record(layer, tier, neuron, out.ctypes.data, nbytes))
    return out


def m2c_debug_read_slot(layer, slot: int, nbytes: int) -> np.ndarray:
    out = np.empty(nbytes, np.uint8)
    _check(load().m2c_debug_read_slot(layer, slot, out.ctypes.data, nbytes))
    return out


def m2c_debug_read_tables(layer, d_ff: int, C: int):
    slot_of = np.empty(d_ff, np.int32)
    key = np.empty(max(C, 1), np.int32)
    tier = np.empty(max(C, 1), np.uint8)
    last = np.empty(max(C, 1), np.int32)
    _check(load().m2c_debug_read_tables(layer, slot_of.ctypes.data, key.ctypes.data,
                                        tier.ctypes.data, last.ctypes.data))
    return slot_of, key[:C], tier[:C], last[:C]


def m2c_debug_poison_fill_slots(layer, plan, stream=None):
    _check(load().m2c_debug_poison_fill_slots(layer, _ptr(plan), _stream(stream)))


def m2c_debug_ffn_withhold_h(layer, polls: int):
    _check(load().m2c_debug_ffn_withhold_h(layer, polls))


def m2c_build_id() -> str:
    return load().m2c_build_id().decode()


def m2c_layer_write_store(layer, path: str, offset: int) -> int:
    n = ctypes.c_int64()
    _check(load().m2c_layer_write_store(layer, path.encode(), offset, ctypes.byref(n)))
    return n.value


def m2c_dram_create(desc: DramDesc, path: str, offsets):
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    out = ctypes.c_void_p()
    _check(load().m2c_dram_create(ctypes.byref(desc), path.encode(), offs.ctypes.data,
                                  ctypes.byref(out)))
    return out.value


def m2c_dram_destroy(dram):
    _check(load().m2c_dram_destroy(dram))


def m2c_dram_acquire(dram, layer: int, nbytes: int) -> np.ndarray:
    """Hold `layer` and return a copy of its first `nbytes` bytes."""
    p = ctypes.c_void_p()
    _check(load().m2c_dram_acquire(dram, layer, ctypes.byref(p)))
    return np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(p.value)).copy()


def m2c_dram_release(dram, layer: int):
    _check(load().m2c_dram_release(dram, layer))


def m2c_dram_get_stats(dram) -> DramStats:
    st = DramStats()
    _check(load().m2c_dram_get_stats(dram, ctypes.byref(st)))
    return st


def m2c_dram_get_log(dram):
    """[(loaded layer, evicted layer or -1)] in decision order."""
    n = ctypes.c_int32()
    _check(load().m2c_dram_get_log(dram, None, None, 0, ctypes.byref(n)))
    a = np.empty(max(n.value, 1), np.int32)
    b = np.empty(max(n.value, 1), np.int32)
    _check(load().m2c_dram_get_log(dram, a.ctypes.data, b.ctypes.data, n.value, ctypes.byref(n)))
    return list(zip(a[:n.value].tolist(), b[:n.value].tolist()))


def m2c_layer_create_from_dram(desc: LayerDesc, dram, index: int, pred_a, pred_b, score_bias=None):
    pred_a, pred_b = _host16(pred_a), _host16(pred_b)
    if score_bias is not None:
        score_bias = np.ascontiguousarray(score_bias, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(load().m2c_layer_create_from_dram(ctypes.byref(desc), dram, index, _ptr(pred_a),
                                             _ptr(pred_b), _ptr(score_bias), ctypes.byref(out)))
    return out.value


def m2c_ratio_search(layer, x, T: int, n_low0: int, step: int, bit_ratio: int, stream=None):
    """Algorithm 1 on the FFN-error proxy: ([(n_high, n_low)], [uq], best index)."""
    cap = max(1, n_low0 // max(1, step * bit_ratio) + 1)
    nh = np.empty(cap, np.int32)
    nl = np.empty(cap, np.int32)
    uq = np.empty(cap, np.float64)
    cnt, best = ctypes.c_int32(), ctypes.c_int32()
    _check(load().m2c_ratio_search(layer, _ptr(x), T, n_low0, step, bit_ratio, cap, nh.ctypes.data,
                                   nl.ctypes.data, uq.ctypes.data, ctypes.byref(cnt),
                                   ctypes.byref(best), _stream(stream)))
    n = cnt.value
    return list(zip(nh[:n].tolist(), nl[:n].tolist())), uq[:n].tolist(), best.value


def m2c_debug_read_pool_tables(layer, tier: int, d_ff: int, C: int):
    """(slot_of [d_ff], slot_key [C], slot_last [C]) of tier `tier`'s pool."""
    slot_of = np.empty(d_ff, np.int32)
    key = np.empty(max(C, 1), np.int32)
    last = np.empty(max(C, 1), np.int32)
    _check(load().m2c_debug_read_pool_tables(layer, tier, slot_of.ctypes.data, key.ctypes.data,
                                             last.ctypes.data))
    return slot_of, key[:C], last[:C]


def m2c_last_error() -> str:
    return load().m2c_last_error().decode()


# ---------------------------------------------------------------------------
# Convenience: one layer with its own plan buffer (torch device memory).

class Layer:
    """Owns a layer handle and one plan buffer; methods map 1:1 onto the ABI."""

    def __init__(self, desc: LayerDesc, data=None, weights_of: "Layer | None" = None,
                 dram=None, dram_index: int = -1):
        import torch
        self.desc = desc
        if dram is not None:
            self.handle = m2c_layer_create_from_dram(desc, dram, dram_index, data.pred_a,
                                                     data.pred_b, data.bias)
        elif weights_of is None:
            self.handle = m2c_layer_create(desc, data.w_gate, data.w_up, data.w_down, data.pred_a,
                                           data.pred_b, data.bias)
        else:
            self.handle = m2c_layer_create_shared(desc, weights_of.handle, data.pred_a,
                                                  data.pred_b, data.bias)
        self.info = m2c_layer_get_info(self.handle)
        self.layout = m2c_plan_get_layout(self.handle)
        dev = torch.device("cuda", desc.device)
        # plan buffers must be 256-byte aligned: over-allocate and offset
        self._plan_raw = torch.empty(self.info.plan_bytes + 256, dtype=torch.uint8, device=dev)
        off = (-self._plan_raw.data_ptr()) % 256
        self.plan = self._plan_raw[off:off + self.info.plan_bytes]

    def predict_rank(self, x, batch, k, n16, n8, scores, tier_map, stream=None):
        m2c_predict_rank(self.handle, x, batch, k, n16, n8, scores, tier_map, stream)

    def cache_plan(self, tier_map, batch, step, stream=None, plan=None):
        m2c_cache_plan(self.handle, tier_map, batch, step, self.plan if plan is None else plan, stream)

    def cache_fill(self, stream=None, plan=None):
        m2c_cache_fill(self.handle, self.plan if plan is None else plan, stream)

    def sparse_ffn(self, x, batch, y, stream=None, plan=None):
        """y += FFN(x) (zero y first for the plain output)."""
        m2c_sparse_ffn(self.handle, x, batch, self.plan if plan is None else plan, y, stream)

    def reset_cache(self, stream=None):
        m2c_layer_reset_cache(self.handle, stream)

    def stats(self) -> Stats:
        return m2c_layer_stats(self.handle)

    def read_plan(self, plan=None) -> dict:
        """Copy a plan to the host as numpy arrays trimmed to their counts."""
        raw = (self.plan if plan is None else plan).cpu().numpy()
        lay = self.layout
        cap = self.info.plan_capacity

        def arr(field, dtype, n):
            off = getattr(lay, field)
            return raw[off:off + n * np.dtype(dtype).itemsize].view(dtype).copy()

        counts = arr("counts", np.int32, NCOUNTS)
        nreq, nfill, nev = int(counts[CNT_REQ]), int(counts[CNT_FILL]), int(counts[CNT_EVICT])
        res = {"counts": counts}
        for f, dt in (("req_ids", np.int32), ("req_tier", np.uint8), ("req_hit", np.uint8),
                      ("req_slot", np.int32), ("req_mask", np.uint32), ("work_slot", np.int32),
                      ("work_mask", np.uint32)):
            res[f] = arr(f, dt, min(nreq, cap))
        for f, dt in (("fill_ids", np.int32), ("fill_tier", np.uint8), ("fill_slot", np.int32),
                      ("fill_from", np.uint8)):
            res[f] = arr(f, dt, min(nfill, cap))
        res["evicted_ids"] = arr("evicted_ids", np.int32, min(nev, cap))
        return res

    def close(self):
        if self.handle:
            m2c_layer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def make_desc(d_model, d_ff, pred_rank, k_max, cache_slots, max_batch=1, staging_slots=-1,
              device=0, flags=0, tier_slots=None) -> LayerDesc:
    """tier_slots: {tier: resident slots} of the per-tier arena; sets
    FLAG_TIER_POOLS and cache_slots to their sum."""
    ts = (ctypes.c_int32 * 4)(0, 0, 0, 0)
    if tier_slots is not None:
        for t in (1, 2, 3):
            ts[t] = tier_slots[t]
        cache_slots = sum(tier_slots[t] for t in (1, 2, 3))
        flags |= FLAG_TIER_POOLS
    return LayerDesc(d_model, d_ff, pred_rank, 128, k_max, max_batch, cache_slots, staging_slots,
                     device, flags, ts)


def pool_slots_for_budget(d_model: int, counts, budget_bytes: int) -> dict:
    """Resident slots per tier for a per-tier arena of at most `budget_bytes`
    of records: every pool gets the same multiple of its tier's per-step
    demand (counts = {tier: neurons per step}), rounded down."""
    stride = {t: (m2c_record_bytes(d_model, t) + 15) // 16 * 16 for t in (1, 2, 3)}
    demand = sum(counts[t] * stride[t] for t in (1, 2, 3))
    return {t: int(counts[t] * budget_bytes // demand) for t in (1, 2, 3)}
