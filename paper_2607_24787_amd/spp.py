"""ctypes binding of libspp.so (the C ABI declared in include/spp.h).

Argument marshalling only: every step of the hot path runs in the HIP library.
Pointers are passed as Python ints (device or pinned-host addresses); numpy
arrays carry small host inputs and outputs.  The library must have been built
(``python -m paper_2607_24787_amd.build``); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p

import numpy as np

# SPP_LIB_PATH selects another build of the same library (a sanitized host runtime)
LIB_PATH = os.environ.get("SPP_LIB_PATH") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspp.so")

SPP_OK, SPP_EINVAL, SPP_ENOMEM, SPP_EHIP, SPP_ESTATE = 0, -1, -2, -3, -4
DTYPE_F32, DTYPE_BF16 = 0, 1
LAYOUT_UNITS, LAYOUT_TILED, LAYOUT_Q4_UNITS = 0, 1, 2
CODEC_PLAIN, CODEC_Q4 = 0, 1
PREFETCH_ADAPTER, PREFETCH_PREV_TOKEN = 0, 1
COPY_KERNEL, COPY_SDMA, COPY_SPLIT = 0, 1, 2


class SppError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"spp status {status}: {msg}")
        self.status = status


class ModelDesc(ctypes.Structure):
    _fields_ = [(f, c_int32) for f in ("L", "D", "n", "K", "I", "r", "n_shared", "S", "max_batch", "dtype",
                                       "has_proj")] + [("rms_eps", c_float), ("expert_codec", c_int32)]


class LayerStats(ctypes.Structure):
    _fields_ = ([(f, c_int32) for f in ("hits", "misses", "prefetched", "prefetch_used", "ready_on_time",
                                        "token_hits", "waited")]
                + [("exposed_us", c_float), ("layer_us", c_float)])


class RunStats(ctypes.Structure):
    _fields_ = ([(f, c_int64) for f in ("layer_calls", "hits", "misses", "prefetched", "prefetch_used",
                                         "ready_on_time", "copies", "copy_bytes", "ffn_launches",
                                         "window_samples")]
                + [(f, c_double) for f in ("router_us", "exposed_us", "ffn_us", "tail_us", "span_us",
                                           "window_us", "compute_window_us", "exposed_load_us",
                                           "exposed_wait_us")]
                + [("recall_tokens", c_int64), ("recall_hits", c_int64 * 3), ("pred_events", c_int64),
                   ("demand_exceeds", c_int64 * 3), ("demand_hist", (c_int64 * 17) * 3),
                   ("ffn_split_launches", c_int64), ("exposed_shared_us", c_double), ("shared_calls", c_int64),
                   ("waited", c_int64), ("prefetch_hist", c_int64 * 17),
                   ("host_route_us", c_double), ("host_decide_us", c_double)])

    def as_dict(self):
        out = {}
        for f, _ in self._fields_:
            v = getattr(self, f)
            out[f] = ([list(r) if isinstance(r, ctypes.Array) else r for r in v] if isinstance(v, ctypes.Array)
                      else v)
        return out


_SIGS = {
    "spp_blob_stride": (c_size_t, [POINTER(ModelDesc)]),
    "spp_blob_layout": (c_int32, [POINTER(ModelDesc)]),
    "spp_pack_expert": (c_int32, [POINTER(ModelDesc), c_void_p, c_void_p, c_void_p, c_void_p]),
    "spp_pack_expert_q4": (c_int32, [POINTER(ModelDesc), c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p]),
    "spp_create": (c_int32, [POINTER(ModelDesc), c_void_p, POINTER(c_void_p)]),
    "spp_destroy": (c_int32, [c_void_p]),
    "spp_bind_layer": (c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "spp_set_resident": (c_int32, [c_void_p, c_int32, POINTER(c_int32), c_int32]),
    "adapter_predict": (c_int32, [c_void_p, c_int32, c_void_p, c_int32, POINTER(c_float)]),
    "select_prefetch_budget": (c_int32, [c_double, c_double, c_int32, POINTER(c_int32)]),
    "expert_cache_issue_prefetch": (c_int32, [c_void_p, c_int32, POINTER(c_float), c_int32, POINTER(c_int32),
                                              POINTER(c_int32)]),
    "spp_decode_step": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_int32, POINTER(c_int32),
                                  POINTER(c_float), c_void_p]),
    "moe_layer_forward": (c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_int32, c_int32, POINTER(c_int32),
                                    POINTER(c_float), POINTER(LayerStats)]),
    "spp_last_error": (c_char_p, []),
    "adapter_predict_static": (c_int32, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_void_p, c_int32,
                                         c_void_p, c_void_p]),
    "spp_get_slot_table": (c_int32, [c_void_p, c_int32, POINTER(c_int32), POINTER(c_int64)]),
    "spp_set_slot_table": (c_int32, [c_void_p, c_int32, POINTER(c_int32), POINTER(c_int64)]),
    "spp_get_clock": (c_int32, [c_void_p, POINTER(c_int64)]),
    "spp_set_clock": (c_int32, [c_void_p, c_int64]),
    "spp_get_last_transfers": (c_int32, [c_void_p, POINTER(c_int32), POINTER(c_int32), POINTER(c_int32),
                                         POINTER(c_int32), c_int32]),
    "spp_get_last_priorities": (c_int32, [c_void_p, POINTER(c_float)]),
    "spp_get_last_router_input": (c_int32, [c_void_p, POINTER(c_float), c_int32]),
    "spp_set_timing": (c_int32, [c_void_p, c_int32]),
    "spp_get_run_stats": (c_int32, [c_void_p, POINTER(RunStats)]),
    "spp_reset_run_stats": (c_int32, [c_void_p]),
    "spp_get_layer_times": (c_int32, [c_void_p, c_int32, POINTER(c_int64), POINTER(c_double), POINTER(c_double),
                                      POINTER(c_int64)]),
    "spp_profile_expert_copy": (c_int32, [c_void_p, c_int32, c_int32, POINTER(c_double)]),
    "spp_probe_read_ceiling": (c_int32, [c_void_p, c_int32, POINTER(c_double), POINTER(c_double)]),
    "spp_probe_stream_read": (c_int32, [c_void_p, c_int32, POINTER(c_double), POINTER(c_double)]),
    "spp_set_prefetch_source": (c_int32, [c_void_p, c_int32]),
    "spp_set_copy_engine": (c_int32, [c_void_p, c_int32]),
    "spp_set_tier_delay": (c_int32, [c_void_p, c_int32]),
    "spp_get_last_logits": (c_int32, [c_void_p, POINTER(c_float), c_int32]),
    "spp_set_ffn_workgroups": (c_int32, [c_void_p, c_int32]),
    "spp_set_ffn_overlap": (c_int32, [c_void_p, c_int32]),
    "spp_set_prefetch_parallel": (c_int32, [c_void_p, c_int32]),
    "spp_debug_set_poison": (c_int32, [c_void_p, c_int32]),
    "spp_debug_set_copy_delay": (c_int32, [c_void_p, c_int32]),
    "spp_policy_create": (c_int32, [c_int32, c_int32, POINTER(c_int32), c_int32, POINTER(c_void_p)]),
    "spp_policy_destroy": (c_int32, [c_void_p]),
    "spp_policy_on_demand": (c_int32, [c_void_p, POINTER(c_int32), c_int32, c_int64, POINTER(c_int32),
                                       POINTER(c_int32)]),
    "spp_policy_prefetch": (c_int32, [c_void_p, POINTER(c_float), c_int32, c_int64, POINTER(c_int32),
                                      POINTER(c_int32)]),
    "spp_policy_get": (c_int32, [c_void_p, POINTER(c_int32), POINTER(c_int64)]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_24787_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _check(status: int):
    if status != SPP_OK:
        raise SppError(status, lib().spp_last_error().decode())


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(POINTER(c_int32))


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data_as(POINTER(c_float))


def _i64(a):
    a = np.ascontiguousarray(a, dtype=np.int64)
    return a, a.ctypes.data_as(POINTER(c_int64))


# ------------------------------------------------------------------ lifecycle

def make_desc(L, D, n, K, I, r, S, max_batch=1, n_shared=0, dtype=DTYPE_BF16, has_proj=0, rms_eps=1e-6,
              expert_codec=0):
    return ModelDesc(L, D, n, K, I, r, n_shared, S, max_batch, dtype, int(has_proj), rms_eps, expert_codec)


def spp_blob_stride(desc: ModelDesc) -> int:
    return int(lib().spp_blob_stride(byref(desc)))


def spp_blob_layout(desc: ModelDesc) -> int:
    return int(lib().spp_blob_layout(byref(desc)))


def spp_pack_expert(desc: ModelDesc, gate, up, down, out=None):
    """Pack one expert (storage-dtype arrays gate/up [I, D], down [D, I]) into
    `out` (writable uint8, at least spp_blob_stride bytes) or a new array."""
    import numpy as np
    want = np.uint16 if desc.dtype == DTYPE_BF16 else np.float32
    mats = [np.ascontiguousarray(m, dtype=want) for m in (gate, up, down)]
    if mats[0].shape != (desc.I, desc.D) or mats[1].shape != (desc.I, desc.D) or mats[2].shape != (desc.D, desc.I):
        raise ValueError("gate/up must be [I, D] and down [D, I]")
    stride = spp_blob_stride(desc)
    if out is None:
        out = np.empty(stride, dtype=np.uint8)
    if out.dtype != np.uint8 or out.nbytes < stride or not out.flags.c_contiguous or not out.flags.writeable:
        raise ValueError("out must be a writable contiguous uint8 array of at least the blob stride")
    _check(lib().spp_pack_expert(byref(desc), mats[0].ctypes.data, mats[1].ctypes.data, mats[2].ctypes.data,
                                 out.ctypes.data))
    return out


def spp_pack_expert_q4(desc: ModelDesc, gq, gs, uq, us, dq, ds, out=None):
    """Pack one 4-bit expert: codes uint8 gate/up [I, D], down [D, I]; scales
    float16 [I, D/32] each; into `out` (writable uint8, >= blob stride) or a new array."""
    import numpy as np
    nb = desc.D // 32
    codes = [np.ascontiguousarray(q, dtype=np.uint8) for q in (gq, uq, dq)]
    scales = [np.ascontiguousarray(np.asarray(sc, dtype=np.float16)).view(np.uint16) for sc in (gs, us, ds)]
    if (codes[0].shape != (desc.I, desc.D) or codes[1].shape != (desc.I, desc.D)
            or codes[2].shape != (desc.D, desc.I) or any(sc.shape != (desc.I, nb) for sc in scales)):
        raise ValueError("codes gate/up [I, D], down [D, I]; scales [I, D/32]")
    stride = spp_blob_stride(desc)
    if out is None:
        out = np.empty(stride, dtype=np.uint8)
    if out.dtype != np.uint8 or out.nbytes < stride or not out.flags.c_contiguous or not out.flags.writeable:
        raise ValueError("out must be a writable contiguous uint8 array of at least the blob stride")
    _check(lib().spp_pack_expert_q4(byref(desc), codes[0].ctypes.data, scales[0].ctypes.data, codes[1].ctypes.data,
                                    scales[1].ctypes.data, codes[2].ctypes.data, scales[2].ctypes.data,
                                    out.ctypes.data))
    return out


def spp_create(desc: ModelDesc, stream: int = 0) -> int:
    out = c_void_p()
    _check(lib().spp_create(byref(desc), c_void_p(stream), byref(out)))
    return out.value


def spp_destroy(ctx: int):
    _check(lib().spp_destroy(c_void_p(ctx)))


def spp_bind_layer(ctx, l, router_w, adapter_a, adapter_b, proj_w, shared_blobs, host_store):
    _check(lib().spp_bind_layer(c_void_p(ctx), l, c_void_p(router_w or None), c_void_p(adapter_a or None),
                                c_void_p(adapter_b or None), c_void_p(proj_w or None),
                                c_void_p(shared_blobs or None), c_void_p(host_store or None)))


def spp_set_resident(ctx, l, experts):
    a, p = _i32(experts)
    _check(lib().spp_set_resident(c_void_p(ctx), l, p, len(a)))


# --------------------------------------------------------------- the four calls

def adapter_predict(ctx, l, x_dev: int, B: int, n: int) -> np.ndarray:
    s = np.zeros(n, dtype=np.float32)
    _check(lib().adapter_predict(c_void_p(ctx), l, c_void_p(x_dev), B, s.ctypes.data_as(POINTER(c_float))))
    return s


STATIC_SCRATCH_FLOATS = 81920


def adapter_predict_static(A_dev: int, B_dev: int, dtype: int, D: int, n: int, r: int, x_dev: int, B: int,
                           s_out_dev: int, stream: int = 0):
    """s into device memory s_out_dev (fp32 [n]) on `stream`; no context, no allocation, no wait."""
    _check(lib().adapter_predict_static(c_void_p(A_dev or None), c_void_p(B_dev or None), dtype, D, n, r,
                                        c_void_p(x_dev or None), B, c_void_p(s_out_dev or None),
                                        c_void_p(stream or None)))


def select_prefetch_budget(window_us: float, per_expert_cost_us: float, n_experts: int) -> int:
    m = c_int32()
    _check(lib().select_prefetch_budget(window_us, per_expert_cost_us, n_experts, byref(m)))
    return m.value


def expert_cache_issue_prefetch(ctx, target_layer, s, M_max):
    s, ps = _f32(s)
    issued = np.zeros(max(M_max, 1), dtype=np.int32)
    m = c_int32()
    _check(lib().expert_cache_issue_prefetch(c_void_p(ctx), target_layer, ps, M_max,
                                             issued.ctypes.data_as(POINTER(c_int32)), byref(m)))
    return issued[:m.value].tolist()


def moe_layer_forward(ctx, l, h_in_dev: int, h_out_dev: int, B: int, K: int, M_max: int):
    """Returns (topk int32 [B,K], gates fp32 [B,K], LayerStats)."""
    topk = np.zeros((B, K), dtype=np.int32)
    gates = np.zeros((B, K), dtype=np.float32)
    st = LayerStats()
    _check(lib().moe_layer_forward(c_void_p(ctx), l, c_void_p(h_in_dev), c_void_p(h_out_dev), B, M_max,
                                   topk.ctypes.data_as(POINTER(c_int32)), gates.ctypes.data_as(POINTER(c_float)),
                                   byref(st)))
    return topk, gates, st


def spp_decode_step(ctx, L: int, h_in_dev: int, h_out_dev: int, h_scratch_dev: int, B: int, K: int, M_max: int):
    """All L layers of one decode step; returns (topk [L,B,K], gates [L,B,K], [LayerStats] * L)."""
    topk = np.zeros((L, B, K), dtype=np.int32)
    gates = np.zeros((L, B, K), dtype=np.float32)
    st = (LayerStats * L)()
    _check(lib().spp_decode_step(c_void_p(ctx), c_void_p(h_in_dev), c_void_p(h_out_dev), c_void_p(h_scratch_dev),
                                 B, M_max, topk.ctypes.data_as(POINTER(c_int32)),
                                 gates.ctypes.data_as(POINTER(c_float)), st))
    return topk, gates, list(st)


def spp_last_error() -> str:
    return lib().spp_last_error().decode()


# ----------------------------------------------------------------- inspection

def spp_get_slot_table(ctx, l, S):
    e = np.zeros(S, dtype=np.int32)
    t = np.zeros(S, dtype=np.int64)
    _check(lib().spp_get_slot_table(c_void_p(ctx), l, e.ctypes.data_as(POINTER(c_int32)),
                                    t.ctypes.data_as(POINTER(c_int64))))
    return e, t


def spp_set_slot_table(ctx, l, experts, stamps):
    e, pe = _i32(experts)
    t, pt = _i64(stamps)
    _check(lib().spp_set_slot_table(c_void_p(ctx), l, pe, pt))


def spp_get_clock(ctx) -> int:
    t = c_int64()
    _check(lib().spp_get_clock(c_void_p(ctx), byref(t)))
    return t.value


def spp_set_clock(ctx, tau: int):
    _check(lib().spp_set_clock(c_void_p(ctx), tau))


def spp_get_last_transfers(ctx, cap: int = 1024):
    loads = np.zeros(3 * cap, dtype=np.int32)
    pref = np.zeros(3 * cap, dtype=np.int32)
    nl, npf = c_int32(), c_int32()
    _check(lib().spp_get_last_transfers(c_void_p(ctx), loads.ctypes.data_as(POINTER(c_int32)), byref(nl),
                                        pref.ctypes.data_as(POINTER(c_int32)), byref(npf), cap))
    tri = lambda a, k: [tuple(int(v) for v in a[3 * i:3 * i + 3]) for i in range(min(k, cap))]
    return tri(loads, nl.value), tri(pref, npf.value)


def spp_get_last_priorities(ctx, n):
    s = np.zeros(n, dtype=np.float32)
    _check(lib().spp_get_last_priorities(c_void_p(ctx), s.ctypes.data_as(POINTER(c_float))))
    return s


def spp_get_last_router_input(ctx, B, D):
    x = np.zeros((B, D), dtype=np.float32)
    _check(lib().spp_get_last_router_input(c_void_p(ctx), x.ctypes.data_as(POINTER(c_float)), B))
    return x


def spp_get_last_logits(ctx, B, n):
    z = np.zeros((B, n), dtype=np.float32)
    _check(lib().spp_get_last_logits(c_void_p(ctx), z.ctypes.data_as(POINTER(c_float)), B))
    return z


def spp_set_timing(ctx, level: int):
    """0 off, 1 on (totals only), 2 on with per-call layer times (each call waits for its layer)."""
    _check(lib().spp_set_timing(c_void_p(ctx), int(level)))


def spp_get_layer_times(ctx, L: int):
    """Per-layer totals of the timed calls: dict of numpy arrays calls, exposed_us,
    latency_us, latency_calls (each [L])."""
    calls = np.zeros(L, dtype=np.int64)
    lat_calls = np.zeros(L, dtype=np.int64)
    exposed = np.zeros(L, dtype=np.float64)
    latency = np.zeros(L, dtype=np.float64)
    _check(lib().spp_get_layer_times(c_void_p(ctx), L, calls.ctypes.data_as(POINTER(c_int64)),
                                     exposed.ctypes.data_as(POINTER(c_double)),
                                     latency.ctypes.data_as(POINTER(c_double)),
                                     lat_calls.ctypes.data_as(POINTER(c_int64))))
    return {"calls": calls, "exposed_us": exposed, "latency_us": latency, "latency_calls": lat_calls}


def spp_get_run_stats(ctx) -> RunStats:
    st = RunStats()
    _check(lib().spp_get_run_stats(c_void_p(ctx), byref(st)))
    return st


def spp_reset_run_stats(ctx):
    _check(lib().spp_reset_run_stats(c_void_p(ctx)))


def spp_probe_read_ceiling(ctx, reps: int = 40):
    """(average us per launch, GB/s) of the FFN's loads without its arithmetic."""
    us, gbs = c_double(), c_double()
    _check(lib().spp_probe_read_ceiling(c_void_p(ctx), reps, byref(us), byref(gbs)))
    return us.value, gbs.value


def spp_probe_stream_read(ctx, reps: int = 40):
    """(average us per launch, GB/s) of a plain contiguous read of K expert blobs' bytes."""
    us, gbs = c_double(), c_double()
    _check(lib().spp_probe_stream_read(c_void_p(ctx), reps, byref(us), byref(gbs)))
    return us.value, gbs.value


def spp_profile_expert_copy(ctx, l, reps) -> float:
    us = c_double()
    _check(lib().spp_profile_expert_copy(c_void_p(ctx), l, reps, byref(us)))
    return us.value


def spp_set_tier_delay(ctx, delay_us: int):
    _check(lib().spp_set_tier_delay(c_void_p(ctx), int(delay_us)))


def spp_set_prefetch_source(ctx, source: int):
    _check(lib().spp_set_prefetch_source(c_void_p(ctx), source))


def spp_set_copy_engine(ctx, engine: int):
    _check(lib().spp_set_copy_engine(c_void_p(ctx), engine))


def spp_set_ffn_workgroups(ctx, wgs: int):
    _check(lib().spp_set_ffn_workgroups(c_void_p(ctx), wgs))


def spp_set_ffn_overlap(ctx, enabled: int):
    _check(lib().spp_set_ffn_overlap(c_void_p(ctx), enabled))


def spp_set_prefetch_parallel(ctx, enabled: int):
    _check(lib().spp_set_prefetch_parallel(c_void_p(ctx), enabled))


def spp_debug_set_poison(ctx, enabled: bool):
    _check(lib().spp_debug_set_poison(c_void_p(ctx), int(bool(enabled))))


def spp_debug_set_copy_delay(ctx, delay_us: int):
    _check(lib().spp_debug_set_copy_delay(c_void_p(ctx), delay_us))


# ------------------------------------------------------- host policy (no GPU)

class SlotPolicy:
    """Host-only replacement / prefetch-selection policy (same code the context runs)."""

    def __init__(self, S, n, resident=()):
        self._h = None
        self.S, self.n = S, n
        a, p = _i32(list(resident))
        out = c_void_p()
        _check(lib().spp_policy_create(S, n, p, len(a), byref(out)))
        self._h = out.value

    def close(self):
        if getattr(self, "_h", None):
            _check(lib().spp_policy_destroy(c_void_p(self._h)))
            self._h = None

    __del__ = close

    def on_demand(self, needed, tau):
        a, p = _i32(list(needed))
        out = np.zeros(3 * self.n, dtype=np.int32)
        k = c_int32()
        _check(lib().spp_policy_on_demand(c_void_p(self._h), p, len(a), tau, out.ctypes.data_as(POINTER(c_int32)),
                                          byref(k)))
        return [tuple(int(v) for v in out[3 * i:3 * i + 3]) for i in range(k.value)]

    def prefetch(self, s, M_max, tau):
        s, ps = _f32(s)
        out = np.zeros(3 * max(M_max, 1), dtype=np.int32)
        k = c_int32()
        _check(lib().spp_policy_prefetch(c_void_p(self._h), ps, M_max, tau, out.ctypes.data_as(POINTER(c_int32)),
                                         byref(k)))
        return [tuple(int(v) for v in out[3 * i:3 * i + 3]) for i in range(k.value)]

    def table(self):
        e = np.zeros(self.S, dtype=np.int32)
        t = np.zeros(self.S, dtype=np.int64)
        _check(lib().spp_policy_get(c_void_p(self._h), e.ctypes.data_as(POINTER(c_int32)),
                                    t.ctypes.data_as(POINTER(c_int64))))
        return e, t
