"""ctypes binding of libinertiakv.so: argument marshalling only.

Every function carries the name of the C entry point it calls and takes torch tensors for device buffers;
it passes their device pointers and the current HIP stream, and raises KVError on a non-zero status.  All
computation happens in the HIP kernels behind the C ABI; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libinertiakv.so")

KV_OK, KV_ERR_INVALID_ARG, KV_ERR_UNSUPPORTED, KV_ERR_WORKSPACE, KV_ERR_HIP = 0, -1, -2, -3, -4
KV_F32, KV_BF16 = 0, 1
KV_INIT_MEAN, KV_INIT_MIN = 0, 1
KV_RULE_EMA, KV_RULE_SINGLE_STEP, KV_RULE_CUMULATIVE = 0, 1, 2
KV_SCORE_ATTENTION, KV_SCORE_VNORM, KV_SCORE_ENTROPY, KV_SCORE_NORMS_EMITTED = 0, 1, 2, 4
KV_EMIT_SCORES, KV_EMIT_VNORMS = 1, 2
KV_FAULT_EXCHANGE_TIMEOUT = 1
KV_PATH_LDS, KV_PATH_EXCHANGE, KV_PATH_LOGITS = 0, 1, 2
KV_PHASES = 5
PHASES = ("append", "score", "fold", "select", "compact")

EXPORTED = ("kv_workspace_bytes", "kv_score_ema", "kv_topk_select", "kv_compact", "kv_evict_step",
            "kv_append", "kv_attend_score", "kv_evict_finish", "kv_rank_trace_state_bytes", "kv_score_merge",
            "kv_score_plan", "kv_fault_status", "kv_set_exchange_wait_limit", "kv_evict_step_static",
            "kv_value_norms", "kv_status_string")
KV_STATIC_SCRATCH_BYTES = 64 << 20
KV_TRACE_COUNTS = 10


class KVError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")
        self.status = status


class KvShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class KvParams(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("budget", ctypes.c_int32), ("refresh_period", ctypes.c_int32),
                ("score_free", ctypes.c_int32), ("nonrefresh_init", ctypes.c_int32),
                ("recency_bias", ctypes.c_float), ("recency_window", ctypes.c_int32), ("rule", ctypes.c_int32),
                ("score_variant", ctypes.c_int32), ("score_merge", ctypes.c_int32)]


class KvTrace(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_void_p * KV_PHASES), ("end", ctypes.c_void_p * KV_PHASES)]


class KvScoreInfo(ctypes.Structure):
    _fields_ = [("merge", ctypes.c_int32), ("path", ctypes.c_int32), ("chunks", ctypes.c_int32)]


class KvRankTrace(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("max_pos", ctypes.c_int32), ("state", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("raw_keep", ctypes.c_void_p), ("ema_keep", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads the built library; raises if it is missing (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2609_03515_amd.build.build()")
    lib = ctypes.CDLL(path)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    shp, prm, trc = ctypes.POINTER(KvShape), ctypes.POINTER(KvParams), ctypes.POINTER(KvTrace)
    rtr = ctypes.POINTER(KvRankTrace)
    lib.kv_workspace_bytes.argtypes = [shp, i32, ctypes.POINTER(sz)]
    lib.kv_score_ema.argtypes = [shp, i32, vp, vp, vp, i32, f32, f32, i32, vp, vp, vp, sz, vp]
    lib.kv_topk_select.argtypes = [shp, i32, i32, vp, vp, vp, vp, sz, vp]
    lib.kv_compact.argtypes = [shp, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.kv_evict_step.argtypes = [shp, prm, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                  ctypes.POINTER(i32), vp, vp, trc, rtr, vp, sz, vp]
    lib.kv_append.argtypes = [shp, prm, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.kv_attend_score.argtypes = [shp, i32, i32, i32, vp, vp, vp, vp, i32, f32, i32, i32, vp, vp, sz, vp]
    lib.kv_evict_finish.argtypes = [shp, prm, i32, i32, vp, vp, vp, vp, vp, ctypes.POINTER(i32), vp, vp, rtr, vp,
                                    sz, vp]
    lib.kv_value_norms.argtypes = [shp, i32, vp, vp, vp]
    lib.kv_rank_trace_state_bytes.argtypes = [i32, i32, ctypes.POINTER(sz)]
    lib.kv_score_merge.argtypes = [shp, i32, prm, ctypes.POINTER(i32)]
    lib.kv_score_plan.argtypes = [shp, i32, prm, ctypes.POINTER(KvScoreInfo)]
    lib.kv_fault_status.argtypes = [vp, sz, vp, i32, vp]
    lib.kv_set_exchange_wait_limit.argtypes = [i32]
    lib.kv_evict_step_static.argtypes = [shp, prm, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.POINTER(i32), vp, vp, trc, rtr, vp]
    for fn in EXPORTED[:-1]:
        getattr(lib, fn).restype = i32
    lib.kv_status_string.argtypes = [i32]
    lib.kv_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().kv_status_string(int(status)).decode()


def _check(fn, status):
    if status != KV_OK:
        raise KVError(fn, status)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_shape(batch, layers, n_q_heads, n_kv_heads, head_dim, capacity, dtype) -> KvShape:
    if isinstance(dtype, str):
        dtype = {"f32": KV_F32, "bf16": KV_BF16}[dtype]
    elif dtype in (torch.float32, torch.bfloat16):
        dtype = KV_F32 if dtype == torch.float32 else KV_BF16
    return KvShape(batch, layers, n_q_heads, n_kv_heads, head_dim, capacity, dtype)


def make_params(alpha, budget, refresh_period=1, score_free=False, nonrefresh_init="mean", recency_bias=0.0,
                recency_window=0, rule="ema", vnorm=False, entropy=False, norms_emitted=False,
                score_merge=0) -> KvParams:
    init = {"mean": KV_INIT_MEAN, "min": KV_INIT_MIN}[nonrefresh_init] if isinstance(nonrefresh_init, str) \
        else int(nonrefresh_init)
    rl = {"ema": KV_RULE_EMA, "single": KV_RULE_SINGLE_STEP, "cumulative": KV_RULE_CUMULATIVE}[rule] \
        if isinstance(rule, str) else int(rule)
    variant = (KV_SCORE_VNORM if vnorm else 0) | (KV_SCORE_ENTROPY if entropy else 0) | \
        (KV_SCORE_NORMS_EMITTED if norms_emitted else 0)
    return KvParams(float(alpha), int(budget), int(refresh_period), int(bool(score_free)), init,
                    float(recency_bias), int(recency_window), rl, variant, int(score_merge))


def kv_workspace_bytes(shape: KvShape, n_max: int) -> int:
    out = ctypes.c_size_t(0)
    _check("kv_workspace_bytes", load_library().kv_workspace_bytes(ctypes.byref(shape), int(n_max),
                                                                    ctypes.byref(out)))
    return out.value


def kv_score_merge(shape: KvShape, n: int, params: KvParams) -> int:
    out = ctypes.c_int32(0)
    _check("kv_score_merge", load_library().kv_score_merge(ctypes.byref(shape), int(n), ctypes.byref(params),
                                                            ctypes.byref(out)))
    return out.value


def kv_score_plan(shape: KvShape, n: int, params: KvParams) -> KvScoreInfo:
    out = KvScoreInfo()
    _check("kv_score_plan", load_library().kv_score_plan(ctypes.byref(shape), int(n), ctypes.byref(params),
                                                          ctypes.byref(out)))
    return out


def kv_fault_status(ws, out=None, clear=False, stream=None):
    """Queues the copy of the workspace's fault word into `out` (a device int32/uint32 tensor of one element,
    or None) and/or its clearing."""
    _check("kv_fault_status", load_library().kv_fault_status(_ptr(ws), _ws_bytes(ws), _ptr(out), int(bool(clear)),
                                                              _stream(stream)))


def kv_set_exchange_wait_limit(polls: int) -> int:
    return int(load_library().kv_set_exchange_wait_limit(int(polls)))


def kv_score_ema(shape, n, q, k, pos, cur_pos, alpha, recency_bias, recency_window, u, s_out, ws, stream=None):
    _check("kv_score_ema", load_library().kv_score_ema(
        ctypes.byref(shape), int(n), _ptr(q), _ptr(k), _ptr(pos), int(cur_pos), float(alpha),
        float(recency_bias), int(recency_window), _ptr(u), _ptr(s_out), _ptr(ws),
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))


def kv_topk_select(shape, n, budget, u, pos, keep, ws, stream=None):
    _check("kv_topk_select", load_library().kv_topk_select(
        ctypes.byref(shape), int(n), int(budget), _ptr(u), _ptr(pos), _ptr(keep), _ptr(ws),
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))


def kv_compact(shape, n, budget, keep, k, v, u, pos, ws, stream=None, v_norms=None):
    _check("kv_compact", load_library().kv_compact(
        ctypes.byref(shape), int(n), int(budget), _ptr(keep), _ptr(k), _ptr(v), _ptr(u), _ptr(pos), _ptr(v_norms),
        _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))


def kv_value_norms(shape, n, v, v_norms, stream=None):
    """Fills the value-norm cache v_norms [layers][batch][n_kv][cap] float for rows [0, n) from V."""
    _check("kv_value_norms", load_library().kv_value_norms(ctypes.byref(shape), int(n), _ptr(v), _ptr(v_norms),
                                                            _stream(stream)))


def kv_evict_step(shape, params, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, ws, keep_out=None,
                  s_out=None, trace: KvTrace | None = None, rank_trace: KvRankTrace | None = None,
                  stream=None, v_norms=None) -> int:
    """Returns n_out = min(B, n_in + 1)."""
    n_out = ctypes.c_int32(-1)
    _check("kv_evict_step", load_library().kv_evict_step(
        ctypes.byref(shape), ctypes.byref(params), int(t), int(n_in), int(new_pos), _ptr(q), _ptr(k_new),
        _ptr(v_new), _ptr(k), _ptr(v), _ptr(u), _ptr(pos), _ptr(v_norms), ctypes.byref(n_out), _ptr(keep_out),
        _ptr(s_out),
        ctypes.byref(trace) if trace is not None else None,
        ctypes.byref(rank_trace) if rank_trace is not None else None, _ptr(ws),
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return n_out.value


def kv_evict_step_static(shape, params, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, keep_out=None,
                         s_out=None, trace: KvTrace | None = None, rank_trace: KvRankTrace | None = None,
                         stream=None, v_norms=None) -> int:
    """kv_evict_step with the library's static scratch instead of a workspace.  Returns n_out."""
    n_out = ctypes.c_int32(-1)
    _check("kv_evict_step_static", load_library().kv_evict_step_static(
        ctypes.byref(shape), ctypes.byref(params), int(t), int(n_in), int(new_pos), _ptr(q), _ptr(k_new),
        _ptr(v_new), _ptr(k), _ptr(v), _ptr(u), _ptr(pos), _ptr(v_norms), ctypes.byref(n_out), _ptr(keep_out),
        _ptr(s_out),
        ctypes.byref(trace) if trace is not None else None,
        ctypes.byref(rank_trace) if rank_trace is not None else None, _stream(stream)))
    return n_out.value


def kv_rank_trace_state_bytes(batch: int, max_pos: int) -> int:
    out = ctypes.c_size_t(0)
    _check("kv_rank_trace_state_bytes", load_library().kv_rank_trace_state_bytes(int(batch), int(max_pos),
                                                                                  ctypes.byref(out)))
    return out.value


def make_rank_trace(k, max_pos, state, counts, raw_keep=None, ema_keep=None) -> KvRankTrace:
    """state: a zero-filled device tensor of kv_rank_trace_state_bytes() bytes; counts: int32 device tensor
    [batch][KV_TRACE_COUNTS].  Keep the tensors alive while the struct is in use."""
    return KvRankTrace(int(k), int(max_pos), _ptr(state), _ptr(counts), _ptr(raw_keep), _ptr(ema_keep))


def _ws_bytes(ws):
    return ws.numel() * ws.element_size() if ws is not None else 0


def kv_append(shape, params, t, n_in, new_pos, k_new, v_new, k, v, u, pos, stream=None, v_norms=None):
    _check("kv_append", load_library().kv_append(
        ctypes.byref(shape), ctypes.byref(params), int(t), int(n_in), int(new_pos), _ptr(k_new), _ptr(v_new),
        _ptr(k), _ptr(v), _ptr(u), _ptr(pos), _ptr(v_norms), _stream(stream)))


def kv_attend_score(shape, layer0, layer_count, n, q, k, v, pos, cur_pos, recency_bias, recency_window,
                    emit_scores, o, ws, stream=None):
    _check("kv_attend_score", load_library().kv_attend_score(
        ctypes.byref(shape), int(layer0), int(layer_count), int(n), _ptr(q), _ptr(k), _ptr(v), _ptr(pos),
        int(cur_pos), float(recency_bias), int(recency_window), int(emit_scores), _ptr(o), _ptr(ws),
        _ws_bytes(ws), _stream(stream)))


def kv_evict_finish(shape, params, t, n, k, v, u, pos, ws, keep_out=None, s_out=None,
                    rank_trace: KvRankTrace | None = None, stream=None, v_norms=None) -> int:
    """Returns n_out = min(B, n)."""
    n_out = ctypes.c_int32(-1)
    _check("kv_evict_finish", load_library().kv_evict_finish(
        ctypes.byref(shape), ctypes.byref(params), int(t), int(n), _ptr(k), _ptr(v), _ptr(u), _ptr(pos),
        _ptr(v_norms), ctypes.byref(n_out), _ptr(keep_out), _ptr(s_out),
        ctypes.byref(rank_trace) if rank_trace is not None else None, _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return n_out.value


def workspace(shape: KvShape, n_max: int, device="cuda") -> torch.Tensor:
    """A caller-owned workspace tensor of kv_workspace_bytes() bytes (256-byte aligned by the allocator), its
    fault word cleared on the current stream."""
    nbytes = kv_workspace_bytes(shape, n_max)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    kv_fault_status(ws, None, clear=True)
    return ws


class KvCache:
    """One cache's device buffers (caller-owned torch tensors) and its cached row count n, for `evict_step`.

    k, v: [layers][batch][n_kv_heads][capacity][head_dim] of the shape's dtype; u: [batch][capacity] f32;
    pos: [batch][capacity] int32; ws: a workspace of kv_workspace_bytes(shape, capacity) bytes; v_norms: the
    optional per-row value-norm cache [layers][batch][n_kv_heads][capacity] f32 (VNorm scoring)."""

    def __init__(self, shape: KvShape, k, v, u, pos, n: int, ws, v_norms=None):
        self.shape, self.k, self.v, self.u, self.pos, self.n, self.ws = shape, k, v, u, pos, int(n), ws
        self.v_norms = v_norms

    @classmethod
    def allocate(cls, shape: KvShape, device="cuda", v_norms=False) -> "KvCache":
        """Zero-filled buffers for `shape` with n = 0; the caller fills the prefill rows and sets n."""
        dt = torch.float32 if shape.dtype == KV_F32 else torch.bfloat16
        rows = (shape.layers, shape.batch, shape.n_kv_heads, shape.capacity)
        return cls(shape, torch.zeros(rows + (shape.head_dim,), dtype=dt, device=device),
                   torch.zeros(rows + (shape.head_dim,), dtype=dt, device=device),
                   torch.zeros(shape.batch, shape.capacity, dtype=torch.float32, device=device),
                   torch.zeros(shape.batch, shape.capacity, dtype=torch.int32, device=device), 0,
                   workspace(shape, shape.capacity, device),
                   torch.zeros(rows, dtype=torch.float32, device=device) if v_norms else None)


def evict_step(cache: KvCache, q, k_new, v_new, t: int, params: KvParams, new_pos: int, keep_out=None,
               s_out=None, stream=None) -> int:
    """One decode step t (1-based) through kv_evict_step on `cache`'s buffers: the newcomer (q, k_new, v_new at
    position new_pos) is appended, and on refresh steps the cache is scored, folded, selected and compacted to
    the budget.  Sets cache.n to the new row count and returns it; raises KVError on a non-zero status."""
    cache.n = kv_evict_step(cache.shape, params, t, cache.n, new_pos, q, k_new, v_new, cache.k, cache.v,
                            cache.u, cache.pos, cache.ws, keep_out=keep_out, s_out=s_out, stream=stream,
                            v_norms=cache.v_norms)
    return cache.n


def faults(ws, clear=False) -> int:
    """The workspace's fault word (kv_fault bits), read after synchronising the current stream."""
    out = torch.zeros(1, dtype=torch.int32, device=ws.device)
    kv_fault_status(ws, out, clear=clear)
    return int(out.item()) & 0xffffffff


# --- HIP events for the timing hooks (runtime plumbing, no computation) -------------------------------------
_hip = None


def _hip_runtime():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        _hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        _hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        _hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        _hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        _hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    return _hip


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence


class HipEvent:
    """A HIP event.  timing_only: created with hipEventDisableSystemFence, so recording it does not write back
    and invalidate the caches (a timestamp between kernels that leaves them undisturbed); read it only after
    the stream has been synchronized."""

    def __init__(self, timing_only: bool = False):
        self.handle = ctypes.c_void_p()
        if timing_only:
            rc = _hip_runtime().hipEventCreateWithFlags(ctypes.byref(self.handle), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        else:
            rc = _hip_runtime().hipEventCreate(ctypes.byref(self.handle))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")

    def record(self, stream=None):
        rc = _hip_runtime().hipEventRecord(self.handle, _stream(stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_ms(self, later: "HipEvent") -> float:
        _hip_runtime().hipEventSynchronize(later.handle)
        out = ctypes.c_float(0)
        rc = _hip_runtime().hipEventElapsedTime(ctypes.byref(out), self.handle, later.handle)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return out.value

    def __del__(self):
        if _hip is not None and self.handle:
            _hip.hipEventDestroy(self.handle)
            self.handle = ctypes.c_void_p()


def make_trace(pairs: dict) -> KvTrace:
    """pairs: phase name -> (begin HipEvent, end HipEvent)."""
    tr = KvTrace()
    for i, name in enumerate(PHASES):
        if name in pairs:
            tr.begin[i] = pairs[name][0].handle.value
            tr.end[i] = pairs[name][1].handle.value
    return tr
