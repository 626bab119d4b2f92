"""The C ABI library loads on a machine without a GPU, exports every declared entry point, and rejects bad
arguments on the host before any HIP call (every call here is invalid, so nothing is launched)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2609_03515_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "inertiakv.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:kv_status|const char\*|int32_t)\s+(kv_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2609_03515_amd import build
        build.build()
    return B.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert names == sorted(B.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name
    assert ctypes.CDLL(B.LIB_PATH).kv_evict_step is not None


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert B.status_string(code)
    assert B.status_string(-99) == "unknown status"


GOOD = dict(batch=2, layers=3, n_q_heads=8, n_kv_heads=2, head_dim=128, capacity=100, dtype="bf16")


def shape(**kw):
    d = dict(GOOD)
    d.update(kw)
    return B.make_shape(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), B.KV_ERR_UNSUPPORTED),
    (dict(n_q_heads=7), B.KV_ERR_INVALID_ARG),
    (dict(n_q_heads=64, n_kv_heads=2), B.KV_ERR_UNSUPPORTED),          # group 32 > 16
    (dict(n_q_heads=32, n_kv_heads=2, head_dim=64), B.KV_ERR_UNSUPPORTED),  # group 16 > 8 lanes of a d64 bf16 row
    (dict(dtype=7), B.KV_ERR_UNSUPPORTED),
    (dict(batch=0), B.KV_ERR_INVALID_ARG),
    (dict(layers=300), B.KV_ERR_UNSUPPORTED),
])
def test_bad_shapes(lib, kw, status):
    with pytest.raises(B.KVError) as e:
        B.kv_workspace_bytes(shape(**kw), 10)
    assert e.value.status == status


def test_workspace_monotone(lib):
    s = shape(capacity=40000)
    sizes = [B.kv_workspace_bytes(s, n) for n in (1, 100, 3278, 5000, 6000, 40000)]
    assert sizes == sorted(sizes)
    with pytest.raises(B.KVError):
        B.kv_workspace_bytes(s, 40001)


FAKE = 1 << 20   # a host-side stand-in address, never dereferenced: every call below fails validation


def _score(s, n=10, alpha=0.9, ws=None, ws_bytes=0, q=FAKE, window=0):
    return lib_().kv_score_ema(ctypes.byref(s), n, q, FAKE, FAKE, 0, alpha, 0.0, window, FAKE, None, ws,
                               ws_bytes, None)


def lib_():
    return B.load_library()


def test_score_validation(lib):
    s = shape()
    assert _score(s, n=0) == B.KV_ERR_INVALID_ARG
    assert _score(s, n=101) == B.KV_ERR_INVALID_ARG
    assert _score(s, alpha=1.0) == B.KV_ERR_INVALID_ARG
    assert _score(s, alpha=-0.1) == B.KV_ERR_INVALID_ARG
    assert _score(s, alpha=float("nan")) == B.KV_ERR_INVALID_ARG
    assert _score(s, q=None) == B.KV_ERR_INVALID_ARG
    assert _score(s, q=FAKE + 4) == B.KV_ERR_UNSUPPORTED      # misaligned rows
    assert _score(s, window=-1) == B.KV_ERR_INVALID_ARG
    assert _score(s) == B.KV_ERR_WORKSPACE                  # no workspace
    need = B.kv_workspace_bytes(s, 10)
    assert _score(s, ws=FAKE, ws_bytes=need - 1) == B.KV_ERR_WORKSPACE
    assert _score(s, ws=FAKE + 16, ws_bytes=need) == B.KV_ERR_INVALID_ARG   # workspace not 256-aligned


def test_select_compact_validation(lib):
    s = shape()
    L = lib_()
    assert L.kv_topk_select(ctypes.byref(s), 10, 0, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_topk_select(ctypes.byref(s), 10, 5, None, FAKE, FAKE, FAKE, 1 << 30, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_topk_select(ctypes.byref(s), 10, 5, FAKE, FAKE, FAKE, None, 0, None) == B.KV_ERR_WORKSPACE
    assert L.kv_compact(ctypes.byref(s), 10, 5, None, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == \
        B.KV_ERR_INVALID_ARG
    assert L.kv_compact(ctypes.byref(s), 10, 5, FAKE, FAKE + 8, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == \
        B.KV_ERR_UNSUPPORTED
    # n <= B is a no-op that still validates the workspace
    assert L.kv_compact(ctypes.byref(s), 10, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, FAKE, 1 << 30, None) == \
        B.KV_ERR_UNSUPPORTED                                      # misaligned norm cache
    assert L.kv_compact(ctypes.byref(s), 10, 50, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == \
        B.KV_ERR_WORKSPACE


def _step(s, p, t=1, n_in=10, n_out=True, **kw):
    args = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k=FAKE, v=FAKE, u=FAKE, pos=FAKE, ws=None, ws_bytes=0, norms=None)
    args.update(kw)
    out = ctypes.c_int32(-7)
    rc = lib_().kv_evict_step(ctypes.byref(s), ctypes.byref(p) if p is not None else None, t, n_in, 5,
                              args["q"], args["k_new"], args["v_new"], args["k"], args["v"], args["u"], args["pos"],
                              args["norms"], ctypes.byref(out) if n_out else None, None, None, None, args.get("rt"),
                              args["ws"], args["ws_bytes"], None)
    return rc, out.value


def test_score_merge_query(lib):
    s = shape()   # 2 KV heads
    assert B.kv_score_merge(s, 50, B.make_params(0.9, 20, score_merge=2)) == 2
    assert B.kv_score_merge(s, 50, B.make_params(0.9, 20, score_merge=1)) == 1
    assert B.kv_score_merge(s, 50, B.make_params(0.9, 20, vnorm=True)) == 1
    out = ctypes.c_int32(-7)
    L = lib_()
    for p, n in ((B.make_params(0.9, 20, score_merge=4), 50), (B.make_params(0.9, 20, vnorm=True, score_merge=2), 50),
                 (B.make_params(0.9, 20), 0), (B.make_params(0.9, 20), 101)):
        assert L.kv_score_merge(ctypes.byref(s), n, ctypes.byref(p), ctypes.byref(out)) == B.KV_ERR_INVALID_ARG
    assert L.kv_score_merge(ctypes.byref(s), 50, ctypes.byref(B.make_params(0.9, 20)), None) == B.KV_ERR_INVALID_ARG
    assert out.value == -7


def test_step_validation(lib):
    s = shape()
    good = B.make_params(0.9, 20)
    assert _step(s, None)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, good, n_out=False)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, good, t=0)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, good, n_in=100)[0] == B.KV_ERR_INVALID_ARG          # n_in + 1 > capacity
    assert _step(s, good, n_in=-1)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, B.make_params(1.0, 20))[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, B.make_params(0.9, 0))[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, B.make_params(0.9, 20, refresh_period=0))[0] == B.KV_ERR_INVALID_ARG
    bad_init = B.make_params(0.9, 20)
    bad_init.nonrefresh_init = 5
    assert _step(s, bad_init)[0] == B.KV_ERR_INVALID_ARG
    bad_rule = B.make_params(0.9, 20)
    bad_rule.rule = 9
    assert _step(s, bad_rule)[0] == B.KV_ERR_INVALID_ARG
    bad_variant = B.make_params(0.9, 20, vnorm=True, entropy=True)
    assert bad_variant.score_variant == B.KV_SCORE_VNORM | B.KV_SCORE_ENTROPY
    bad_variant.score_variant = 8
    assert _step(s, bad_variant)[0] == B.KV_ERR_INVALID_ARG
    for merge in (-1, 9):
        assert _step(s, B.make_params(0.9, 20, score_merge=merge))[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, B.make_params(0.9, 20, score_merge=3))[0] == B.KV_ERR_INVALID_ARG   # not a divisor of n_kv
    assert _step(s, B.make_params(0.9, 20, vnorm=True, score_merge=2))[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, B.make_params(0.9, 20, vnorm=True, score_merge=1))[0] == B.KV_ERR_WORKSPACE
    assert _step(s, B.make_params(0.9, 20, score_merge=2))[0] == B.KV_ERR_WORKSPACE
    assert _step(s, good, v_new=None)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, good, k=FAKE + 2)[0] == B.KV_ERR_UNSUPPORTED
    assert _step(s, good, norms=FAKE + 2)[0] == B.KV_ERR_UNSUPPORTED
    rc, out = _step(s, good)
    assert rc == B.KV_ERR_WORKSPACE and out == -7                      # nothing written on failure


def test_append_validation(lib):
    s = shape()
    good = B.make_params(0.9, 20)
    L = lib_()

    def call(p=good, t=1, n_in=10, new_pos=5, k_new=FAKE, k=FAKE, u=FAKE, norms=None):
        return L.kv_append(ctypes.byref(s), ctypes.byref(p) if p is not None else None, t, n_in, new_pos, k_new,
                           FAKE, k, FAKE, u, FAKE, norms, None)
    assert call(p=None) == B.KV_ERR_INVALID_ARG
    assert call(p=B.make_params(0.9, 0)) == B.KV_ERR_INVALID_ARG
    assert call(t=0) == B.KV_ERR_INVALID_ARG
    assert call(n_in=100) == B.KV_ERR_INVALID_ARG
    assert call(new_pos=-1) == B.KV_ERR_INVALID_ARG
    assert call(k_new=None) == B.KV_ERR_INVALID_ARG
    assert call(k=FAKE + 8) == B.KV_ERR_UNSUPPORTED
    assert call(u=FAKE + 2) == B.KV_ERR_UNSUPPORTED
    assert call(norms=FAKE + 2) == B.KV_ERR_UNSUPPORTED


def test_attend_validation(lib):
    s = shape()   # 3 layers
    L = lib_()
    need = B.kv_workspace_bytes(s, 10)

    def call(layer0=0, count=3, n=10, q=FAKE, o=FAKE, window=0, ws=FAKE, ws_bytes=need, emit=1):
        return L.kv_attend_score(ctypes.byref(s), layer0, count, n, q, FAKE, FAKE, FAKE, 9, 0.5, window, emit, o,
                                 ws, ws_bytes, None)
    assert call(emit=4) == B.KV_ERR_INVALID_ARG                  # unknown emit bit
    assert call(layer0=-1) == B.KV_ERR_INVALID_ARG
    assert call(count=0) == B.KV_ERR_INVALID_ARG
    assert call(layer0=2, count=2) == B.KV_ERR_INVALID_ARG        # past the last layer
    assert call(n=0) == B.KV_ERR_INVALID_ARG
    assert call(n=101) == B.KV_ERR_INVALID_ARG
    assert call(window=-2) == B.KV_ERR_INVALID_ARG
    assert call(o=None) == B.KV_ERR_INVALID_ARG
    assert call(q=FAKE + 4) == B.KV_ERR_UNSUPPORTED
    assert call(o=FAKE + 1) == B.KV_ERR_UNSUPPORTED                # bf16 output needs 2-byte alignment
    assert call(ws=None, ws_bytes=0) == B.KV_ERR_WORKSPACE
    assert call(ws_bytes=need - 1) == B.KV_ERR_WORKSPACE


def test_finish_validation(lib):
    s = shape()
    good = B.make_params(0.9, 20)
    L = lib_()
    out = ctypes.c_int32(-7)

    def call(p=good, t=1, n=10, k=FAKE, n_out=True, ws=None, ws_bytes=0):
        return L.kv_evict_finish(ctypes.byref(s), ctypes.byref(p) if p is not None else None, t, n, k, FAKE, FAKE,
                                 FAKE, None, ctypes.byref(out) if n_out else None, None, None, None, ws, ws_bytes,
                                 None)
    assert call(p=None) == B.KV_ERR_INVALID_ARG
    assert call(t=0) == B.KV_ERR_INVALID_ARG
    assert call(n=0) == B.KV_ERR_INVALID_ARG
    assert call(n=101) == B.KV_ERR_INVALID_ARG
    assert call(n_out=False) == B.KV_ERR_INVALID_ARG
    assert call(k=FAKE + 8) == B.KV_ERR_UNSUPPORTED
    assert call(p=B.make_params(0.9, 20, score_merge=3)) == B.KV_ERR_INVALID_ARG
    assert call(p=B.make_params(0.9, 20, vnorm=True, score_merge=4)) == B.KV_ERR_INVALID_ARG
    assert call() == B.KV_ERR_WORKSPACE and out.value == -7



def test_rank_trace_validation(lib):
    s = shape()
    good = B.make_params(0.9, 20)
    need = B.kv_workspace_bytes(s, 11)
    assert B.kv_rank_trace_state_bytes(2, 64) == 2 * (4 + 2 * 2) * 4
    assert B.kv_rank_trace_state_bytes(1, 65) == (4 + 2 * 3) * 4
    with pytest.raises(B.KVError):
        B.kv_rank_trace_state_bytes(0, 10)
    for bad in (B.KvRankTrace(0, 100, FAKE, FAKE), B.KvRankTrace(5, 0, FAKE, FAKE), B.KvRankTrace(5, 100, None, FAKE),
                B.KvRankTrace(5, 100, FAKE, None)):
        assert _step(s, good, rt=ctypes.byref(bad), ws=FAKE, ws_bytes=need)[0] == B.KV_ERR_INVALID_ARG
    assert _step(s, good, rt=ctypes.byref(B.KvRankTrace(5, 100, FAKE + 2, FAKE)), ws=FAKE,
                 ws_bytes=need)[0] == B.KV_ERR_UNSUPPORTED


def test_score_plan_query(lib):
    s = shape()
    info = B.kv_score_plan(s, 50, B.make_params(0.9, 20, score_merge=2))
    assert (info.merge, info.path, info.chunks) == (2, B.KV_PATH_LDS, 1)
    L = lib_()
    out = B.KvScoreInfo(-7, -7, -7)
    for p, n in ((B.make_params(0.9, 20, score_merge=4), 50), (B.make_params(0.9, 20), 0),
                 (B.make_params(0.9, 20), 101)):
        assert L.kv_score_plan(ctypes.byref(s), n, ctypes.byref(p), ctypes.byref(out)) == B.KV_ERR_INVALID_ARG
    assert L.kv_score_plan(ctypes.byref(s), 50, ctypes.byref(B.make_params(0.9, 20)), None) == B.KV_ERR_INVALID_ARG
    assert (out.merge, out.path, out.chunks) == (-7, -7, -7)


def test_fault_status_validation(lib):
    L = lib_()
    assert L.kv_fault_status(None, 1 << 20, FAKE, 0, None) == B.KV_ERR_WORKSPACE
    assert L.kv_fault_status(FAKE, 255, FAKE, 0, None) == B.KV_ERR_WORKSPACE
    assert L.kv_fault_status(FAKE + 16, 1 << 20, FAKE, 0, None) == B.KV_ERR_INVALID_ARG   # workspace not aligned
    assert L.kv_fault_status(FAKE, 1 << 20, FAKE + 2, 0, None) == B.KV_ERR_INVALID_ARG    # misaligned output word
    assert L.kv_fault_status(FAKE, 1 << 20, None, 0, None) == B.KV_ERR_INVALID_ARG        # nothing asked for


def test_exchange_wait_limit_setter(lib):
    default = B.kv_set_exchange_wait_limit(7)
    assert default > 1000                       # about 0.1 s of sleeps
    assert B.kv_set_exchange_wait_limit(-1) == 7
    assert B.kv_set_exchange_wait_limit(-1) == default


def test_static_step_rejects_what_its_scratch_cannot_hold(lib):
    """The allocation-free step refuses, on the host, a step whose slabs need chunked scoring (first step over
    32k tokens) and one whose scratch exceeds the static array (batch 64 x 4,097 tokens), queueing nothing."""
    out = ctypes.c_int32(-7)

    def call(s, p, t, n_in, new_pos):
        return lib_().kv_evict_step_static(ctypes.byref(s), ctypes.byref(p), t, n_in, new_pos, *(FAKE,) * 7, None,
                                           ctypes.byref(out), None, None, None, None, None)
    s = B.make_shape(8, 32, 32, 8, 128, 32769, "bf16")
    assert call(s, B.make_params(0.9, 3277), 1, 32768, 32768) == B.KV_ERR_UNSUPPORTED
    big = B.make_shape(64, 32, 32, 8, 128, 4097, "bf16")
    assert call(big, B.make_params(0.9, 4096), 2, 4096, 5000) == B.KV_ERR_WORKSPACE
    assert call(s, B.make_params(0.9, 3277), 0, 3277, 40000) == B.KV_ERR_INVALID_ARG   # argument checks as the step
    assert call(s, B.make_params(1.0, 3277), 2, 3277, 40000) == B.KV_ERR_INVALID_ARG
    assert out.value == -7


def test_value_norms_validation(lib):
    s = shape()
    L = lib_()
    assert L.kv_value_norms(ctypes.byref(s), 0, FAKE, FAKE, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_value_norms(ctypes.byref(s), 101, FAKE, FAKE, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_value_norms(ctypes.byref(s), 10, None, FAKE, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_value_norms(ctypes.byref(s), 10, FAKE, None, None) == B.KV_ERR_INVALID_ARG
    assert L.kv_value_norms(ctypes.byref(s), 10, FAKE + 8, FAKE, None) == B.KV_ERR_UNSUPPORTED
    assert L.kv_value_norms(ctypes.byref(s), 10, FAKE, FAKE + 1, None) == B.KV_ERR_UNSUPPORTED


def test_cache_wrapper_raises_and_keeps_n(lib):
    """evict_step(cache, ...) raises KVError on a rejected call and leaves the cache's row count alone (CPU
    tensors stand in for the buffers: the host validation rejects both calls before any HIP call)."""
    s = shape(capacity=16)
    rows = (3, 2, 2, 16, 128)
    cache = B.KvCache(s, torch.zeros(rows, dtype=torch.bfloat16), torch.zeros(rows, dtype=torch.bfloat16),
                      torch.zeros(2, 16), torch.zeros(2, 16, dtype=torch.int32), 5, torch.zeros(256, dtype=torch.uint8))
    q, kv_new = torch.zeros(2, 8, 128, dtype=torch.bfloat16), torch.zeros(3, 2, 2, 128, dtype=torch.bfloat16)
    params = B.make_params(0.9, 8)
    with pytest.raises(B.KVError) as e:
        B.evict_step(cache, q, kv_new, kv_new, 0, params, new_pos=20, stream=0)     # steps are 1-based
    assert e.value.status == B.KV_ERR_INVALID_ARG and cache.n == 5
    cache.n = 16                                                                   # no room for the newcomer
    with pytest.raises(B.KVError):
        B.evict_step(cache, q, kv_new, kv_new, 1, params, new_pos=20, stream=0)
    assert cache.n == 16
