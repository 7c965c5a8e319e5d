"""The C ABI on the host: the library loads, exports what include/catekv.h
declares, and rejects bad arguments before touching the GPU.  Head
classification is host-only and is checked against the oracle here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2608_30295_amd as ck
from paper_2608_30295_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "catekv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(_lib.LIB_PATH), reason="libcatekv.so not built")

FAKE = 0x100000   # a non-null pointer value; never dereferenced on these paths


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(catekv_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) == 17
    L = ck.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.SIGNATURES)


def test_version():
    assert b"gfx950" in ck.lib().catekv_version()


def _status_and_msg(rc):
    return rc, ck.lib().catekv_last_error().decode()


def test_decode_plan_rejects_bad_lengths():
    L = ck.lib()
    plan = _lib.DecodePlanT()
    ml = np.array([5, -1], dtype=np.int64)
    rc, msg = _status_and_msg(L.catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), 1, 8, 2, 0, ctypes.byref(plan),
                                                   FAKE, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG and "negative" in msg
    ml = np.array([5, 1 << 31], dtype=np.int64)
    rc, _ = _status_and_msg(L.catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), 1, 8, 2, 0, ctypes.byref(plan),
                                                 FAKE, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_UNSUPPORTED
    ml = np.array([5, 6], dtype=np.int64)
    rc, _ = _status_and_msg(L.catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), 1, 6, 2, 0, ctypes.byref(plan),
                                                 FAKE, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_UNSUPPORTED          # group size 3
    rc, msg = _status_and_msg(L.catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), 1, 8, 2, 0, ctypes.byref(plan),
                                                   FAKE, 16, None))
    assert rc == _lib.CATEKV_ERR_WORKSPACE
    rc, _ = _status_and_msg(L.catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), 1, 8, 2, 0, ctypes.byref(plan),
                                                 FAKE + 8, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_WORKSPACE           # misaligned


def test_decode_workspace_sizes():
    ml = np.array([131072] * 3 + [2112] * 5, dtype=np.int64)
    ws = ck.decode_workspace(ml, 32, 8)
    assert ws > 0
    assert ck.decode_workspace(ml, 32, 8, split_tokens=131072) < ws
    assert ck.decode_workspace(np.array([-1, 2], dtype=np.int64), 8, 2) == 0


def test_decode_attn_rejects_unplanned_use():
    L = ck.lib()
    plan = _lib.DecodePlanT()   # never filled: magic is 0
    rc, msg = _status_and_msg(L.catekv_decode_attn(1, ctypes.byref(plan), FAKE, FAKE, FAKE, 1, 32, 8, 128,
                                                   0.08, FAKE, None, FAKE, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG and "plan" in msg
    rc, _ = _status_and_msg(L.catekv_decode_attn(7, ctypes.byref(plan), FAKE, FAKE, FAKE, 1, 32, 8, 128,
                                                 0.08, FAKE, None, FAKE, 1 << 20, None))
    assert rc == _lib.CATEKV_ERR_UNSUPPORTED


def test_decode_attn_rejects_non_positive_scale():
    # the softmax needs scale > 0: a zero or negative scale is refused before any launch
    L = ck.lib()
    plan = _lib.DecodePlanT()
    ml = np.array([64, 64], dtype=np.int64)
    ws = np.zeros(1, dtype=np.uint8)
    assert L.catekv_decode_workspace(ml.ctypes.data_as(_lib.P_i64), 1, 8, 2, 0) > 0
    plan.magic = 0x43617465504c414e                    # a plan header as catekv_decode_plan fills it
    plan.batch, plan.hq, plan.hkv, plan.ws_bytes = 1, 8, 2, 1 << 20
    for scale in (0.0, -0.088, float("inf"), float("nan")):
        rc, msg = _status_and_msg(L.catekv_decode_attn(1, ctypes.byref(plan), FAKE, FAKE, FAKE, 1, 8, 2, 128,
                                                       scale, FAKE, None, FAKE, 1 << 20, None))
        assert rc == _lib.CATEKV_ERR_INVALID_ARG and "scale" in msg, scale
    del ws


# --------------------------------------------- retention budget (Algorithm 1, argtopk(C_chunk, n eta))

def _budget(n, l_obs, cs, eta):
    b = ctypes.c_int64(-7)
    rc = ck.lib().catekv_adaptive_budget(n, l_obs, cs, eta, ctypes.byref(b))
    return rc, b.value


def test_adaptive_budget_hand_values():
    # n - l_obs = 90 keys -> 12 chunks of 8 (the last one partial)
    assert [_budget(100, 10, 8, e) for e in (1.0, 0.5, 0.3, 0.25, 0.0)] == [(0, 12), (0, 6), (0, 4), (0, 3), (0, 0)]
    # 131072 - 64 keys -> 16376 chunks: the workloads' sweep
    assert [_budget(131072, 64, 8, e)[1] for e in (0.5, 0.25, 0.1)] == [8188, 4094, 1638]
    # eta is the decimal ratio: 10 chunks at 0.1, 0.3, 0.7 keep 1, 3, 7 (the
    # stored 0.1 lies above 1/10, the stored 0.3 and 0.7 below), and 0.55 keeps 6
    assert [_budget(88, 8, 8, e)[1] for e in (0.1, 0.3, 0.7, 0.5, 0.55)] == [1, 3, 7, 5, 6]
    # one chunk over an integer product stays exact for large counts
    assert _budget(8 * 1000003 + 8, 8, 8, 0.5)[1] == 500002
    assert ck.adaptive_budget(100, 10, 8, 0.3) == 4


def test_adaptive_budget_rejects_bad_arguments():
    for args in ((100, 10, 8, 1.5), (100, 10, 8, -0.1), (100, 10, 0, 0.5), (100, 100, 8, 0.5), (100, -1, 8, 0.5),
                 (100, 10, 8, float("nan"))):
        rc, b = _budget(*args)
        assert rc == _lib.CATEKV_ERR_INVALID_ARG and b == -7, args
    assert ck.lib().catekv_adaptive_budget(100, 10, 8, 0.5, None) == _lib.CATEKV_ERR_INVALID_ARG


def test_select_rejects_bad_arguments():
    L = ck.lib()
    heads = (ctypes.c_int32 * 2)(0, 1)
    dup = (ctypes.c_int32 * 2)(1, 1)
    bad = (ctypes.c_int32 * 1)(8)
    call = lambda **kw: L.catekv_select_critical(*[kw.get(k, v) for k, v in [
        ("dt", 1), ("q", FAKE), ("k", FAKE), ("hq", 32), ("hkv", 8), ("l_obs", 64), ("n", 4096), ("d", 128),
        ("cs", 8), ("heads", heads), ("n_sel", 2), ("b", 32), ("idx", FAKE), ("ws", FAKE), ("wsb", 1 << 30),
        ("s", None)]])
    assert call(d=64) == _lib.CATEKV_ERR_UNSUPPORTED
    assert call(l_obs=4096) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(l_obs=0) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(cs=0) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(b=0) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(heads=dup) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(heads=bad, n_sel=1) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(q=None) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(wsb=16) == _lib.CATEKV_ERR_WORKSPACE
    assert call(hq=30) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(l_obs=200) == _lib.CATEKV_ERR_UNSUPPORTED     # 4 * 200 rows
    assert ck.select_workspace(32, 8, 64, 4096, 8, 2) > 0


def test_select_noalloc_refuses_a_selection_beyond_its_scratch():
    # cs = 12 does not divide the 64-column tile, so the per-key column mass
    # is kept: 8 heads at 2^20 keys need more than the 16 MiB scratch
    L = ck.lib()
    assert ck.select_workspace(32, 8, 64, 1 << 20, 12, 8) > 16 << 20
    heads = (ctypes.c_int32 * 8)(*range(8))
    rc, msg = _status_and_msg(L.catekv_select_critical_noalloc(1, FAKE, FAKE, 32, 8, 64, 1 << 20, 128, 12, heads,
                                                               8, 64, FAKE, None))
    assert rc == _lib.CATEKV_ERR_UNSUPPORTED and "scratch" in msg
    rc, _ = _status_and_msg(L.catekv_select_critical_noalloc(1, FAKE, FAKE, 32, 8, 64, 4096, 128, 8, heads, 8, 0,
                                                             FAKE, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG                       # b = 0, as for the workspace call


def test_compact_rejects_bad_arguments():
    L = ck.lib()
    heads = (ctypes.c_int32 * 2)(0, 9)
    rc = L.catekv_compact_kv(1, FAKE, FAKE, 8, 4096, 128, 8, 64, heads, 2, FAKE, 32, FAKE, FAKE, FAKE, None)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG
    heads = (ctypes.c_int32 * 2)(0, 1)
    rc = L.catekv_compact_kv(1, FAKE, FAKE, 8, 4096, 128, 8, 4096, heads, 2, FAKE, 32, FAKE, FAKE, FAKE, None)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG
    rc = L.catekv_compact_kv(1, FAKE, FAKE, 8, 4096, 128, 8, 64, heads, 2, FAKE, 32, FAKE, FAKE, None, None)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG


def test_score_heads_rejects_bad_arguments():
    L = ck.lib()
    call = lambda **kw: L.catekv_score_heads(*[kw.get(k, v) for k, v in [
        ("dt", 1), ("q", FAKE), ("pos0", 4032), ("k", FAKE), ("hq", 32), ("hkv", 8), ("lq", 64), ("n", 4096),
        ("d", 128), ("li", 64), ("lr", 16), ("kp", 0.996), ("al", 1.0), ("causal", 1), ("cv", FAKE),
        ("ws", FAKE), ("wsb", 1 << 34), ("s", None)]])
    assert call(li=4000, lr=96) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(li=-1) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(kp=1.5) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(al=0.0) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(pos0=10) == _lib.CATEKV_ERR_INVALID_ARG        # row 0 would see no key
    assert call(lq=0) == _lib.CATEKV_ERR_INVALID_ARG
    assert call(wsb=100) == _lib.CATEKV_ERR_WORKSPACE
    assert call(dt=3) == _lib.CATEKV_ERR_UNSUPPORTED
    assert ck.score_heads_workspace(32, 8, 64, 4096, 64, 16) > 8 * 64 * 4016 * 4


# ------------------------------------------------------------ classification

@pytest.mark.parametrize("seed", range(12))
def test_classify_matches_oracle(seed):
    r_ = np.random.default_rng(seed)
    S, H = int(r_.integers(1, 6)), int(r_.integers(2, 33))
    cv = r_.random((S, H)).astype(np.float32)
    if seed % 3 == 0:
        cv = np.round(cv * 4) / 4          # ties
    for r in (0.25, 0.4, 0.5, 0.7):
        got = ck.classify_heads(cv, r)
        want = O.static_head_types(cv.astype(np.float64), r)
        assert got.tolist() == want.tolist()


def test_classify_counts_for_eight_heads():
    cv = np.arange(8, dtype=np.float32)[None] * 0.1
    for r, n in [(0.25, 6), (0.4, 5), (0.5, 4)]:
        assert ck.classify_heads(cv, r).sum() == n


def test_classify_rejects_bad_ratio():
    with pytest.raises(ck.CateKVError):
        ck.classify_heads(np.ones((1, 4), dtype=np.float32), 1.0)


def test_append_kv_rejects_bad_arguments():
    L = ck.lib()
    args = dict(kv=FAKE, cap=FAKE, lens=FAKE, k=FAKE, v=FAKE)

    def call(dtype=1, batch=1, hkv=2, d=128, **kw):
        a = {**args, **kw}
        return _status_and_msg(L.catekv_append_kv(dtype, a["kv"], a["cap"], a["lens"], a["k"], a["v"],
                                                  batch, hkv, d, None, None))

    rc, msg = call(lens=None)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG and "null" in msg
    rc, _ = call(batch=0)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG
    rc, _ = call(hkv=0)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG
    rc, msg = call(d=64)
    assert rc == _lib.CATEKV_ERR_INVALID_ARG and "d=64" in msg
    rc, _ = call(dtype=7)
    assert rc == _lib.CATEKV_ERR_UNSUPPORTED


def test_retrieval_rejects_bad_arguments():
    L = ck.lib()
    heads = (ctypes.c_int32 * 1)(0)
    rc, _ = _status_and_msg(L.catekv_page_bounds(1, FAKE, 2, 100, 128, 0, heads, 1, FAKE, FAKE, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG                       # cs = 0
    rc, _ = _status_and_msg(L.catekv_page_bounds(1, FAKE, 2, 0, 128, 8, heads, 1, FAKE, FAKE, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG                       # n = 0
    bad = (ctypes.c_int32 * 1)(5)
    rc, _ = _status_and_msg(L.catekv_page_bounds(1, FAKE, 2, 100, 128, 8, bad, 1, FAKE, FAKE, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG                       # head out of range
    need = L.catekv_retrieve_workspace(1, 13)
    assert need >= 13 * 4 and need % 256 == 0
    rc, _ = _status_and_msg(L.catekv_retrieve_pages(1, FAKE, FAKE, FAKE, 8, 2, 13, 128, heads, 1, 0, FAKE, FAKE,
                                                    need, None))
    assert rc == _lib.CATEKV_ERR_INVALID_ARG                       # n_keep = 0
    rc, _ = _status_and_msg(L.catekv_retrieve_pages(1, FAKE, FAKE, FAKE, 8, 2, 13, 128, heads, 1, 4, FAKE, FAKE,
                                                    need - 256, None))
    assert rc == _lib.CATEKV_ERR_WORKSPACE
