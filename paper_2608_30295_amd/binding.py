"""Python binding of the CateKV C ABI: argument marshalling only.

Every function takes torch tensors that live on the GPU, passes their device
pointers and the current HIP stream to ``libcatekv.so`` and returns torch
tensors.  No step of the method runs in Python or in torch.
"""
from __future__ import annotations

import ctypes
import math
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import _lib
from ._lib import check, lib

D = 128


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return _lib.CATEKV_BF16
    if t.dtype == torch.float32:
        return _lib.CATEKV_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _need_cuda(*ts: torch.Tensor) -> None:
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensor must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensor must be contiguous")


def _heads_arg(heads: Sequence[int]):
    arr = (ctypes.c_int32 * len(heads))(*[int(h) for h in heads])
    return arr


def workspace(nbytes: int, device) -> torch.Tensor:
    """A byte tensor usable as a library workspace (256-byte aligned)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- CV score

def score_heads_workspace(hq: int, hkv: int, lq: int, n: int, l_init: int, l_rec: int) -> int:
    return int(lib().catekv_score_heads_workspace(hq, hkv, lq, n, l_init, l_rec))


def score_heads(q_rows: torch.Tensor, k: torch.Tensor, *, q_pos0: int, l_init: int, l_rec: int,
                k_pct: float, alpha: float, causal: bool = True,
                ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """CV score per KV head (Eq. 1-4).  q_rows [Hq][Lq][d], k [Hkv][n][d] -> fp32 [Hkv]."""
    _need_cuda(q_rows, k)
    hq, lq, d = q_rows.shape
    hkv, n, _ = k.shape
    need = score_heads_workspace(hq, hkv, lq, n, l_init, l_rec)
    if ws is None:
        ws = workspace(need, k.device)
    out = torch.empty(hkv, dtype=torch.float32, device=k.device)
    check(lib().catekv_score_heads(_dtype_code(k), q_rows.data_ptr(), int(q_pos0), k.data_ptr(), hq, hkv, lq,
                                   n, d, int(l_init), int(l_rec), float(k_pct), float(alpha), int(bool(causal)),
                                   out.data_ptr(), ws.data_ptr(), ws.numel(), _stream(k.device)))
    return out


def classify_heads(cv: np.ndarray, r: float) -> np.ndarray:
    """Eq. 5 and static identification on the host.  cv [S][H] -> bool [H]."""
    cv = np.ascontiguousarray(np.atleast_2d(cv), dtype=np.float32)
    S, H = cv.shape
    out = np.zeros(H, dtype=np.uint8)
    check(lib().catekv_classify_heads(cv.ctypes.data_as(_lib.P_f32), S, H, float(r),
                                      out.ctypes.data_as(_lib.P_u8)))
    return out.astype(bool)


# -------------------------------------------------------------- selection

def select_workspace(hq: int, hkv: int, l_obs: int, n: int, cs: int, n_sel: int) -> int:
    return int(lib().catekv_select_workspace(hq, hkv, l_obs, n, cs, n_sel))


def select_critical(q_obs: torch.Tensor, k: torch.Tensor, heads: Sequence[int], cs: int, b: int,
                    ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Critical chunk indices (Algorithm 1).  q_obs [Hq][L_obs][d], k [Hkv][n][d] ->
    int32 [n_sel][b], ascending, -1 padded."""
    _need_cuda(q_obs, k)
    hq, l_obs, d = q_obs.shape
    hkv, n, _ = k.shape
    if ws is None:
        ws = workspace(select_workspace(hq, hkv, l_obs, n, cs, len(heads)), k.device)
    idx = torch.empty((len(heads), b), dtype=torch.int32, device=k.device)
    check(lib().catekv_select_critical(_dtype_code(k), q_obs.data_ptr(), k.data_ptr(), hq, hkv, l_obs, n, d, cs,
                                       _heads_arg(heads), len(heads), b, idx.data_ptr(), ws.data_ptr(),
                                       ws.numel(), _stream(k.device)))
    return idx


def compact_kv(k: torch.Tensor, v: torch.Tensor, heads: Sequence[int], idx: torch.Tensor, cs: int,
               l_obs: int, lens_out: torch.Tensor,
               out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Cache(K, V, i_k, L_obs): dense compact K/V [n_sel][b*cs + l_obs][d] per
    selected head; writes each head's length into lens_out[head] (int64)."""
    _need_cuda(k, v, idx, lens_out)
    hkv, n, d = k.shape
    n_sel, b = idx.shape
    cap = b * cs + l_obs
    if out is None:
        k_c = torch.empty((n_sel, cap, d), dtype=k.dtype, device=k.device)
        v_c = torch.empty_like(k_c)
    else:
        k_c, v_c = out
    if lens_out.dtype != torch.int64:
        raise TypeError("lens_out must be int64")
    check(lib().catekv_compact_kv(_dtype_code(k), k.data_ptr(), v.data_ptr(), hkv, n, d, cs, l_obs,
                                  _heads_arg(heads), n_sel, idx.data_ptr(), b, k_c.data_ptr(), v_c.data_ptr(),
                                  lens_out.data_ptr(), _stream(k.device)))
    return k_c, v_c


# ----------------------------------------------------------------- decode

@dataclass
class DecodePlan:
    plan: _lib.DecodePlanT
    ws: torch.Tensor
    batch: int
    hq: int
    hkv: int
    max_len: np.ndarray


def decode_workspace(max_len, hq: int, hkv: int, split_tokens: int = 0) -> int:
    ml = np.ascontiguousarray(max_len, dtype=np.int64).ravel()
    return int(lib().catekv_decode_workspace(ml.ctypes.data_as(_lib.P_i64), ml.size // hkv, hq, hkv,
                                             int(split_tokens)))


def decode_plan(max_len, hq: int, hkv: int, device, split_tokens: int = 0,
                ws: Optional[torch.Tensor] = None) -> DecodePlan:
    """Split-KV work list for upper-bound lengths max_len [B][Hkv] (blocking)."""
    ml = np.ascontiguousarray(max_len, dtype=np.int64).reshape(-1, hkv)
    B = ml.shape[0]
    need = int(lib().catekv_decode_workspace(ml.ctypes.data_as(_lib.P_i64), B, hq, hkv, int(split_tokens)))
    if need == 0:
        raise ValueError("invalid decode plan request")
    if ws is None:
        ws = workspace(need, device)
    plan = _lib.DecodePlanT()
    check(lib().catekv_decode_plan(ml.ctypes.data_as(_lib.P_i64), B, hq, hkv, int(split_tokens),
                                   ctypes.byref(plan), ws.data_ptr(), ws.numel(), _stream(ws.device)))
    return DecodePlan(plan, ws, B, hq, hkv, ml.copy())


def kv_table(pairs: Sequence[Tuple[int, int]], device) -> torch.Tensor:
    """Device array of catekv_kv_ptrs from (k_ptr, v_ptr) pairs, [B*Hkv] entries."""
    arr = torch.tensor([[int(a), int(b)] for a, b in pairs], dtype=torch.int64)
    return arr.to(device)


def decode_attn(plan: DecodePlan, q: torch.Tensor, kv: torch.Tensor, lens: torch.Tensor,
                scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                lse: Optional[torch.Tensor] = None, want_lse: bool = True):
    """One decode step.  q [B][Hq][d]; kv from kv_table; lens int64 [B][Hkv] on
    the GPU.  Returns (out fp32 [B][Hq][d], lse fp32 [B][Hq] or None)."""
    _need_cuda(q, kv, lens)
    B, hq, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty((B, hq, d), dtype=torch.float32, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, hq), dtype=torch.float32, device=q.device)
    check(lib().catekv_decode_attn(_dtype_code(q), ctypes.byref(plan.plan), q.data_ptr(), kv.data_ptr(),
                                   lens.data_ptr(), B, hq, plan.hkv, d, float(scale), out.data_ptr(),
                                   lse.data_ptr() if lse is not None else None, plan.ws.data_ptr(),
                                   plan.ws.numel(), _stream(q.device)))
    return out, lse


def append_kv(kv: torch.Tensor, capacity: torch.Tensor, lens: torch.Tensor, k_new: torch.Tensor,
              v_new: torch.Tensor, overflow: Optional[torch.Tensor] = None) -> None:
    """Appends the newest token's K/V rows to every view of the kv table and
    bumps lens on the device.  capacity, lens: int64 [B][Hkv] on the GPU;
    k_new, v_new [B][Hkv][d]; overflow: int32 [1] on the GPU (set to 1 when a
    view is full) or None."""
    _need_cuda(kv, capacity, lens, k_new, v_new)
    B, hkv, d = k_new.shape
    if v_new.shape != k_new.shape or v_new.dtype != k_new.dtype:
        raise ValueError("k_new and v_new must have the same shape and dtype")
    if capacity.numel() != B * hkv or lens.numel() != B * hkv or kv.shape[0] != B * hkv:
        raise ValueError("kv, capacity and lens must have B * Hkv entries")
    check(lib().catekv_append_kv(_dtype_code(k_new), kv.data_ptr(), capacity.data_ptr(), lens.data_ptr(),
                                 k_new.data_ptr(), v_new.data_ptr(), B, hkv, d,
                                 overflow.data_ptr() if overflow is not None else None,
                                 _stream(k_new.device)))


def adaptive_budget(n: int, l_obs: int, cs: int, eta: float) -> int:
    """Chunk budget of an adaptive head for retention ratio eta
    (catekv_adaptive_budget: Algorithm 1, argtopk(C_chunk, n eta) in chunks)."""
    b = ctypes.c_int64(0)
    check(lib().catekv_adaptive_budget(int(n), int(l_obs), int(cs), float(eta), ctypes.byref(b)))
    return int(b.value)


def page_bounds(k: torch.Tensor, heads: Sequence[int], cs: int) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-page key minima and maxima of the given KV heads (pages of cs rows):
    k [Hkv][n][d] -> (kmin, kmax) [n_sel][ceil(n / cs)][d] in k's dtype."""
    _need_cuda(k)
    hkv, n, d = k.shape
    heads = list(heads)
    n_pages = -(-n // cs)
    kmin = torch.empty((len(heads), n_pages, d), dtype=k.dtype, device=k.device)
    kmax = torch.empty_like(kmin)
    check(lib().catekv_page_bounds(_dtype_code(k), k.data_ptr(), hkv, n, d, cs, _heads_arg(heads), len(heads),
                                   kmin.data_ptr(), kmax.data_ptr(), _stream(k.device)))
    return kmin, kmax


def retrieve_pages(q: torch.Tensor, kmin: torch.Tensor, kmax: torch.Tensor, heads: Sequence[int], hkv: int,
                   n_keep: int, ws: Optional[torch.Tensor] = None,
                   out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Query-aware page retrieval for one step of one sequence: q [Hq][d];
    kmin/kmax from page_bounds for the same heads -> int32 [n_sel][n_keep]
    page indices, ascending, -1 padded."""
    _need_cuda(q, kmin, kmax)
    hq, d = q.shape
    heads = list(heads)
    n_sel, n_pages, _ = kmin.shape
    need = int(lib().catekv_retrieve_workspace(n_sel, n_pages))
    if ws is None:
        ws = workspace(need, q.device)
    if out is None:
        out = torch.empty((n_sel, n_keep), dtype=torch.int32, device=q.device)
    check(lib().catekv_retrieve_pages(_dtype_code(q), q.data_ptr(), kmin.data_ptr(), kmax.data_ptr(), hq, hkv,
                                      n_pages, d, _heads_arg(heads), n_sel, n_keep, out.data_ptr(), ws.data_ptr(),
                                      ws.numel(), _stream(q.device)))
    return out
