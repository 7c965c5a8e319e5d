"""Plain CPU oracle for CateKV's hybrid-KV decode path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check in
``__graft_entry__`` and the benchmark's CPU-baseline leg use it.  It shares no
code, constants or helpers with the HIP library and imports nothing from it.

Everything is NumPy float64 on exactly-widened inputs (bf16 or fp32 values
are upcast without rounding).  Each function follows one passage of the paper
(CateKV, ICML 2025) and is written for readability, not speed: no blocking,
fusion or reordering beyond what the passage states.

Passages followed
-----------------
* Algorithm 1 (CateKV in an individual head), pre-filling stage:
  token criticality ``A = softmax(Q[-L_obs:] K[:-L_obs]^T / sqrt(d))``,
  ``C = sum_i A[i, :]``, ``BlockMax(C, cs)``, ``argtopk(C_chunk, b)`` and
  ``Cache(K, V, i_k, L_obs)``.
* Section 3.2, last paragraph: for GQA, ``A`` is the mean of the ``A`` of the
  query heads of a group.
* Algorithm 1, decoding stage: ``Attention(q, k, v)`` over the compact cache
  (consistent heads) or the retained cache (adaptive heads).
* Section 3.2, Eq. 1-4: observation matrix over keys
  ``[L_init, n - L_rec)``, percentile binarisation ``B = 1(A >= Phi(k, alpha))``,
  frequency vector ``C = sum_i B[i, :]`` and the coefficient-of-variation score.
* Section 3.2, Eq. 5 and the reference-based static identification paragraph:
  consistent iff ``S > Gamma(r)``; model-wise head types from the frequency
  with which a head is classified consistent across reference samples.
* Algorithm 1, adaptive branch: ``argtopk(C_chunk, n eta)`` (retention
  below 1) and ``Retrieval(q, cache_k, cache_v)``, "all or query-aware";
  Section 4 integrates page-based query-aware retrieval (Quest) in the
  adaptive heads.
* Figure 4 and its discussion: attention recall of the consistent,
  streaming, query-aware and top-k patterns under one sparse budget.

Readings where the paper is silent or ambiguous
-----------------------------------------------
* GQA groups are contiguous: query head ``g`` uses KV head ``g // G``.
* The softmax of Eq. 1 and of Algorithm 1 runs over the restricted key range
  only, as printed (not over the full causal row then sliced).
* Eq. 1 rows are prefill rows at absolute positions ``q_pos0 + i`` and see
  keys at positions ``<= q_pos0 + i`` (causal); decode-time calibration rows
  sit at positions ``>= n`` where the mask removes nothing.
* "k-th percentile element" is the linearly interpolated quantile
  (the common type-7 definition).
* The sums of Eq. 3 and Algorithm 1 run over all ``L_obs`` rows.
* Chunks are aligned at 0; a partial last chunk competes with the maximum of
  its valid tokens and contributes only those tokens.  Ties in the chunk
  top-k go to the lower chunk index; indices are returned ascending.  A
  budget above the number of chunks keeps every chunk.
* The chunk budget ``b`` counts chunks; the last ``L_obs`` tokens are kept on
  top of it.
* ``mu(C) = 0`` gives a score of 0.  Eq. 5 uses a strict ``>``.
* Static identification keeps as many heads as Eq. 5 marks consistent in a
  sample with distinct scores, ``H - 1 - floor((H - 1) r)``: the heads with
  the highest consistency frequency, ties broken by the higher mean score and
  then the lower head index.
* New tokens of the generation loop join every view, compact or full; the
  paper does not say where a token generated after prefill goes.
* ``argtopk(C_chunk, n eta)`` counts chunks: ``ceil(eta * ceil((n - L_obs) / cs))``.
* Query-aware retrieval uses chunks of cs rows as pages with per-page
  elementwise key minima and maxima (the Quest bound); with GQA a page's score
  is the largest bound over the group's query heads.
* Attention recall is the share of the full softmax mass of a decode query
  that falls on the kept rows; the streaming pattern keeps a few initial
  rows plus the most recent ones.

Parity status
-------------
Every function here is pinned by tests that do not re-type its formula
(closed forms, invariants, brute force, library routines and a hand-worked
example).  The readings above are pinned only by themselves: the paper
prints no worked example for them.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# shared small definitions
# --------------------------------------------------------------------------

def softmax_rows(S: np.ndarray, keep: np.ndarray | None = None) -> np.ndarray:
    """Row-wise softmax of a float64 matrix.  ``keep`` (bool, same shape)
    restricts each row to its kept entries; dropped entries get weight 0.
    A row with no kept entry is all zeros."""
    S = np.asarray(S, dtype=np.float64)
    if keep is None:
        keep = np.ones(S.shape, dtype=bool)
    Sm = np.where(keep, S, -np.inf)
    m = Sm.max(axis=1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(keep, np.exp(Sm - m), 0.0)
    z = e.sum(axis=1, keepdims=True)
    return np.divide(e, z, out=np.zeros_like(e), where=z > 0)


def quantile_type7(x: np.ndarray, p: float) -> float:
    """Linearly interpolated p-quantile of all entries of ``x``: with the
    values sorted ascending as x_(0..N-1) and h = (N - 1) p, the result is
    x_(floor h) + (h - floor h) (x_(floor h + 1) - x_(floor h))."""
    v = np.sort(np.asarray(x, dtype=np.float64).ravel())
    N = v.size
    if N == 0:
        raise ValueError("quantile of an empty array")
    h = (N - 1) * float(p)
    lo = int(math.floor(h))
    hi = min(lo + 1, N - 1)
    return float(v[lo] + (h - lo) * (v[hi] - v[lo]))


# --------------------------------------------------------------------------
# Algorithm 1, pre-filling stage: critical-token selection
# --------------------------------------------------------------------------

def selection_observation_matrix(q_win: np.ndarray, k_prefix: np.ndarray,
                                 scale: float) -> np.ndarray:
    """``A`` of Algorithm 1 for one KV head.

    q_win: [G][L_obs][d] window queries of the G query heads of the group.
    k_prefix: [n'][d], the keys before the window (``K[:-L_obs]``).
    Returns the group mean of the G softmax matrices, [L_obs][n'].
    """
    G = q_win.shape[0]
    A = np.zeros((q_win.shape[1], k_prefix.shape[0]), dtype=np.float64)
    for g in range(G):
        A += softmax_rows(q_win[g] @ k_prefix.T * scale)
    return A / G


def block_max(C: np.ndarray, cs: int) -> np.ndarray:
    """``BlockMax(C, cs)``: maximum of C over each chunk of cs tokens."""
    n = C.shape[0]
    nc = -(-n // cs)
    return np.array([C[c * cs:min((c + 1) * cs, n)].max() for c in range(nc)],
                    dtype=np.float64)


def argtopk_ascending(scores: np.ndarray, b: int) -> np.ndarray:
    """Indices of the b largest scores (ties to the lower index), ascending."""
    nc = scores.shape[0]
    b = min(int(b), nc)
    order = np.lexsort((np.arange(nc), -scores))
    return np.sort(order[:b]).astype(np.int64)


def chunk_scores(q_obs: np.ndarray, k: np.ndarray, h: int, G: int, l_obs: int,
                 cs: int, scale: float) -> np.ndarray:
    """``C_chunk`` of KV head h: window A, column sums, BlockMax."""
    n = k.shape[1]
    A = selection_observation_matrix(q_obs[h * G:(h + 1) * G], k[h, :n - l_obs], scale)
    C = A.sum(axis=0)
    return block_max(C, cs)


def select_critical(q_obs: np.ndarray, k: np.ndarray, heads: Sequence[int], cs: int,
                    b: int, scale: float | None = None) -> List[np.ndarray]:
    """Critical-chunk indices for the given KV heads (Algorithm 1).

    q_obs: [Hq][L_obs][d] last L_obs prefill query rows; k: [Hkv][n][d].
    Returns one ascending int64 index array per head in ``heads``.
    """
    Hq, l_obs, d = q_obs.shape
    Hkv = k.shape[0]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    return [argtopk_ascending(chunk_scores(q_obs, k, h, G, l_obs, cs, scale), b)
            for h in heads]


def compact_rows(n: int, l_obs: int, cs: int, idx: np.ndarray) -> np.ndarray:
    """Token positions kept by ``Cache(K, V, i_k, L_obs)``: the tokens of the
    selected chunks in ascending order, then the last L_obs tokens."""
    n_sel = n - l_obs
    parts = [np.arange(c * cs, min((c + 1) * cs, n_sel)) for c in idx]
    parts.append(np.arange(n - l_obs, n))
    return np.concatenate(parts).astype(np.int64)


def compact_kv(k: np.ndarray, v: np.ndarray, heads: Sequence[int], idx: Sequence[np.ndarray],
               cs: int, l_obs: int) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """Compact caches of the given heads: gathered K and V rows."""
    n = k.shape[1]
    kc, vc = [], []
    for h, ih in zip(heads, idx):
        rows = compact_rows(n, l_obs, cs, ih)
        kc.append(k[h][rows])
        vc.append(v[h][rows])
    return kc, vc


# --------------------------------------------------------------------------
# Algorithm 1, decoding stage
# --------------------------------------------------------------------------

def attention_decode(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     scale: float) -> Tuple[np.ndarray, float, np.ndarray]:
    """``Attention(q, k, v)`` for one query row.

    Returns (o [d], lse, w [L]) with w the softmax weights.  L = 0 gives
    o = 0, lse = -inf.
    """
    L = k.shape[0]
    if L == 0:
        return np.zeros(v.shape[1]), -math.inf, np.zeros(0)
    s = (k @ q) * scale
    M = s.max()
    e = np.exp(s - M)
    z = e.sum()
    return (e @ v) / z, float(M + math.log(z)), e / z


def decode_gqa(q: np.ndarray, views: Sequence[Tuple[np.ndarray, np.ndarray]],
               scale: float | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """One decode step of one sequence: q [Hq][d]; views[h] = (K_h, V_h) is the
    cache KV head h attends over (full for adaptive heads, compact for
    consistent heads).  Returns out [Hq][d] and lse [Hq]."""
    Hq, d = q.shape
    G = Hq // len(views)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((Hq, d))
    lse = np.zeros(Hq)
    for g in range(Hq):
        kh, vh = views[g // G]
        out[g], lse[g], _ = attention_decode(q[g], kh, vh, scale)
    return out, lse


def masked_attention_decode(q: np.ndarray, k: np.ndarray, v: np.ndarray, keep: np.ndarray,
                            scale: float) -> np.ndarray:
    """Attention of q over the full cache with dropped positions at -inf: the
    masked twin of compaction followed by decoding."""
    w = softmax_rows(((k @ q) * scale)[None, :], keep[None, :])[0]
    return w @ v


# --------------------------------------------------------------------------
# Section 3.2: CV head scoring and classification
# --------------------------------------------------------------------------

def cv_observation_matrix(q_rows: np.ndarray, k: np.ndarray, q_pos0: int, l_init: int,
                          l_rec: int, scale: float, causal: bool = True) -> np.ndarray:
    """Eq. 1 for one KV head, with the GQA group mean.

    q_rows: [G][Lq][d], row i at absolute position q_pos0 + i; k: [n][d].
    Keys [l_init, n - l_rec); key j (absolute l_init + j) is visible to row i
    when ``l_init + j <= q_pos0 + i`` or when ``causal`` is false.
    Returns [Lq][n - l_init - l_rec].
    """
    G, Lq, _ = q_rows.shape
    n = k.shape[0]
    kr = k[l_init:n - l_rec]
    keep = np.ones((Lq, kr.shape[0]), dtype=bool)
    if causal:
        key_pos = l_init + np.arange(kr.shape[0])
        row_pos = q_pos0 + np.arange(Lq)
        keep = key_pos[None, :] <= row_pos[:, None]
    A = np.zeros((Lq, kr.shape[0]))
    for g in range(G):
        A += softmax_rows(q_rows[g] @ kr.T * scale, keep)
    return A / G


def cv_from_observation(A: np.ndarray, k_pct: float, alpha: float) -> Tuple[float, np.ndarray, float]:
    """Eq. 2-4: binarise at Phi = alpha * Quantile_k(A), count per column and
    return (score, C, Phi)."""
    phi = alpha * quantile_type7(A, k_pct)
    B = (A >= phi)
    C = B.sum(axis=0).astype(np.int64)
    N = C.shape[0]
    mu = C.sum() / N
    if mu == 0:
        return 0.0, C, phi
    sigma = math.sqrt(((C - mu) ** 2).sum() / N)
    return float(sigma / mu), C, phi


def score_heads(q_rows: np.ndarray, q_pos0: int, k: np.ndarray, l_init: int, l_rec: int,
                k_pct: float, alpha: float, causal: bool = True,
                scale: float | None = None) -> np.ndarray:
    """CV score of every KV head.  q_rows: [Hq][Lq][d]; k: [Hkv][n][d]."""
    Hq, _, d = q_rows.shape
    Hkv = k.shape[0]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros(Hkv)
    for h in range(Hkv):
        A = cv_observation_matrix(q_rows[h * G:(h + 1) * G], k[h], q_pos0, l_init, l_rec,
                                  scale, causal)
        out[h] = cv_from_observation(A, k_pct, alpha)[0]
    return out


def classify_sample(scores: np.ndarray, r: float) -> np.ndarray:
    """Eq. 5 for one sample: consistent iff S > Gamma(r), Gamma(r) being the
    r-quantile of the sample's head scores."""
    s = np.asarray(scores, dtype=np.float64).ravel()
    return s > quantile_type7(s, r)


def static_head_types(scores: np.ndarray, r: float) -> np.ndarray:
    """Reference-based static identification over S samples.

    scores: [S][H].  Each sample is classified by Eq. 5; a head's frequency is
    the fraction of samples in which it is consistent.  The model-wise
    consistent set holds as many heads as Eq. 5 marks consistent in one
    sample whose scores all differ, ``H - 1 - floor((H - 1) r)`` (5 of 8 at
    r = 0.3 and at r = 0.4, 6 of 8 at r = 0.25): the most frequent heads, ties broken by the
    higher mean score, then the lower index.  Returns bool [H].
    """
    sc = np.atleast_2d(np.asarray(scores, dtype=np.float64))
    S, H = sc.shape
    freq = np.mean([classify_sample(sc[s], r) for s in range(S)], axis=0)
    mean = sc.mean(axis=0)
    order = np.lexsort((np.arange(H), -mean, -freq))
    n_cons = H - 1 - int(math.floor((H - 1) * float(r)))
    out = np.zeros(H, dtype=bool)
    out[order[:n_cons]] = True
    return out


# --------------------------------------------------------------------------
# Around Algorithm 1's decoding stage: the generation loop, adaptive
# retention below 1, query-aware retrieval in adaptive heads (the
# "CateKV + Quest" integration of Section 4) and the attention-recall
# comparison of Figure 4.
# --------------------------------------------------------------------------

def append_token(k_view: np.ndarray, v_view: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
                 capacity: int) -> Tuple[np.ndarray, np.ndarray, bool]:
    """One generated token joins a cache view (compact or full alike) while
    the view holds fewer than ``capacity`` rows.  Returns (k, v, appended)."""
    if k_view.shape[0] >= capacity:
        return k_view, v_view, False
    return (np.concatenate([k_view, k_new[None, :]]), np.concatenate([v_view, v_new[None, :]]), True)


def adaptive_budget(n: int, l_obs: int, cs: int, eta: float) -> int:
    """Chunk budget of an adaptive head, ``argtopk(C_chunk, n eta)`` of
    Algorithm 1 read as a chunk count: ``ceil(eta * ceil((n - l_obs) / cs))``.
    eta = 1 keeps every chunk (the whole cache)."""
    nc = -(-(n - l_obs) // cs)
    return int(math.ceil(eta * nc - 1e-12))


def page_bounds(k: np.ndarray, cs: int) -> Tuple[np.ndarray, np.ndarray]:
    """Per chunk of cs rows (aligned at 0, last one partial): elementwise
    minimum and maximum of the keys, the page metadata of query-aware
    retrieval."""
    n, d = k.shape
    nc = -(-n // cs)
    kmin = np.zeros((nc, d))
    kmax = np.zeros((nc, d))
    for c in range(nc):
        rows = k[c * cs:min((c + 1) * cs, n)]
        kmin[c] = rows.min(axis=0)
        kmax[c] = rows.max(axis=0)
    return kmin, kmax


def page_scores(q_group: np.ndarray, kmin: np.ndarray, kmax: np.ndarray) -> np.ndarray:
    """Upper bound of q . k over each page, ``sum_d max(q_d kmin_d, q_d kmax_d)``,
    for each query head of the group; a page's score is the largest bound
    over the group's heads (it may matter to any of them)."""
    best = np.full(kmin.shape[0], -np.inf)
    for q in q_group:
        ub = np.maximum(kmin * q[None, :], kmax * q[None, :]).sum(axis=1)
        best = np.maximum(best, ub)
    return best


def retrieve_pages(q_group: np.ndarray, k: np.ndarray, cs: int, n_pages: int) -> np.ndarray:
    """The n_pages pages with the highest scores (ties to the lower index),
    ascending: the query-aware Retrieval(q, cache_k, cache_v) of an adaptive
    head."""
    kmin, kmax = page_bounds(k, cs)
    return argtopk_ascending(page_scores(q_group, kmin, kmax), n_pages)


def attention_recall(q: np.ndarray, k: np.ndarray, keep: np.ndarray, scale: float) -> float:
    """Share of the full attention mass of query q that falls on the kept
    rows."""
    w = softmax_rows(((k @ q) * scale)[None, :])[0]
    return float(w[np.asarray(keep, dtype=np.int64)].sum())


def streaming_keep(n: int, budget: int, n_sink: int) -> np.ndarray:
    """Rows of the streaming pattern: the first n_sink rows and the most
    recent ones, budget rows in all."""
    if budget >= n:
        return np.arange(n)
    return np.concatenate([np.arange(min(n_sink, budget)), np.arange(n - (budget - min(n_sink, budget)), n)])


def topk_keep(q: np.ndarray, k: np.ndarray, budget: int, scale: float) -> np.ndarray:
    """Rows of the upper-bound pattern: the budget rows with the largest
    attention weights for this query."""
    s = (k @ q) * scale
    order = np.lexsort((np.arange(s.shape[0]), -s))
    return np.sort(order[:min(budget, s.shape[0])])


def chunk_rows(n: int, cs: int, pages: np.ndarray) -> np.ndarray:
    """Rows of the given chunks, ascending."""
    pages = np.sort(np.asarray(pages, dtype=np.int64))
    return np.concatenate([np.arange(c * cs, min((c + 1) * cs, n)) for c in pages]) if pages.size else \
        np.zeros(0, dtype=np.int64)
