"""Seeded input generators for the five benchmark workloads.

Every tensor comes from its own counter-addressed NumPy stream,
``SeedSequence(seed, spawn_key=(tag, ...))`` with PCG64, so a tensor's bytes do
not depend on which other tensors were drawn or in which order.  Values are
drawn as float32 and, for bf16 workloads, rounded to bf16 with
round-to-nearest-even.  bf16 tensors are carried as ``uint16`` bit patterns.

The workloads mirror the attention shapes the paper evaluates on
(Llama-3-8B: 32 query heads, 8 KV heads, head dim 128; Section 4.1 and
Table 4), its context lengths (128K for RULER, 40K per sample for batched
throughput, 500K-1M single samples) and its selection hyperparameters
(observation window 64, chunk size 8, sparse budget 2048, initial and recent
exclusion of 1/32 and 1/128 of the budget, percentile 0.996 for Llama-3;
Appendix B.1).  The planted structure (aligned keys or scaled heavy-hitter
keys) stands in for the real prompts the paper uses, which are not available.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

# stream tags (first element of every spawn_key)
_TAG_LENGTHS = 1
_TAG_K = 2
_TAG_V = 3
_TAG_QOBS = 4
_TAG_QCAL = 5
_TAG_PLANT = 6
_TAG_DECODE = 7


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16.  NaN maps to the canonical quiet
    NaN; overflow rounds to +-inf as IEEE rounding prescribes.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    out = ((u + bias) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def storage_to_f64(arr: np.ndarray) -> np.ndarray:
    """Exact widening of a storage array (uint16 bf16 bits or float32) to float64."""
    if arr.dtype == np.uint16:
        return bf16_bits_to_f32(arr).astype(np.float64)
    if arr.dtype == np.float32:
        return arr.astype(np.float64)
    raise TypeError(f"unexpected storage dtype {arr.dtype}")


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, method knobs and input recipe."""

    name: str
    dtype: str                      # "f32" or "bf16": storage type of K, V and Q
    n: int                          # context length (single sequence) or max length
    batch: int = 1
    len_range: Optional[Tuple[int, int]] = None   # ragged batches: U[lo, hi] lengths
    hq: int = 32
    hkv: int = 8
    d: int = 128
    l_obs: int = 64                 # selection observation window (last prefill rows)
    budget: int = 2048              # consistent-head budget in tokens (chunks = budget / cs)
    cs: int = 8                     # chunk size
    r: float = 0.4                  # adaptive-head ratio
    k_pct: float = 0.996            # CV binarisation percentile
    alpha: float = 1.0              # CV threshold scale
    l_init: int = 64                # tokens excluded at the start for CV
    l_rec: int = 16                 # tokens excluded at the end for CV
    cv_calib_rows: int = 0          # >0: CV rows are fresh decode-time queries (positions >= n)
    plant: str = "heavy"            # "direction" or "heavy"
    n_plant: int = 16               # "direction": aligned keys per KV head
    heavy_frac: float = 0.01        # "heavy": fraction of positions with scaled keys
    heavy_scale: float = 3.0
    steps: int = 100                # decode steps in the benchmark loop
    seed: int = 20261

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def chunk_budget(self) -> int:
        return self.budget // self.cs

    @property
    def itemsize(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 4K context, fp32, aligned planted keys; the whole pipeline in one pass
    "ctx4k_f32": Workload(
        name="ctx4k_f32", dtype="f32", n=4096, l_obs=32, budget=256, r=0.5,
        l_init=8, l_rec=2, plant="direction", n_plant=16, steps=1, seed=20261),
    # 32K context, bf16, 1% heavy-hitter keys scaled by 3, 4 of 8 heads consistent
    "ctx32k_bf16": Workload(
        name="ctx32k_bf16", dtype="bf16", n=32768, l_obs=64, budget=1024, r=0.5,
        l_init=32, l_rec=8, steps=100, seed=20262),
    # 128K context, bf16, 5 of 8 heads consistent with budget 2048
    "ctx128k_bf16": Workload(
        name="ctx128k_bf16", dtype="bf16", n=131072, l_obs=64, budget=2048, r=0.4,
        l_init=64, l_rec=16, steps=100, seed=20263),
    # 16 ragged sequences of 16K-64K tokens, budget 1024 plus the 64-token window
    "batch16_ragged_bf16": Workload(
        name="batch16_ragged_bf16", dtype="bf16", n=65536, batch=16,
        len_range=(16384, 65536), l_obs=64, budget=1024, r=0.5,
        l_init=32, l_rec=8, steps=100, seed=20264),
    # 1M context, 6 of 8 heads consistent with budget 4096, CV on 32 decode queries
    "ctx1m_bf16": Workload(
        name="ctx1m_bf16", dtype="bf16", n=1048576, l_obs=64, budget=4096, r=0.25,
        l_init=128, l_rec=32, cv_calib_rows=32, steps=20, seed=20265),
}


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def _to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(dtype)


def sequence_lengths(wl: Workload) -> List[int]:
    """Context length of every sequence in the batch."""
    if wl.len_range is None:
        return [wl.n] * wl.batch
    lo, hi = wl.len_range
    r = _rng(wl.seed, _TAG_LENGTHS)
    return [int(x) for x in r.integers(lo, hi + 1, size=wl.batch)]


@dataclasses.dataclass
class SequenceInputs:
    """Prefill-time tensors of one sequence, in storage format."""

    n: int
    k: np.ndarray          # [Hkv][n][d]
    v: np.ndarray          # [Hkv][n][d]
    q_obs: np.ndarray      # [Hq][l_obs][d]  last l_obs prefill query rows
    q_cv: np.ndarray       # [Hq][Lcv][d]    rows the CV score observes
    q_cv_pos0: int         # absolute position of q_cv row 0
    planted: List[np.ndarray]  # per KV head: planted key positions


def make_sequence(wl: Workload, b: int = 0, n: Optional[int] = None) -> SequenceInputs:
    """Draw the prefill tensors of sequence ``b``.

    K, V and the window queries are i.i.d. N(0, 1).  Structure is then planted
    into K, per KV head:

    * ``"direction"``: ``n_plant`` positions in ``[0, n - l_obs)`` get
      ``4 * sqrt(d) * u_h`` added, where ``u_h`` is the unit mean direction of
      the group's window queries (keys pointing along the query direction).
    * ``"heavy"``: a ``heavy_frac`` fraction of positions are multiplied by
      ``heavy_scale`` (heavy-hitter tokens).
    """
    if n is None:
        n = sequence_lengths(wl)[b]
    hkv, hq, d, G = wl.hkv, wl.hq, wl.d, wl.group
    if n <= wl.l_obs:
        raise ValueError("context must exceed the observation window")
    q_obs32 = _rng(wl.seed, _TAG_QOBS, b).standard_normal((hq, wl.l_obs, d), dtype=np.float32)
    k_st = np.empty((hkv, n, d), dtype=np.float32 if wl.dtype == "f32" else np.uint16)
    v_st = np.empty_like(k_st)
    planted = []
    for h in range(hkv):
        kh = _rng(wl.seed, _TAG_K, b, h).standard_normal((n, d), dtype=np.float32)
        pr = _rng(wl.seed, _TAG_PLANT, b, h)
        if wl.plant == "direction":
            pos = np.sort(pr.choice(n - wl.l_obs, size=wl.n_plant, replace=False))
            u = q_obs32[h * G:(h + 1) * G].reshape(-1, d).astype(np.float64).mean(axis=0)
            u = (u / np.linalg.norm(u)).astype(np.float32)
            kh[pos] += np.float32(4.0 * np.sqrt(d)) * u
        elif wl.plant == "heavy":
            cnt = max(1, int(round(wl.heavy_frac * n)))
            pos = np.sort(pr.choice(n, size=cnt, replace=False))
            kh[pos] *= np.float32(wl.heavy_scale)
        else:
            raise ValueError(wl.plant)
        planted.append(pos)
        k_st[h] = _to_storage(kh, wl.dtype)
        del kh
        vh = _rng(wl.seed, _TAG_V, b, h).standard_normal((n, d), dtype=np.float32)
        v_st[h] = _to_storage(vh, wl.dtype)
        del vh
    if wl.cv_calib_rows > 0:
        q_cv32 = _rng(wl.seed, _TAG_QCAL, b).standard_normal(
            (hq, wl.cv_calib_rows, d), dtype=np.float32)
        q_cv_pos0 = n
    else:
        q_cv32 = q_obs32
        q_cv_pos0 = n - wl.l_obs
    return SequenceInputs(
        n=n, k=k_st, v=v_st,
        q_obs=_to_storage(q_obs32, wl.dtype),
        q_cv=_to_storage(q_cv32, wl.dtype),
        q_cv_pos0=q_cv_pos0, planted=planted)


def decode_queries(wl: Workload, step: int) -> np.ndarray:
    """Fresh N(0, 1) decode queries for one step: [batch][Hq][d] in storage format."""
    q = _rng(wl.seed, _TAG_DECODE, step).standard_normal((wl.batch, wl.hq, wl.d), dtype=np.float32)
    return _to_storage(q, wl.dtype)
