"""Helpers shared by the GPU tests: moving storage arrays to the device and
the parity comparisons (tolerances from the paper-path contract: bf16 inputs
with fp32 accumulation must match the fp64 oracle within max-abs 2e-3 and
relative L2 1e-3; fp32 inputs within 1e-5)."""
import numpy as np
import torch

import synth

DEV = "cuda:0"


def to_dev(st: np.ndarray) -> torch.Tensor:
    if st.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(st).view(np.int16)).to(DEV).view(torch.bfloat16)
    if st.dtype == np.float32:
        return torch.from_numpy(np.ascontiguousarray(st)).to(DEV)
    raise TypeError(st.dtype)


def to_host_storage(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


f64 = synth.storage_to_f64


def tolerances(dtype: str):
    return (2e-3, 1e-3) if dtype == "bf16" else (1e-5, 1e-5)


def assert_rows_close(got: np.ndarray, want: np.ndarray, dtype: str, what: str = ""):
    """Per output row (one query head): max-abs and relative L2 error."""
    max_abs, rel_l2 = tolerances(dtype)
    got = np.asarray(got, dtype=np.float64).reshape(-1, want.shape[-1])
    want = np.asarray(want, dtype=np.float64).reshape(-1, want.shape[-1])
    err = np.abs(got - want)
    worst = err.max(axis=1)
    rel = np.linalg.norm(got - want, axis=1) / np.maximum(np.linalg.norm(want, axis=1), 1e-30)
    zero = np.linalg.norm(want, axis=1) == 0
    rel[zero] = np.linalg.norm(got, axis=1)[zero]
    bad = np.nonzero((worst > max_abs) | (rel > rel_l2))[0]
    assert bad.size == 0, (f"{what}: {bad.size} rows out of tolerance; worst row {bad[0]} "
                           f"max-abs {worst[bad[0]]:.3e} rel-L2 {rel[bad[0]]:.3e}")
    return float(worst.max()), float(rel.max())


def check_topk(got: np.ndarray, scores: np.ndarray, b: int, rel_band: float = 1e-5):
    """GPU chunk selection against the oracle's chunk scores: bit-exact
    except for chunks whose score lies within rel_band of the k-th largest;
    ascending, -1 padded, right count."""
    nc = scores.shape[0]
    k = min(b, nc)
    got = np.asarray(got)
    assert (got[k:] == -1).all(), "padding"
    sel = got[:k]
    assert (np.diff(sel) > 0).all(), "not strictly ascending"
    assert sel.min() >= 0 and sel.max() < nc
    order = np.lexsort((np.arange(nc), -scores))
    kth = scores[order[k - 1]]
    band = np.abs(scores - kth) <= rel_band * abs(kth)
    must = set(np.nonzero((scores > kth) & ~band)[0].tolist())
    never = set(np.nonzero((scores < kth) & ~band)[0].tolist())
    s = set(sel.tolist())
    assert must <= s, f"missing {sorted(must - s)[:8]}"
    assert not (s & never), f"extra {sorted(s & never)[:8]}"
    exact = set(order[:k].tolist())
    return len(s ^ exact) // 2      # swaps inside the band
