"""Comparison rules between the GPU library and the oracle.

Kept and surviving token sets: identical except for tokens whose fp32 oracle
score lies within 1e-5 (relative) of the k-th (resp. n_surv-th) score of the
unit.  Kept keys: bit copies of the input rows.  Fused values: the oracle
re-fuses with the GPU's own kept / dropped sets (so a legitimate boundary swap
does not cascade), and the largest per-row error relative to that row's largest
magnitude must stay within 1e-4 (fp32 storage) or 2e-2 (bf16 storage).
"""
from __future__ import annotations

import numpy as np

BAND = 1e-5
TOL_FP32 = 1e-4
TOL_BF16 = 2e-2


def ranking(S32: np.ndarray) -> np.ndarray:
    """Token order: score descending, then index ascending."""
    return np.lexsort((np.arange(len(S32)), -S32.astype(np.float64)))


def check_sets(S32: np.ndarray, k: int, ns: int, kept: np.ndarray, drop: np.ndarray, what=""):
    """Returns the number of boundary swaps (all within the band)."""
    kept = np.asarray(kept, dtype=np.int64)
    drop = np.asarray(drop, dtype=np.int64)
    assert len(kept) == k, f"{what}: kept {len(kept)} != {k}"
    assert len(drop) == ns - k, f"{what}: dropped {len(drop)} != {ns - k}"
    assert np.all(np.diff(kept) > 0) and np.all(np.diff(drop) > 0), f"{what}: not ascending"
    assert not (set(kept.tolist()) & set(drop.tolist())), f"{what}: kept and dropped overlap"
    n = len(S32)
    assert np.all((kept >= 0) & (kept < n)) and np.all((drop >= 0) & (drop < n)), f"{what}: index range"
    order = ranking(S32)
    S = S32.astype(np.float64)
    swaps = 0
    for cut, got in ((k, set(kept.tolist())), (ns, set(kept.tolist()) | set(drop.tolist()))):
        if cut == 0:
            continue
        beta = S[order[cut - 1]]
        diff = got ^ set(order[:cut].tolist())
        bad = [v for v in diff if abs(S[v] - beta) > BAND * beta]
        assert not bad, (f"{what}: tokens {bad[:8]} differ at cut {cut} with scores "
                         f"{[float(S[v]) for v in bad[:4]]} vs boundary {beta}")
        swaps += len(diff) // 2
    return swaps


def fused_error(ref: np.ndarray, got: np.ndarray) -> float:
    """max over rows of ||got - ref||_inf / ||ref||_inf."""
    if ref.size == 0:
        return 0.0
    num = np.abs(got.astype(np.float64) - ref).max(axis=1)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return float((num / den).max())


def rel_err(ref: np.ndarray, got: np.ndarray, floor: float = 0.0) -> float:
    ref = ref.astype(np.float64)
    den = np.maximum(np.abs(ref), floor)
    den[den == 0] = 1.0
    return float((np.abs(got.astype(np.float64) - ref) / den).max()) if ref.size else 0.0
