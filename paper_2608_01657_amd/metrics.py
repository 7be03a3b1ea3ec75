"""Request-level metrics on the replay's per-request output (host side).

The paper scores a request by the fraction of its prompt tokens served from
the cache, and averages that over the victim's requests (attack traces) or
over all requests (benign traces); differences between policies come with
paired bootstrap confidence intervals over seeds (Sec. V-A).  The replay
reports, per request, the length h of the resident leading run of full
blocks, so a request's ratio is 16 h / prompt tokens.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np

BLOCK_TOKENS = 16


def hit_ratios(per_request: np.ndarray, lengths: np.ndarray) -> np.ndarray:
    """Per-request cached-token ratio: 16 * h / prompt length (0 for an empty
    prompt).  `per_request` is the [R, 4] (h, m, e, orphans) output."""
    h = np.asarray(per_request)[:, 0].astype(np.float64)
    L = np.asarray(lengths).astype(np.float64)
    out = np.zeros_like(h)
    nz = L > 0
    out[nz] = BLOCK_TOKENS * h[nz] / L[nz]
    return out


def mean_hit_ratio(per_request: np.ndarray, trace, group: Optional[int] = None) -> float:
    """Mean of the per-request ratios over the requests of `group` (all
    requests when None)."""
    r = hit_ratios(per_request, trace.length)
    if group is not None:
        r = r[np.asarray(trace.group) == group]
    return float(r.mean()) if r.size else 0.0


def paired_bootstrap(a: Sequence[float], b: Sequence[float], n_boot: int = 10000,
                     seed: int = 0, level: float = 0.95) -> Tuple[float, float, float]:
    """Mean of the paired differences a_i - b_i and its percentile bootstrap
    confidence interval (seeds resampled with replacement)."""
    d = np.asarray(a, np.float64) - np.asarray(b, np.float64)
    if d.size == 0:
        return 0.0, 0.0, 0.0
    rng = np.random.Generator(np.random.PCG64(seed))
    idx = rng.integers(0, d.size, size=(n_boot, d.size))
    means = d[idx].mean(axis=1)
    lo, hi = np.quantile(means, [(1 - level) / 2, 1 - (1 - level) / 2])
    return float(d.mean()), float(lo), float(hi)
