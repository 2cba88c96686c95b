"""Float64 reference for the drafting metrics (test infrastructure).

Sec. 3.1, "Metrics": step-wise draft acceptance rates alpha_k (k = 0 .. K - 1)
and the expected mean accepted tokens

    MAT = 1 + sum_{k=0}^{K-1} prod_{j=0}^{k} alpha_j ;

the KV-only tables add the long-range retention ratio alpha_6 / alpha_0.

Reading (m-a): alpha_k is the acceptance rate of draft step k among the
verifications whose steps 0 .. k - 1 were all accepted (a conditional rate), as
the product form of MAT implies: prod_{j<=k} alpha_j is then the probability
that at least k + 1 draft tokens are accepted, and MAT is one (the target's own
token) plus the expected number of accepted draft tokens.  From per-verification
accepted lengths a_i in 0 .. K:

    c_k     = #{ i : a_i >= k }            (c_0 = the number of verifications)
    alpha_k = c_{k+1} / c_k                (0 / 0 is taken as 0)

Pins (tests/test_oracle_metrics_pins.py): MAT from the paper's printed
step-wise rates reproduces the printed MAT of every row of the complete
acceptance-rate table, and the printed retention ratios, within the printing
precision; MAT from counts equals one plus the mean accepted length (a
telescoping identity, independent of the product form); a Markov chain with a
row's printed rates reproduces that row's MAT statistically.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def mat_from_alphas(alphas: Sequence[float]) -> float:
    """1 + sum_{k=0}^{K-1} prod_{j=0}^{k} alpha_j, the formula as printed."""
    total, prod = 1.0, 1.0
    for a in alphas:
        prod *= float(a)
        total += prod
    return total


def acceptance_counts(accepted: np.ndarray, K: int) -> np.ndarray:
    """c_k = #{i : accepted_i >= k} for k = 0 .. K (lengths clamped into [0, K])."""
    a = np.clip(np.asarray(accepted, dtype=np.int64), 0, K)
    return np.array([int(np.count_nonzero(a >= k)) for k in range(K + 1)], dtype=np.int64)


def acceptance_rates(counts: np.ndarray) -> np.ndarray:
    """alpha_k = c_{k+1} / c_k (0 when c_k = 0), k = 0 .. K - 1."""
    c = np.asarray(counts, dtype=np.float64)
    out = np.zeros(len(c) - 1)
    for k in range(len(c) - 1):
        out[k] = c[k + 1] / c[k] if c[k] > 0 else 0.0
    return out


def retention(alphas: Sequence[float], far: int = 6) -> float:
    """Long-range retention ratio alpha_far / alpha_0."""
    return float(alphas[far]) / float(alphas[0])
