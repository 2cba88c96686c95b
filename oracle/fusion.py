"""Float64 reference for the gated delta fusion of the hybrid drafter (test infrastructure).

Sec. 3.4.1 ("Gated Delta Rule"), Eqs. (delta) and (fusion), with the shapes of
App. B ("Shared gate"): for every draft token i with self-attention output n_i
and cross-attention output o_i (both in R^d),

    Delta_i = o_i - n_i
    g_i     = sigmoid(W_g [n_i; o_i; Delta_i] + b_g),   W_g in R^{d x 3d}, b_g in R^d
    h_i     = n_i + g_i (elementwise) W_Delta Delta_i,   W_Delta in R^{d x d}

Weights follow the usual linear-layer storage: row c of W_g holds the weights
of output channel c over the stacked input [n; o; Delta] (n-part first).

Cross-only variant (Sec. 3.4.2, "Cross-only"): the self-attention output is
removed from the forward pass; this oracle reads that as n_i = 0 everywhere
(so Delta_i = o_i), which is a reading, not a printed formula -- parity of the
cross-only variant is unpinned against the paper.

Pins (tests/test_oracle_fusion_pins.py): gate saturated shut reduces to n exactly;
gate saturated open with W_Delta = I gives o exactly; the block identity
W_g [n; o; o - n] = (A - C) n + (B + C) o; a unit Delta selects one column of
W_Delta; W_g = 0 gives the gate sigmoid(b_g) per channel.
"""
from __future__ import annotations

import numpy as np


def sigmoid(z: np.ndarray) -> np.ndarray:
    """Logistic function, evaluated without overflow for either sign of z."""
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def gated_delta_fusion(n: np.ndarray, o: np.ndarray, w_g: np.ndarray, b_g: np.ndarray, w_delta: np.ndarray,
                       cross_only: bool = False, return_gate: bool = False):
    """h (and optionally g) for every row of n / o, in float64.

    n, o: [tokens][d]; w_g: [d][3d]; b_g: [d]; w_delta: [d][d].
    """
    n = np.asarray(n, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    w_g = np.asarray(w_g, dtype=np.float64)
    b_g = np.asarray(b_g, dtype=np.float64)
    w_delta = np.asarray(w_delta, dtype=np.float64)
    tokens, d = o.shape
    assert n.shape == (tokens, d) and w_g.shape == (d, 3 * d) and b_g.shape == (d,) and w_delta.shape == (d, d)
    if cross_only:
        n = np.zeros_like(o)
    delta = o - n                                           # Eq. (delta)
    stacked = np.concatenate([n, o, delta], axis=1)         # [n_i; o_i; Delta_i]
    g = sigmoid(stacked @ w_g.T + b_g)                      # Eq. (fusion), gate
    h = n + g * (delta @ w_delta.T)                         # Eq. (fusion), output
    return (h, g) if return_gate else h
