"""Pins for the gated delta fusion oracle (Sec. 3.4.1, Eqs. (delta) and (fusion)).

Each test checks a closed form or an identity the definition implies, chosen so
that a slip in the oracle (wrong sign of Delta, wrong block order of
[n; o; Delta], transposed W_Delta, missing bias, gate applied to the wrong
term) fails at least one of them.
"""
import math

import numpy as np

from oracle.fusion import gated_delta_fusion, sigmoid


def data(tokens=5, d=6, seed=0, integer=False):
    rng = np.random.default_rng(seed)
    if integer:   # small integers: every sum and difference below is exact in float64
        n = rng.integers(-8, 9, (tokens, d)).astype(np.float64)
        o = rng.integers(-8, 9, (tokens, d)).astype(np.float64)
    else:
        n, o = rng.standard_normal((tokens, d)), rng.standard_normal((tokens, d))
    w_g = rng.standard_normal((d, 3 * d)) / math.sqrt(3 * d)
    b_g = rng.standard_normal(d)
    w_delta = rng.standard_normal((d, d)) / math.sqrt(d)
    return n, o, w_g, b_g, w_delta


def test_gate_shut_reduces_to_self_attention_output_exactly():
    # sigmoid(-1e4) underflows to 0 in float64, so h = n + 0 * (...) = n bit for bit
    n, o, w_g, _, w_delta = data()
    d = n.shape[1]
    h, g = gated_delta_fusion(n, o, np.zeros_like(w_g), np.full(d, -1e4), w_delta, return_gate=True)
    assert np.all(g == 0.0)
    assert np.array_equal(h, n)


def test_gate_open_with_identity_delta_projection_gives_cross_output_exactly():
    # g = 1 and W_Delta = I: h = n + (o - n) = o (exact for integer-valued inputs)
    n, o, w_g, _, _ = data(integer=True)
    d = n.shape[1]
    h, g = gated_delta_fusion(n, o, np.zeros_like(w_g), np.full(d, 1e4), np.eye(d), return_gate=True)
    assert np.all(g == 1.0)
    assert np.array_equal(h, o)


def test_unit_delta_selects_a_column_of_the_delta_projection():
    # Delta = e_k with the gate open: h - n = W_Delta e_k = column k (a transposed W_Delta gives row k)
    n, _, w_g, _, w_delta = data(tokens=1, d=7, integer=True, seed=3)
    d = n.shape[1]
    for k in range(d):
        o = n.copy()
        o[0, k] += 1.0
        h = gated_delta_fusion(n, o, np.zeros_like(w_g), np.full(d, 1e4), w_delta)
        np.testing.assert_allclose(h[0] - n[0], w_delta[:, k], rtol=0, atol=1e-15)


def test_gate_pre_activation_block_identity():
    # W_g [n; o; o - n] with W_g = [A | B | C] equals (A - C) n + (B + C) o: the same h with
    # W_g' = [A - C | B + C | 0].  A flipped Delta or a reordered stack breaks it.
    n, o, w_g, b_g, w_delta = data(tokens=4, d=5, seed=11)
    d = n.shape[1]
    A, B, C = w_g[:, :d], w_g[:, d:2 * d], w_g[:, 2 * d:]
    w_alt = np.concatenate([A - C, B + C, np.zeros_like(C)], axis=1)
    h1, g1 = gated_delta_fusion(n, o, w_g, b_g, w_delta, return_gate=True)
    h2, g2 = gated_delta_fusion(n, o, w_alt, b_g, w_delta, return_gate=True)
    np.testing.assert_allclose(g1, g2, rtol=0, atol=1e-13)
    np.testing.assert_allclose(h1, h2, rtol=0, atol=1e-13)


def test_each_block_of_the_gate_reads_its_own_input():
    # W_g = [s I | 0 | 0] opens the gate exactly where n > 0, [0 | s I | 0] where o > 0,
    # [0 | 0 | s I] where o - n > 0 (s large enough to saturate the sigmoid)
    n, o, _, _, w_delta = data(tokens=6, d=4, integer=True, seed=5)
    d = n.shape[1]
    o = np.where(o == n, o + 1, o)               # no zero Delta
    n = np.where(n == 0, 1.0, n)
    o = np.where(o == 0, 2.0, o)
    big = 1e4 * np.eye(d)
    zero = np.zeros((d, d))
    for block, ref in ((0, n), (1, o), (2, o - n)):
        w_g = np.concatenate([big if i == block else zero for i in range(3)], axis=1)
        _, g = gated_delta_fusion(n, o, w_g, np.zeros(d), w_delta, return_gate=True)
        assert np.array_equal(g, (ref > 0).astype(np.float64)), block


def test_bias_alone_sets_the_gate():
    # W_g = 0: g = sigmoid(b_g) per channel; sigmoid(0) = 1/2, sigmoid(+-ln 3) = 3/4, 1/4
    n, o, w_g, _, w_delta = data(tokens=3, d=3, seed=2)
    b = np.array([0.0, math.log(3.0), -math.log(3.0)])
    _, g = gated_delta_fusion(n, o, np.zeros_like(w_g), b, w_delta, return_gate=True)
    np.testing.assert_allclose(g, np.tile([0.5, 0.75, 0.25], (3, 1)), rtol=0, atol=1e-15)


def test_sigmoid_is_stable_and_symmetric():
    z = np.array([-800.0, -30.0, -1.0, 0.0, 1.0, 30.0, 800.0])
    s = sigmoid(z)
    assert np.all(np.isfinite(s)) and s[0] == 0.0 and s[-1] == 1.0 and s[3] == 0.5
    np.testing.assert_allclose(s + sigmoid(-z), 1.0, rtol=0, atol=1e-15)


def test_tokens_are_independent():
    # row i of h depends on row i of n and o only: permuting tokens permutes h
    n, o, w_g, b_g, w_delta = data(tokens=7, d=4, seed=9)
    perm = np.random.default_rng(1).permutation(7)
    h = gated_delta_fusion(n, o, w_g, b_g, w_delta)
    hp = gated_delta_fusion(n[perm], o[perm], w_g, b_g, w_delta)
    np.testing.assert_allclose(hp, h[perm], rtol=0, atol=1e-14)


def test_cross_only_with_open_gate_and_identity_returns_cross_output():
    # reading: the cross-only variant drops n (n = 0, so Delta = o); gate open, W_Delta = I gives o
    n, o, w_g, _, _ = data(integer=True, seed=4)
    d = n.shape[1]
    h = gated_delta_fusion(n, o, np.zeros_like(w_g), np.full(d, 1e4), np.eye(d), cross_only=True)
    assert np.array_equal(h, o)
