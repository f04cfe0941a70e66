"""Pins for the layer-by-layer oracle (the unfused baseline's reference), all on the CPU.

Each check compares against something the oracle cannot agree with by construction: torch's
binary32 -> bfloat16 conversion, hand-worked rounding ties, exact integer arithmetic in Python,
closed forms of softmax on constant rows, scipy's logsumexp, Python's exactly rounded ``math.fsum``,
and the pinned naive oracle within the error bound of the three bfloat16 roundings. A missing or
doubled rounding, a transposed operand, a wrong mask alignment or a sign error fails one of them.
"""

import math
from fractions import Fraction

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import (lbl_error_bound, lbl_pv_head, lbl_scores_head, lbl_softmax_head, layer_by_layer_attention,
                    naive_attention, round_bf16)

RNG = np.random.default_rng(2024)


def is_bf16_value(y: np.ndarray) -> bool:
    """Every finite entry is exactly a bfloat16 value (binary32 with the low 16 bits zero)."""
    y = np.asarray(y, dtype=np.float64)
    f = y.astype(np.float32)
    return bool(np.array_equal(f.astype(np.float64), y) and not np.any(f.view(np.uint32) & 0xFFFF))


def bf16_rand(*shape, sigma=1.0):
    return torch.from_numpy(RNG.standard_normal(shape) * sigma).float().to(torch.bfloat16).double().numpy()


# ---------------------------------------------------------------------------------------------
# float64 -> bfloat16 rounding
# ---------------------------------------------------------------------------------------------

def test_round_bf16_matches_torch_on_binary32_values():
    # Random binary32 bit patterns over the whole finite range (normal and subnormal): for inputs
    # that are binary32 values, one correct rounding to bfloat16 is what torch's conversion does.
    bits = RNG.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x.copy()).to(torch.bfloat16).double().numpy()
    got = round_bf16(x.astype(np.float64))
    assert np.array_equal(got, want)


def test_round_bf16_ties_to_even():
    u = 2.0 ** -8
    cases = {
        1 + u: 1.0,                      # halfway between 1 and 1 + 2^-7: the even one is 1
        1 + 3 * u: 1 + 4 * u,            # halfway between 1 + 2^-7 (odd) and 1 + 2^-6 (even)
        -(1 + u): -1.0,
        2.0 ** -134: 0.0,                # half of the smallest subnormal 2^-133 rounds to 0
        3 * 2.0 ** -134: 2.0 ** -132,    # halfway between 2^-133 (odd) and 2^-132 (even)
        (2 - 2.0 ** -8) * 2.0 ** 127: math.inf,  # halfway between the largest finite and 2^128
        (2 - 2.0 ** -7) * 2.0 ** 127: (2 - 2.0 ** -7) * 2.0 ** 127,
    }
    for x, want in cases.items():
        assert round_bf16(np.array([x]))[0] == want, x


def test_round_bf16_rounds_once_not_through_binary32():
    # 1 + 2^-8 + 2^-40 lies just above a tie. Rounding to binary32 first would land exactly on the
    # tie and then go to 1.0; a single correct rounding goes up.
    eps = 2.0 ** -40
    x = np.array([1 + 2.0 ** -8 + eps, 1 + 2.0 ** -8 - eps, -(1 + 2.0 ** -8 + eps)])
    assert list(round_bf16(x)) == [1 + 2.0 ** -7, 1.0, -(1 + 2.0 ** -7)]


def test_round_bf16_is_nearest_on_random_float64():
    x = RNG.standard_normal(50_000) * np.exp2(RNG.integers(-30, 30, 50_000))
    y = round_bf16(x)
    assert is_bf16_value(y)
    # the neighbours of y one bfloat16 spacing away are never closer to x
    _, e = np.frexp(y)
    sp = np.ldexp(1.0, e - 8)
    assert np.all(np.abs(y - x) <= np.abs(y + sp - x)) and np.all(np.abs(y - x) <= np.abs(y - sp - x))
    assert np.all(np.abs(y - x) <= 2.0 ** -8 * np.abs(x))


# ---------------------------------------------------------------------------------------------
# score operator
# ---------------------------------------------------------------------------------------------

def test_scores_exact_on_integers():
    # Integer Q, K with |dot| <= 144 < 256 and scale 1/8: every score is exactly a bfloat16 value, so
    # the operator must return the exact products, checked against Python integer arithmetic.
    n, sk, d = 5, 7, 16
    q = RNG.integers(-3, 4, (n, d))
    k = RNG.integers(-3, 4, (sk, d))
    s = lbl_scores_head(q, k, 0.125)
    for i in range(n):
        for j in range(sk):
            assert s[i, j] == sum(int(q[i, t]) * int(k[j, t]) for t in range(d)) / 8
    assert s.shape == (n, sk)


def test_scores_are_correctly_rounded():
    # Scale 1/3: the exact score is a rational; the result is the bfloat16 value nearest to it.
    n, sk, d = 4, 6, 8
    q = RNG.integers(-9, 10, (n, d))
    k = RNG.integers(-9, 10, (sk, d))
    s = lbl_scores_head(q, k, 1.0 / 3.0)
    assert is_bf16_value(s)
    for i in range(n):
        for j in range(sk):
            exact = Fraction(sum(int(q[i, t]) * int(k[j, t]) for t in range(d))) * Fraction(1.0 / 3.0)
            err = abs(Fraction(s[i, j]) - exact)
            _, e = math.frexp(float(exact)) if exact else (0, -132)
            assert err <= Fraction(2) ** (e - 9)  # half a spacing


# ---------------------------------------------------------------------------------------------
# mask + softmax operator
# ---------------------------------------------------------------------------------------------

def test_softmax_constant_rows_closed_form():
    sk = 37
    s = np.full((3, sk), 0.75)
    g, lse = lbl_softmax_head(s, causal=False)
    assert np.all(g == round_bf16(np.array([1.0 / sk]))[0])
    assert np.allclose(lse, 0.75 + math.log(sk), rtol=0, atol=1e-14)


@pytest.mark.parametrize("sq,sk", [(6, 6), (4, 9), (9, 4)])
def test_softmax_causal_bottom_right(sq, sk):
    # Query i sees keys j <= i + (Sk - Sq): row i of a constant score matrix is bf16(1/c) on its
    # first c = clamp(i + 1 + Sk - Sq, 0, Sk) keys and 0 after; rows that see nothing give -inf.
    s = np.full((sq, sk), -1.5)
    g, lse = lbl_softmax_head(s, causal=True)
    for i in range(sq):
        c = min(sk, max(0, i + 1 + sk - sq))
        if c == 0:
            assert np.all(g[i] == 0) and lse[i] == -np.inf
            continue
        assert np.all(g[i, :c] == round_bf16(np.array([1.0 / c]))[0]) and np.all(g[i, c:] == 0)
        assert abs(lse[i] - (-1.5 + math.log(c))) < 1e-14


def test_softmax_matches_logsumexp_and_ratios():
    s = bf16_rand(8, 300, sigma=3.0)
    g, lse = lbl_softmax_head(s, causal=True, sq=8)
    for i in range(8):
        c = i + 1 + 300 - 8
        assert abs(lse[i] - logsumexp(s[i, :c])) < 1e-12
        assert np.all(g[i, c:] == 0)
        # each entry is the rounded exp(s - LSE): relative error at most 2^-8, never a sign slip
        p = np.exp(s[i, :c] - logsumexp(s[i, :c]))
        assert np.all(np.abs(g[i, :c] - p) <= 2.0 ** -8 * p)
    assert is_bf16_value(g)
    assert np.all(np.abs(g.sum(axis=1) - 1) <= 2.0 ** -8)


def test_softmax_shift_invariance():
    s = bf16_rand(5, 64)
    g0, l0 = lbl_softmax_head(s, causal=False)
    g1, l1 = lbl_softmax_head(s + 4.0, causal=False)
    assert np.allclose(l1, l0 + 4.0, rtol=0, atol=1e-12)
    # equal up to a flip of the last bit at a rounding tie
    assert np.all(np.abs(g1 - g0) <= 2.0 ** -7 * g0)


# ---------------------------------------------------------------------------------------------
# value operator
# ---------------------------------------------------------------------------------------------

def test_pv_one_hot_rows_copy_value_rows():
    sk, dv = 11, 16
    v = bf16_rand(sk, dv, sigma=2.0)
    pick = RNG.integers(0, sk, 6)
    g = np.zeros((6, sk))
    g[np.arange(6), pick] = 1.0
    assert np.array_equal(lbl_pv_head(g, v), v[pick])


def test_pv_correctly_rounded_against_fsum():
    g = round_bf16(RNG.random((4, 50)) / 50)
    v = bf16_rand(50, 8)
    o = lbl_pv_head(g, v)
    assert is_bf16_value(o)
    for i in range(4):
        for c in range(8):
            exact = math.fsum(float(g[i, j]) * float(v[j, c]) for j in range(50))
            assert abs(o[i, c] - exact) <= 2.0 ** -8 * abs(exact) + 1e-300


# ---------------------------------------------------------------------------------------------
# the three operators together
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("B,Hq,Hkv,Sq,Sk,d,causal,sigma", [
    (1, 2, 2, 40, 40, 16, False, 1.0),
    (2, 4, 2, 33, 70, 32, True, 1.0),
    (1, 3, 1, 50, 20, 24, True, 2.0),
    (1, 2, 1, 64, 64, 64, True, 3.0),
])
def test_layer_by_layer_within_rounding_bound_of_exact(B, Hq, Hkv, Sq, Sk, d, causal, sigma):
    q = bf16_rand(B, Hq, Sq, d, sigma=sigma)
    k = bf16_rand(B, Hkv, Sk, d, sigma=sigma)
    v = bf16_rand(B, Hkv, Sk, d, sigma=sigma)
    scale = 1 / math.sqrt(d)
    o, lse, s, g = layer_by_layer_attention(q, k, v, scale, causal, return_intermediates=True)
    o_ref, lse_ref = naive_attention(q, k, v, scale, causal)
    group = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            exact = scale * (q[b, h] @ k[b, h // group].T)
            vis = np.ones_like(exact, dtype=bool)
            if causal:
                vis = np.arange(Sk)[None, :] <= np.arange(Sq)[:, None] + (Sk - Sq)
            m = np.where(vis, np.abs(exact), 0).max(axis=1)
            bound = lbl_error_bound(m, np.abs(v[b, h // group]).max()) + 1e-12
            err = np.abs(o[b, h] - o_ref[b, h]).max(axis=1)
            assert np.all(err <= bound)
            fin = np.isfinite(lse_ref[b, h])
            assert np.array_equal(fin, np.isfinite(lse[b, h]))
            assert np.all(np.abs(lse[b, h][fin] - lse_ref[b, h][fin]) <= 2.0 ** -8 * m[fin] + 1e-12)
    # the roundings really happen: the result differs from exact attention, and S~, G, O are bf16
    assert np.abs(o - o_ref).max() > 0
    assert is_bf16_value(s) and is_bf16_value(g) and is_bf16_value(o)


def test_layer_by_layer_gqa_equals_replicated_heads():
    q = bf16_rand(1, 6, 20, 16)
    k = bf16_rand(1, 2, 30, 16)
    v = bf16_rand(1, 2, 30, 16)
    o1, l1 = layer_by_layer_attention(q, k, v, 0.25, True)
    o2, l2 = layer_by_layer_attention(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), 0.25, True)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
