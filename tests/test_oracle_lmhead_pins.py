"""Pins of the oracle's LM-head weight gradient G = dY^T H (appendix "The LM
Head Factorizes Like the Embedding Table": G_i = sum_m (q_mi - 1[y_m = i]) h_m)
against facts that do not come from the oracle itself:

* brute force with exact rational arithmetic on tiny inputs;
* the appendix's target-count term: with q = 0, G_i = -(sum of h_m over the
  positions whose target is i), a plain segmented sum;
* a cross-entropy gradient has zero-sum rows (sum_i q_mi = 1), so every column
  of G sums to zero;
* one token: G is the outer product dY_0 h_0;
* single rounding to nearest-even at hand-picked bf16 boundaries;
* T = 0 gives zeros; swapping the operands transposes G; doubling H doubles G.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def bf16_bits(x) -> np.ndarray:
    """float values that are exact in bf16 -> their bit patterns."""
    a = np.asarray(x, dtype=np.float32)
    b = a.view(np.uint32)
    assert np.all((b & 0xFFFF) == 0), "value not exact in bf16"
    return (b >> 16).astype(np.uint16)


def bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def small_ints(rng, shape, lo=-3, hi=3):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("T,V,D,seed", [(1, 1, 1, 0), (3, 4, 5, 1), (7, 2, 9, 2), (5, 6, 3, 3)])
def test_brute_force_exact_rationals(T, V, D, seed):
    rng = np.random.default_rng(seed)
    # values k * 2^e: products and sums are exact, and |G| stays an integer
    # multiple of 2^-4 below 256, so G is exact in both output dtypes
    dY = small_ints(rng, (T, V)) * np.float32(0.25)
    H = small_ints(rng, (T, D)) * np.float32(0.25)
    want = [[sum(Fraction(float(dY[m, i])) * Fraction(float(H[m, j])) for m in range(T))
             for j in range(D)] for i in range(V)]
    for out in (np.float32, np.uint16):
        G = oracle.lmhead_grad(bf16_bits(dY), bf16_bits(H), out)
        got = G if out == np.float32 else bits_to_f64(G)
        for i in range(V):
            for j in range(D):
                assert Fraction(float(got[i, j])) == want[i][j], (out, i, j)


def test_target_count_term_is_a_segmented_sum():
    rng = np.random.default_rng(4)
    T, V, D = 40, 9, 6
    y = rng.integers(0, V, T)
    dY = np.zeros((T, V), np.float32)
    dY[np.arange(T), y] = -1.0
    H = small_ints(rng, (T, D), -8, 8)
    want = np.zeros((V, D))
    np.add.at(want, y, -H.astype(np.float64))
    G = oracle.lmhead_grad(bf16_bits(dY), bf16_bits(H), np.float32)
    assert np.array_equal(G.astype(np.float64), want)


def test_columns_of_a_cross_entropy_gradient_sum_to_zero():
    rng = np.random.default_rng(5)
    T, V, D = 12, 10, 7
    # q_m with exact binary fractions summing to 1, minus the one-hot target
    q = np.zeros((T, V), np.float32)
    for m in range(T):
        cuts = np.sort(rng.choice(np.arange(1, 16), size=3, replace=False))
        parts = np.diff(np.concatenate([[0], cuts, [16]])) / 16.0
        q[m, rng.choice(V, size=4, replace=False)] = parts
    y = rng.integers(0, V, T)
    dY = q.copy()
    dY[np.arange(T), y] -= 1.0
    assert np.all(dY.astype(np.float64).sum(axis=1) == 0.0)
    H = small_ints(rng, (T, D), -4, 4)
    G = oracle.lmhead_grad(bf16_bits(dY), bf16_bits(H), np.float32)
    assert np.all(G.astype(np.float64).sum(axis=0) == 0.0)
    assert np.any(G != 0.0)


def test_one_token_is_an_outer_product():
    rng = np.random.default_rng(6)
    V, D = 33, 17
    dY = (rng.standard_normal((1, V)) * 1e-2).astype(np.float32)
    H = rng.standard_normal((1, D)).astype(np.float32)
    dYb = (dY.view(np.uint32) >> 16).astype(np.uint16)   # truncate to bf16
    Hb = (H.view(np.uint32) >> 16).astype(np.uint16)
    want = np.outer(bits_to_f64(dYb)[0], bits_to_f64(Hb)[0])  # exact in float64
    G32 = oracle.lmhead_grad(dYb, Hb, np.float32)
    assert np.array_equal(G32, want.astype(np.float32))


@pytest.mark.parametrize("h1,want_bits", [
    (2.0 ** -8 + 2.0 ** -9, 0x3F81),   # 1 + 0.75 ulp -> up
    (2.0 ** -8, 0x3F80),               # exact tie, even neighbour below
    (2.0 ** -7 + 2.0 ** -8, 0x3F82),   # exact tie, even neighbour above
    (2.0 ** -9, 0x3F80),               # quarter ulp -> down
])
def test_single_round_to_nearest_even(h1, want_bits):
    # G = 1 * 1 + 1 * h1, exact in float64, one rounding to bf16
    dY = bf16_bits([[1.0], [1.0]])
    H = bf16_bits([[1.0], [h1]])
    G = oracle.lmhead_grad(dY, H, np.uint16)
    assert int(G[0, 0]) == want_bits


def test_no_tokens_transpose_and_scaling():
    rng = np.random.default_rng(7)
    T, V, D = 21, 13, 11
    dY = (rng.standard_normal((T, V)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    H = (rng.standard_normal((T, D)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert not oracle.lmhead_grad(dY[:0], H[:0], np.float32).any()
    G = oracle.lmhead_grad(dY, H, np.float32)
    Gt = oracle.lmhead_grad(H, dY, np.float32)
    assert np.array_equal(G, Gt.T)
    H2 = bf16_bits(bits_to_f64(H).astype(np.float32) * 2.0)
    assert np.array_equal(oracle.lmhead_grad(dY, H2, np.float32), 2.0 * G)
