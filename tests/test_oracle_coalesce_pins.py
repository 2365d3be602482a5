"""Pins of the oracle's gradient coalescing (token ids + per-position gradient
rows -> distinct ids and summed rows), against what the paper and arithmetic
fix rather than against itself:

* numpy brute force (np.unique for the ids, np.add.at in float64 for the sums,
  which visits positions in ascending order) on random shapes, fp32 and bf16;
* the coherent-signal limit of the appendix "The Fisher is Proportional to
  Inverse Frequency Squared": if every occurrence of token i carries the same
  vector mu_i, row i is K_i mu_i, K_i the count of token i;
* conservation: the rows sum to the sum of all positions (exact data);
* independence of the position order whenever the sums are exact;
* the summation order itself (ascending positions, float64), with data whose
  float64 sum depends on the order;
* one rounding from float64 to bf16 (a sum just above a bf16 tie rounds up,
  which a detour through fp32 would not);
* index errors and the empty batch.
"""
import numpy as np
import pytest

import oracle


def _bf16_bits_from_f64(x: np.ndarray) -> np.ndarray:
    return np.array([oracle.f64_to_bf16(float(v)) for v in x.ravel()], np.uint16).reshape(x.shape)


def _bf16_values(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _brute(tok, U64):
    ids = np.unique(tok)
    acc = np.zeros((ids.size, U64.shape[1]), np.float64)
    np.add.at(acc, np.searchsorted(ids, tok), U64)
    return ids, acc


@pytest.mark.parametrize("P,V,D,seed", [(1, 1, 1, 0), (7, 3, 5, 1), (200, 50, 33, 2), (1000, 4000, 64, 3),
                                        (513, 17, 130, 4)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_coalesce_matches_numpy_brute_force(P, V, D, seed, dtype):
    rng = np.random.default_rng(seed)
    tok = rng.integers(0, V, P)
    x = rng.standard_normal((P, D)) * 10.0 ** rng.uniform(-6, 2, (P, 1))
    if dtype == "f32":
        U = x.astype(np.float32)
        U64 = U.astype(np.float64)
    else:
        U = _bf16_bits_from_f64(x)
        U64 = _bf16_values(U)
    st, idx, G = oracle.coalesce(tok, U, V)
    assert st == oracle.OK
    ids, acc = _brute(tok, U64)
    assert np.array_equal(idx, ids)
    if dtype == "f32":
        assert np.array_equal(G.view(np.uint32), acc.astype(np.float32).view(np.uint32))
    else:
        assert np.array_equal(G, _bf16_bits_from_f64(acc))


def test_coherent_signal_rows_are_count_times_signal():
    rng = np.random.default_rng(5)
    V, D, P = 40, 12, 600
    p = 1.0 / np.arange(1, V + 1) ** 1.1
    tok = rng.choice(V, P, p=p / p.sum())
    mu = rng.integers(-64, 64, (V, D)).astype(np.float32) / 8.0   # exact in bf16 and fp32
    U = mu[tok]
    st, idx, G = oracle.coalesce(tok, U, V)
    assert st == oracle.OK
    K = np.bincount(tok, minlength=V)
    assert np.array_equal(idx, np.nonzero(K)[0])
    assert np.array_equal(G, K[idx, None].astype(np.float32) * mu[idx])


def test_rows_conserve_the_total_and_ignore_position_order_when_exact():
    rng = np.random.default_rng(6)
    V, D, P = 30, 9, 400
    tok = rng.integers(0, V, P)
    U = rng.integers(-1000, 1000, (P, D)).astype(np.float32)
    st, idx, G = oracle.coalesce(tok, U, V)
    assert st == oracle.OK
    assert np.array_equal(G.sum(axis=0, dtype=np.float64), U.sum(axis=0, dtype=np.float64))
    perm = rng.permutation(P)
    st, idx2, G2 = oracle.coalesce(tok[perm], U[perm], V)
    assert np.array_equal(idx2, idx) and np.array_equal(G2, G)


def test_summation_visits_positions_in_ascending_order():
    big = np.float32(2.0 ** 60)
    # float64: (2^60 + 1) rounds back to 2^60, so the order decides the result
    tok = np.array([4, 4, 4])
    st, _, G = oracle.coalesce(tok, np.array([[big], [1.0], [-big]], np.float32), 5)
    assert st == oracle.OK and G[0, 0] == 0.0
    st, _, G = oracle.coalesce(tok, np.array([[big], [-big], [1.0]], np.float32), 5)
    assert st == oracle.OK and G[0, 0] == 1.0
    # other tokens interleaved between them change nothing
    tok = np.array([4, 1, 4, 2, 4])
    U = np.array([[big], [7.0], [1.0], [9.0], [-big]], np.float32)
    st, idx, G = oracle.coalesce(tok, U, 5)
    assert st == oracle.OK and idx.tolist() == [1, 2, 4] and G[:, 0].tolist() == [7.0, 9.0, 0.0]


def test_bf16_output_is_rounded_once_from_float64():
    tie = np.float32(2.0 ** -8)    # 1 + 2^-8 is halfway between bf16 1 and 1 + 2^-7
    above = np.float32(2.0 ** -30)
    tok = np.array([0, 0])
    st, _, G = oracle.coalesce(tok, np.array([[1.0], [tie]], np.float32), 1, out_dtype=np.uint16)
    assert st == oracle.OK and G[0, 0] == 0x3F80          # tie -> even
    tok = np.array([0, 0, 0])
    st, _, G = oracle.coalesce(tok, np.array([[1.0], [tie], [above]], np.float32), 1, out_dtype=np.uint16)
    # the exact sum is just above the tie: one rounding goes up (an fp32 detour
    # would first round it onto the tie and then down to 1.0)
    assert st == oracle.OK and G[0, 0] == 0x3F81
    assert np.float32(np.float64(1.0) + 2.0 ** -8 + 2.0 ** -30) == np.float32(1.0 + 2.0 ** -8)


# (rows of one id, as bf16 bits; the bf16 bits of their once-rounded sum),
# every expected value derived by hand from the bf16 grid
BF16_EDGE_SEGMENTS = [
    ([0x3F80, 0x3B80, 0x3080], 0x3F81),   # 1 + 2^-8 + 2^-30: just above the 1 / 1+2^-7 midpoint -> up
    ([0x3F80, 0x3B80, 0xB080], 0x3F80),   # 1 + 2^-8 - 2^-30: just below it -> down
    ([0x3F80, 0x3B80], 0x3F80),           # the midpoint itself -> the even neighbour 1
    ([0x3F81, 0x3B80], 0x3F82),           # 1 + 2^-7 + 2^-8: midpoint, even neighbour above
    ([0xBF80, 0xBB80, 0xB080], 0xBF81),   # the first three mirrored
    ([0xBF80, 0xBB80, 0x3080], 0xBF80),
    ([0x7F7F, 0x7F7F], 0x7F80),           # 2 x the largest finite value -> +inf
    ([0x7F7F, 0x7B00], 0x7F80),           # largest + half its spacing: a tie, even side is 2^128 -> +inf
    ([0x8000], 0x0000),                   # a row of -0 alone: 0 + (-0) = +0
    ([0x7F80], 0x7F80),                   # +inf alone
    ([0x0001], 0x0001),                   # the smallest subnormal alone
    ([0xFF7F], 0xFF7F),                   # the most negative finite value alone
    ([0x0001, 0x0001], 0x0002),           # subnormals add exactly
]


@pytest.mark.parametrize("rows,want", BF16_EDGE_SEGMENTS)
def test_bf16_edge_segments_round_once(rows, want):
    tok = np.zeros(len(rows), np.int64)
    U = np.array(rows, np.uint16).reshape(-1, 1)
    st, _, G = oracle.coalesce(tok, U, 1, out_dtype=np.uint16)
    assert st == oracle.OK and int(G[0, 0]) == want


def test_index_errors_and_empty_batch():
    U = np.ones((3, 2), np.float32)
    for bad in ([0, 5, 1], [0, -1, 1]):
        st, idx, G = oracle.coalesce(np.array(bad), U, 5)
        assert st == oracle.BAD_INDEX and idx is None
    st, idx, G = oracle.coalesce(np.zeros(0, np.int64), np.zeros((0, 2), np.float32), 5)
    assert st == oracle.OK and idx.size == 0 and G.shape == (0, 2)
