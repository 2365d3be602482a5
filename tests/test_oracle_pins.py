"""Pins for the CPU oracle: each checks it against something other than itself.

The paper prints no worked numeric example of the update, so the anchors are a
hand-derived 2 x 2 example (tests/golden/ember_2x2_worked.txt), identities the
paper proves (the normaliser identity and rank-1 exactness of the appendix
"Outer Product Unit Alignment"), special cases that reduce to a library
routine (torch's Adam with beta1 = 0), brute force with numpy, bitwise
invariants, and the state sizes the paper prints (Table "model scaling").
"""
import bisect
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
B2_F32 = float(np.float32(0.999))


def _golden_2x2():
    vals = {}
    with open(os.path.join(GOLDEN, "ember_2x2_worked.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = (s.strip() for s in line.split("=", 1))
            vals[k] = [Fraction(x.strip()) for x in v.split(",")]
    return vals


def _f32(rows):
    return np.array(rows, dtype=np.float32)


def _zero_state(V, D):
    return np.zeros(V, np.float32), np.zeros(D, np.float32)


# ---------------------------------------------------------------------------
# bf16 storage rounding (the oracle's W store for bf16 tables)
# ---------------------------------------------------------------------------

def _all_positive_bf16():
    bits = np.arange(0, 0x7F80, dtype=np.uint32)           # +0 .. max finite
    vals = (bits << 16).view(np.float32).astype(np.float64)
    return list(vals), list(bits)


_BF16_VALS, _BF16_BITS = _all_positive_bf16()


def _bf16_rne_exact(x: float) -> int:
    """Nearest bf16 by exact search over every bf16 value; ties to even bits."""
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    ax = abs(x)
    vals = _BF16_VALS + [2.0 ** 128]            # 2^128 stands for overflow to inf
    bits = _BF16_BITS + [0x7F80]
    if ax >= vals[-1]:
        return sign | 0x7F80
    k = bisect.bisect_right(vals, ax) - 1
    if vals[k] == ax:
        return sign | bits[k]
    lo, hi = Fraction(vals[k]), Fraction(vals[k + 1])
    fx = Fraction(ax)
    dl, dh = fx - lo, hi - fx
    if dl < dh or (dl == dh and bits[k] % 2 == 0):
        return sign | bits[k]
    return sign | bits[k + 1]


def test_bf16_rounding_matches_exact_nearest_even():
    rng = np.random.default_rng(7)
    xs = list(rng.standard_normal(3000) * 10.0 ** rng.uniform(-40, 38, 3000))
    # exact midpoints between neighbouring bf16 values (ties), and their neighbours
    for b in rng.integers(1, 0x7F7F, 400):
        lo = float(np.uint32(b << 16).view(np.float32))
        hi = float(np.uint32((b + 1) << 16).view(np.float32))
        mid = (lo + hi) / 2
        xs += [mid, np.nextafter(mid, 0), np.nextafter(mid, np.inf), -mid]
    xs += [0.0, -0.0, 1e-45, 2.0 ** -134, 2.0 ** -133, 3 * 2.0 ** -134, 2.0 ** -126,
           3.3895313892515355e38, 3.3961775292304957e38, 3.4e38, 1e39, -1e39]
    for x in xs:
        assert oracle.f64_to_bf16(float(x)) == _bf16_rne_exact(float(x)), x
    assert oracle.f64_to_bf16(float("inf")) == 0x7F80
    assert oracle.f64_to_bf16(float("-inf")) == 0xFF80
    assert (oracle.f64_to_bf16(float("nan")) & 0x7FFF) > 0x7F80


def test_bf16_decode_is_exact():
    for b in [0x0000, 0x8000, 0x3F80, 0xBF80, 0x0001, 0x7F7F, 0x4049]:
        assert oracle.bf16_to_f64(b) == float(np.uint32(b << 16).view(np.float32))


# ---------------------------------------------------------------------------
# Hand-worked 2 x 2 example (Algorithm 1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("eps", [0.0, 1e-8])
def test_worked_2x2_two_steps(eps):
    gd = _golden_2x2()
    beta2 = float(gd["beta2"][0])
    lr = 1e-3
    r, c = _zero_state(2, 2)
    for t, gkey, rkey, ckey, zkey in ((1, "G1", "r1", "c1", "z2sq1"),
                                     (2, "G2", "r2", "c2", "z2sq2")):
        G = _f32(np.array([float(x) for x in gd[gkey]]).reshape(2, 2))
        W = np.zeros((2, 2), np.float32)
        assert oracle.step(W, G, r, c, t, lr=lr, beta2=beta2, eps=eps, maximize=True) == 0
        # state is dyadic -> exact in fp32
        assert r.tolist() == [float(x) for x in gd[rkey]]
        assert c.tolist() == [float(x) for x in gd[ckey]]
        # update: |u| / alpha = |g| / (sqrt(vtil) + eps), vtil from the hand derivation
        for k in range(4):
            g = float(gd[gkey][k])
            sqrt_v = abs(g) / math.sqrt(float(gd[zkey][k]))
            want = lr * g / (sqrt_v + eps)
            got = float(W.reshape(-1)[k])
            assert abs(got - want) <= 1e-7 * abs(want), (t, k, got, want)


def test_t1_update_is_independent_of_beta2():
    rng = np.random.default_rng(1)
    G = rng.standard_normal((5, 3)).astype(np.float32)
    outs = []
    for b2 in (0.0, 0.5, 0.9, B2_F32):
        W = np.zeros((5, 3), np.float32)
        r, c = _zero_state(5, 3)
        assert oracle.step(W, G, r, c, 1, beta2=b2, eps=0.0) == 0
        outs.append(W)
    for W in outs[1:]:
        np.testing.assert_allclose(W, outs[0], rtol=2e-7, atol=0)


def test_t1_closed_form_row_col_grand_means():
    # At t=1: vtil_ij = R_i C_j / M with R, C, M the row, column and grand means of g^2.
    rng = np.random.default_rng(2)
    G = rng.standard_normal((7, 5)).astype(np.float32)
    g = G.astype(np.float64)
    R, C, M = (g * g).mean(1), (g * g).mean(0), (g * g).mean()
    want = -1e-3 * g / np.sqrt(np.outer(R, C) / M)
    W = np.zeros_like(G)
    r, c = _zero_state(7, 5)
    assert oracle.step(W, G, r, c, 1, eps=0.0) == 0
    np.testing.assert_allclose(W, want, rtol=1e-6, atol=0)


# ---------------------------------------------------------------------------
# Brute-force statistics, normaliser identity, state shape
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("V,D", [(1, 1), (1, 64), (63, 1), (63, 64), (64, 65), (65, 63)])
def test_row_col_statistics_brute_force(V, D):
    rng = np.random.default_rng(V * 1000 + D)
    r0 = rng.uniform(0, 2, V).astype(np.float32)
    c0 = rng.uniform(0, 2, D).astype(np.float32)
    G = (rng.standard_normal((V, D)) * rng.uniform(0.1, 3, (V, 1))).astype(np.float32)
    r, c = r0.copy(), c0.copy()
    W = np.zeros((V, D), np.float32)
    assert oracle.step(W, G, r, c, 3, beta2=0.9) == 0
    b2 = float(np.float32(0.9))
    g2 = G.astype(np.float64) ** 2
    want_r = (b2 * r0 + (1 - b2) * g2.mean(axis=1)).astype(np.float32)
    want_c = (b2 * c0 + (1 - b2) * g2.mean(axis=0)).astype(np.float32)
    np.testing.assert_array_max_ulp(r, want_r, maxulp=1)
    np.testing.assert_array_max_ulp(c, want_c, maxulp=1)


def test_normaliser_identity_mean_rhat_equals_mean_chat():
    # Appendix "Outer Product Unit Alignment": mean(rhat) == mean(chat) identically.
    rng = np.random.default_rng(3)
    V, D = 50, 30
    r, c = _zero_state(V, D)
    W = np.zeros((V, D), np.float32)
    for t in range(1, 8):
        G = (rng.standard_normal((V, D)) * rng.uniform(0.01, 10, (V, 1))).astype(np.float32)
        assert oracle.step(W, G, r, c, t) == 0
        mr, mc = r.astype(np.float64).mean(), c.astype(np.float64).mean()
        assert abs(mr - mc) <= 1e-6 * mr


def test_state_bytes_match_paper_table():
    with open(os.path.join(GOLDEN, "state_bytes_table.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert len(rows) == 8
    for model, V, D, tables, kib, adamw in rows:
        V, D, tables, kib = int(V), int(D), int(tables), int(kib)
        ember = tables * oracle.state_bytes(V, D)
        assert abs(ember / 1024 - kib) <= max(0.5, 0.005 * kib), model
        unit = 1e9 if adamw.endswith("GB") else 1e6
        printed = float(adamw[:-2])
        adam_bytes = tables * 2 * V * D * 4
        digits = len(adamw[:-2].split(".")[1]) if "." in adamw else 0
        assert abs(adam_bytes / unit - printed) <= 0.5 * 10.0 ** -digits + 1e-9, model


# ---------------------------------------------------------------------------
# Special cases that reduce to a library routine: Adam with beta1 = 0
# ---------------------------------------------------------------------------

def _adam_updates(grads, lr, beta2, eps, shape):
    p = torch.zeros(shape, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=lr, betas=(0.0, beta2), eps=eps)
    ups = []
    for g in grads:
        with torch.no_grad():
            p.zero_()
        p.grad = torch.from_numpy(g.astype(np.float64))
        opt.step()
        ups.append(p.detach().numpy().copy())
    return ups


def _ember_updates(grads, lr, beta2, eps, shape):
    r, c = _zero_state(*shape)
    ups = []
    for t, g in enumerate(grads, 1):
        W = np.zeros(shape, np.float32)
        assert oracle.step(W, g, r, c, t, lr=lr, beta2=beta2, eps=eps) == 0
        ups.append(W.astype(np.float64))
    return ups


@pytest.mark.parametrize("shape", [(17, 1), (1, 13)])
def test_single_column_or_row_equals_adam_beta1_zero(shape):
    rng = np.random.default_rng(4)
    grads = [(rng.standard_normal(shape) * rng.uniform(0.1, 5)).astype(np.float32) for _ in range(6)]
    for a, b in zip(_adam_updates(grads, 1e-3, B2_F32, 1e-8, shape),
                    _ember_updates(grads, 1e-3, B2_F32, 1e-8, shape)):
        np.testing.assert_allclose(b, a, rtol=1e-6, atol=0)


@pytest.mark.parametrize("scale", [1.0, 1e-8])
def test_rank1_gradients_equal_adam_beta1_zero(scale):
    # Appendix "Outer Product Unit Alignment", paragraph "Exactness": for a rank-1
    # second moment the factored estimate equals the dense one.  With g_t = gamma_t x y^T
    # Ember's vtil equals Adam's vhat element by element.  The tiny scale makes eps
    # (added after the square root) matter.
    rng = np.random.default_rng(5)
    V, D = 9, 6
    x, y = rng.standard_normal(V), rng.standard_normal(D)
    grads = [(scale * rng.uniform(0.2, 3) * np.outer(x, y)).astype(np.float32) for _ in range(5)]
    # fp32 rounding of g breaks exact rank-1 only at the 1e-7 level
    for a, b in zip(_adam_updates(grads, 1e-3, B2_F32, 1e-8, (V, D)),
                    _ember_updates(grads, 1e-3, B2_F32, 1e-8, (V, D))):
        np.testing.assert_allclose(b, a, rtol=2e-6, atol=0)


# ---------------------------------------------------------------------------
# Bitwise invariants and symmetries
# ---------------------------------------------------------------------------

def _random_history(rng, V, D, steps, W_dtype=np.float32):
    W = (rng.standard_normal((V, D)) * 0.02).astype(np.float32)
    r, c = _zero_state(V, D)
    for t in range(1, steps + 1):
        G = (rng.standard_normal((V, D)) * 1e-3).astype(np.float32)
        assert oracle.step(W, G, r, c, t) == 0
    return W, r, c


def test_zero_gradient_keeps_weights_and_decays_state_bitwise():
    rng = np.random.default_rng(6)
    W, r, c = _random_history(rng, 20, 12, 3)
    W0, r0, c0 = W.copy(), r.copy(), c.copy()
    assert oracle.step(W, np.zeros_like(W), r, c, 4) == 0
    assert np.array_equal(W.view(np.uint32), W0.view(np.uint32))
    assert np.array_equal(r, np.float32(B2_F32) * r0)
    assert np.array_equal(c, np.float32(B2_F32) * c0)


def test_all_zero_from_zero_state_is_finite_noop():
    W = np.full((4, 3), -0.0, np.float32)
    r, c = _zero_state(4, 3)
    assert oracle.step(W, np.zeros((4, 3), np.float32), r, c, 1) == 0
    assert np.all(W.view(np.uint32) == np.float32(-0.0).view(np.uint32))
    assert not r.any() and not c.any()


def test_transpose_symmetry_bitwise():
    rng = np.random.default_rng(8)
    V, D = 11, 7
    r, c = rng.uniform(0, 1, V).astype(np.float32), rng.uniform(0, 1, D).astype(np.float32)
    G = rng.standard_normal((V, D)).astype(np.float32)
    W = np.zeros((V, D), np.float32)
    WT = np.zeros((D, V), np.float32)
    rT, cT = c.copy(), r.copy()
    assert oracle.step(W, G, r, c, 2) == 0
    assert oracle.step(WT, np.ascontiguousarray(G.T), rT, cT, 2) == 0
    assert np.array_equal(W.T, WT)
    assert np.array_equal(r, cT) and np.array_equal(c, rT)


def test_sign_flip_negates_update_and_keeps_state():
    rng = np.random.default_rng(9)
    G = rng.standard_normal((6, 5)).astype(np.float32)
    outs = []
    for sgn in (1, -1):
        W = np.zeros((6, 5), np.float32)
        r, c = _zero_state(6, 5)
        assert oracle.step(W, sgn * G, r, c, 1) == 0
        outs.append((W, r, c))
    assert np.array_equal(outs[0][0], -outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1]) and np.array_equal(outs[0][2], outs[1][2])


def test_maximize_is_the_papers_ascent_form():
    rng = np.random.default_rng(10)
    G = rng.standard_normal((6, 5)).astype(np.float32)
    Wd, Wa = np.zeros((6, 5), np.float32), np.zeros((6, 5), np.float32)
    for W, mx in ((Wd, False), (Wa, True)):
        r, c = _zero_state(6, 5)
        assert oracle.step(W, G, r, c, 1, maximize=mx) == 0
    assert np.array_equal(Wa, -Wd)
    assert np.all(np.sign(Wa) == np.sign(G))          # ascend: theta + alpha g / ...


@pytest.mark.parametrize("k", [-20, -3, 5])
def test_power_of_two_gradient_scale_leaves_update_unchanged(k):
    # With eps = 0 the update is unitless (appendix "Outer Product Unit Alignment").
    rng = np.random.default_rng(11)
    V, D = 8, 9
    outs = []
    for scale in (1.0, 2.0 ** k):
        W = np.zeros((V, D), np.float32)
        r, c = _zero_state(V, D)
        rng2 = np.random.default_rng(12)
        for t in range(1, 4):
            G = (rng2.standard_normal((V, D)) * scale).astype(np.float32)
            W[:] = 0
            assert oracle.step(W, G, r, c, t, eps=0.0) == 0
        outs.append(W.copy())
    assert np.array_equal(outs[0], outs[1])


def test_bf16_weights_round_once_from_float64():
    rng = np.random.default_rng(13)
    V, D = 10, 16
    W32 = (rng.standard_normal((V, D)) * 0.02).astype(np.float32)
    Wb = (W32.view(np.uint32) >> 16).astype(np.uint16)        # truncate to bf16 bits
    G = (rng.standard_normal((V, D)) * 1e-3).astype(np.float32)
    Gb = (G.view(np.uint32) >> 16).astype(np.uint16)
    Wf = (Wb.astype(np.uint32) << 16).view(np.float32).copy()
    Gf = (Gb.astype(np.uint32) << 16).view(np.float32).copy()
    r1, c1 = _zero_state(V, D)
    r2, c2 = _zero_state(V, D)
    Wb2 = Wb.copy()
    assert oracle.step(Wb2, Gb, r1, c1, 1) == 0
    # fp32 storage of the same problem in float64 gives the pre-rounding values
    Wd = Wf.astype(np.float64)
    g = Gf.astype(np.float64)
    R, C, M = (g * g).mean(1), (g * g).mean(0), (g * g).mean()
    want = Wd - 1e-3 * g / (np.sqrt(np.outer(R, C) / M) + 1e-8)
    # one round-to-nearest-even of the float64 result (truncation would miss ~half)
    expect = np.array([[_bf16_rne_exact(float(want[i, j])) for j in range(D)] for i in range(V)])
    assert np.array_equal(Wb2.astype(np.int64), expect)
    assert oracle.step(Wf, Gf, r2, c2, 1) == 0
    assert np.array_equal(r1, r2) and np.array_equal(c1, c2)


# ---------------------------------------------------------------------------
# Sparse rows: dense with zero rows
# ---------------------------------------------------------------------------

def test_sparse_rows_equal_dense_with_zero_rows_bitwise():
    rng = np.random.default_rng(14)
    V, D, n = 40, 24, 13
    idx = rng.permutation(V)[:n].astype(np.int64)              # unique, unsorted
    W0, r0, c0 = _random_history(rng, V, D, 2)
    Grows = (rng.standard_normal((n, D)) * 1e-3).astype(np.float32)
    Gd = np.zeros((V, D), np.float32)
    Gd[idx] = Grows
    Ws, rs, cs = W0.copy(), r0.copy(), c0.copy()
    Wd, rd, cd = W0.copy(), r0.copy(), c0.copy()
    assert oracle.step(Ws, Grows, rs, cs, 3, idx=idx) == 0
    assert oracle.step(Wd, Gd, rd, cd, 3) == 0
    assert np.array_equal(Ws.view(np.uint32), Wd.view(np.uint32))
    assert np.array_equal(rs, rd) and np.array_equal(cs, cd)
    untouched = np.setdiff1d(np.arange(V), idx)
    assert np.array_equal(Ws[untouched].view(np.uint32), W0[untouched].view(np.uint32))
    assert np.array_equal(rs[untouched], np.float32(B2_F32) * r0[untouched])


def test_sparse_empty_index_list_is_a_full_step():
    rng = np.random.default_rng(15)
    W0, r0, c0 = _random_history(rng, 9, 5, 2)
    W, r, c = W0.copy(), r0.copy(), c0.copy()
    assert oracle.step(W, np.zeros((0, 5), np.float32), r, c, 3, idx=np.zeros(0, np.int64)) == 0
    assert np.array_equal(W, W0)
    assert np.array_equal(r, np.float32(B2_F32) * r0) and np.array_equal(c, np.float32(B2_F32) * c0)


@pytest.mark.parametrize("bad", [[0, 3, 3], [0, -1], [0, 9]])
def test_sparse_bad_indices_fail_and_modify_nothing(bad):
    rng = np.random.default_rng(16)
    W0, r0, c0 = _random_history(rng, 9, 5, 1)
    W, r, c = W0.copy(), r0.copy(), c0.copy()
    idx = np.array(bad, np.int64)
    G = np.ones((len(bad), 5), np.float32)
    assert oracle.step(W, G, r, c, 2, idx=idx) == oracle.BAD_INDEX
    assert np.array_equal(W, W0) and np.array_equal(r, r0) and np.array_equal(c, c0)


def test_bad_arguments_rejected():
    W = np.zeros((3, 2), np.float32)
    G = np.zeros((3, 2), np.float32)
    r, c = _zero_state(3, 2)
    assert oracle.step(W, G, r, c, 0) == oracle.BAD_ARG              # t >= 1
    assert oracle.step(W, G, r, c, 1, beta2=1.0) == oracle.BAD_ARG   # beta2 in [0, 1)
    assert oracle.step(W, G, r, c, 1, beta2=-0.1) == oracle.BAD_ARG


# ---------------------------------------------------------------------------
# Property: frequency isotropy (Section 2.2; appendix on inverse-frequency Fisher)
# ---------------------------------------------------------------------------

def test_row_update_scale_is_independent_of_token_frequency():
    # Coherent rows with K_i ~ Binomial(B, p_i) occurrences: the raw row gradient grows
    # ~ p_i, the Ember update's row RMS (averaged over steps) does not.  Row directions
    # are random signs so that the column factor is flat and only the row factor acts.
    rng = np.random.default_rng(17)
    V, D, B = 6, 32, 4096
    p = np.array([0.3, 0.1, 0.03, 0.01, 0.003, 0.001])
    mu = rng.choice([-1.0, 1.0], (V, D))
    W = np.zeros((V, D), np.float32)
    r, c = _zero_state(V, D)
    upd = np.zeros(V)
    raw = np.zeros(V)
    for t in range(1, 401):
        K = rng.binomial(B, p)
        G = ((K / B)[:, None] * mu).astype(np.float32)
        W[:] = 0
        assert oracle.step(W, G, r, c, t) == 0
        if t > 200:
            upd += np.sqrt((W.astype(np.float64) ** 2).mean(1))
            raw += np.sqrt((G.astype(np.float64) ** 2).mean(1))
    assert raw.max() / raw.min() > 100
    assert upd.max() / upd.min() < 1.5


# ---------------------------------------------------------------------------
# Row-only Ember (Section 2.1 and the ablation table; reading: vtil_ij = rhat_i)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("eps", [0.0, 1e-8])
def test_row_only_worked_2x2(eps):
    gd = _golden_2x2()
    beta2 = float(gd["beta2"][0])
    lr = 1e-3
    r = np.zeros(2, np.float32)
    c = np.full(2, 7.0, np.float32)                      # must stay untouched
    for t, gkey, rkey, vkey in ((1, "G1", "r1", "vrow1"), (2, "G2", "r2", "vrow2")):
        G = np.array([float(x) for x in gd[gkey]], np.float32).reshape(2, 2)
        W = np.zeros((2, 2), np.float32)
        assert oracle.step(W, G, r, c, t, lr=lr, beta2=beta2, eps=eps, maximize=True, row_only=True) == 0
        assert r.tolist() == [float(x) for x in gd[rkey]]
        assert c.tolist() == [7.0, 7.0]
        for k in range(4):
            g = float(gd[gkey][k])
            want = lr * g / (math.sqrt(float(gd[vkey][k // 2])) + eps)
            got = float(W.reshape(-1)[k])
            assert abs(got - want) <= 1e-7 * abs(want), (t, k, got, want)


def _row_only_updates(grads, shape, lr=1e-3, beta2=B2_F32, eps=1e-8):
    r = np.zeros(shape[0], np.float32)
    ups = []
    for t, g in enumerate(grads, 1):
        W = np.zeros(shape, np.float32)
        assert oracle.step(W, g, r, None, t, lr=lr, beta2=beta2, eps=eps, row_only=True) == 0
        ups.append(W.astype(np.float64))
    return ups


@pytest.mark.parametrize("shape", [(9, 1), (7, 16)])
def test_row_only_equal_magnitude_rows_equal_adam_beta1_zero(shape):
    # |g_ij| constant along each row: mean_j g^2 = g_ij^2, so the row statistic is
    # Adam's elementwise second moment and row-only Ember is Adam with beta1 = 0.
    rng = np.random.default_rng(18)
    V, D = shape
    grads = []
    for _ in range(5):
        x = rng.uniform(0.1, 3, (V, 1)) * rng.uniform(0.5, 2)
        grads.append((x * rng.choice([-1.0, 1.0], (V, D))).astype(np.float32))
    for a, b in zip(_adam_updates(grads, 1e-3, B2_F32, 1e-8, shape), _row_only_updates(grads, shape)):
        np.testing.assert_allclose(b, a, rtol=1e-6, atol=0)


def test_row_only_equals_canonical_when_columns_are_flat():
    # g_ij^2 = x_i^2 for every j: every column statistic is the same number, so
    # s = chat_j and the canonical preconditioner reduces to rhat_i.
    rng = np.random.default_rng(19)
    V, D = 12, 10
    r1, r2 = np.zeros(V, np.float32), np.zeros(V, np.float32)
    c = np.zeros(D, np.float32)
    for t in range(1, 6):
        x = rng.uniform(0.1, 3, (V, 1))
        G = (x * rng.choice([-1.0, 1.0], (V, D))).astype(np.float32)
        Wa, Wb = np.zeros((V, D), np.float32), np.zeros((V, D), np.float32)
        assert oracle.step(Wa, G, r1, c, t) == 0
        assert oracle.step(Wb, G, r2, None, t, row_only=True) == 0
        assert np.array_equal(r1, r2)
        assert np.all(c == c[0])
        np.testing.assert_allclose(Wb, Wa, rtol=1e-6, atol=0)


def test_row_only_sparse_equals_dense_with_zero_rows_bitwise():
    rng = np.random.default_rng(20)
    V, D, n = 30, 16, 9
    idx = rng.permutation(V)[:n].astype(np.int64)
    W0 = (rng.standard_normal((V, D)) * 0.02).astype(np.float32)
    r0 = rng.uniform(0, 1e-6, V).astype(np.float32)
    Grows = (rng.standard_normal((n, D)) * 1e-3).astype(np.float32)
    Gd = np.zeros((V, D), np.float32)
    Gd[idx] = Grows
    Ws, rs = W0.copy(), r0.copy()
    Wd, rd = W0.copy(), r0.copy()
    assert oracle.step(Ws, Grows, rs, None, 4, idx=idx, row_only=True) == 0
    assert oracle.step(Wd, Gd, rd, None, 4, row_only=True) == 0
    assert np.array_equal(Ws.view(np.uint32), Wd.view(np.uint32))
    assert np.array_equal(rs, rd)
    untouched = np.setdiff1d(np.arange(V), idx)
    assert np.array_equal(rs[untouched], np.float32(B2_F32) * r0[untouched])
    assert np.array_equal(Ws[untouched], W0[untouched])


def test_row_only_zero_gradient_is_bitwise():
    rng = np.random.default_rng(21)
    V, D = 8, 6
    W = (rng.standard_normal((V, D)) * 0.02).astype(np.float32)
    r = rng.uniform(0, 1, V).astype(np.float32)
    W0, r0 = W.copy(), r.copy()
    assert oracle.step(W, np.zeros((V, D), np.float32), r, None, 3, row_only=True) == 0
    assert np.array_equal(W, W0)
    assert np.array_equal(r, np.float32(B2_F32) * r0)
