"""GPU parity of the LM-head step with the statistics fused into the weight-
gradient GEMM (ember_lmhead_step), through the C ABI.

Bars:
* G: the library accumulates the T products of each element in fp32 (MFMA)
  and rounds once to the G dtype.  Any order of fp32 additions of T terms is
  within (T - 1) u sum|terms| of the exact sum (u = 2^-24; 2u allowed, in case
  the accumulation truncates), and the final rounding adds at most one ulp of
  the result, so |G - E| <= 2 T 2^-24 sum_m |dY_mi H_mj| + ulp(G), with E the
  exact sum (float64 products of bf16 values are exact; the float64 sum of T
  of them is within T 2^-53 of exact, far inside the bound).
* the step: in lockstep on the G the library wrote, r and c within 1e-5
  relative of the oracle, W by the dense-step rules of test_gpu_parity.
* padding columns of dY and H (also NaN) never reach a stored value; T = 0
  gives G = 0 and leaves W bit-identical; the result is bit-reproducible.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01455_amd import workloads as wl
from parity_checks import B2, DEV, EPS, LR, as_f64, check_state, check_w, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


def _padded(rows, cols, dtype, pad_chunks=0):
    q = 8 if dtype == torch.bfloat16 else 4
    ld = ((cols + q - 1) // q + pad_chunks) * q
    return torch.zeros(rows, ld, dtype=dtype, device=DEV)[:, :cols]


def _ulp(g: np.ndarray, bits_dtype) -> np.ndarray:
    a = np.abs(g)
    if bits_dtype == np.uint16:
        e = np.floor(np.log2(np.maximum(a, 2.0 ** -133)))
        return np.maximum(2.0 ** (e - 7), 2.0 ** -133)
    return np.spacing(a.astype(np.float32)).astype(np.float64)


def check_grad(G_bits: np.ndarray, dY64: np.ndarray, H64: np.ndarray, what: str) -> float:
    """G (host bits, rows x cols) against exact sums over the T tokens; returns
    the fraction of elements equal to the exact sum rounded once."""
    T = dY64.shape[0]
    E = dY64.T @ H64
    S = np.abs(dY64).T @ np.abs(H64)
    g = as_f64(G_bits)
    tol = 2.0 * T * 2.0 ** -24 * S + _ulp(g, G_bits.dtype)
    err = np.abs(g - E)
    bad = ~(err <= tol)
    assert not bad.any(), (f"{what}: {bad.sum()} of {g.size} G elements outside the fp32-accumulation bound; "
                           f"first at {np.argwhere(bad)[:3].tolist()}: got {g[bad][:3]} exact {E[bad][:3]}")
    # for the log: how many equal the exact sum rounded to the dtype (via fp32)
    e32 = E.astype(np.float32)
    if G_bits.dtype == np.uint16:
        b = e32.view(np.uint32).astype(np.uint64)
        once = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
        return float(np.mean(G_bits == once))
    return float(np.mean(g == e32))


def run_steps(em, T, V, D, g_dtype, w_dtype, steps, seed, ldy_pad=0, ldh_pad=0, nan_pad=False,
              lr=LR, maximize=False):
    cfg = wl.Config("lmh", V, D, w_dtype, g_dtype, steps, "logits", batch_tokens=T)
    print(f"lmhead step T={T} V={V} D={D} G={g_dtype} W={w_dtype} pads=({ldy_pad},{ldh_pad}) nan={nan_pad}",
          flush=True)
    W = _padded(V, D, w_dtype, 1)
    W.copy_(wl.make_weights(cfg, seed=seed, device=DEV))
    G = _padded(V, D, g_dtype, 1)
    tab = em.EmberTable(V, D, device=DEV)
    r_o = np.zeros(V, np.float32)
    c_o = np.zeros(D, np.float32)
    for t in range(1, steps + 1):
        ldy = ((V + 7) // 8 + ldy_pad) * 8
        ldh = ((D + 7) // 8 + ldh_pad) * 8
        dY, H = wl.make_lmhead_batch(cfg, t, seed=seed, device=DEV, ldy=ldy, ldh=ldh)
        if nan_pad:
            full_y = dY.as_strided((T, ldy), (ldy, 1))
            full_h = H.as_strided((T, ldh), (ldh, 1))
            full_y[:, V:] = float("nan")
            full_h[:, D:] = float("nan")
        W_prev = host_bits(W)
        tab.t = t - 1
        em.ember_lmhead_step(W, dY, H, G, tab.r, tab.c, t, lr, B2, EPS, maximize, tab.ws)
        torch.cuda.synchronize()
        G_h = host_bits(G)
        frac = check_grad(G_h, as_f64(host_bits(dY)), as_f64(host_bits(H)), f"G step {t}")
        W_ref = W_prev.copy()
        assert oracle.step(W_ref, G_h, r_o, c_o, t, lr=lr, maximize=maximize) == 0
        check_state(tab.r, r_o, f"r step {t}")
        check_state(tab.c, c_o, f"c step {t}")
        check_w(host_bits(W), W_ref, W_prev, f"W step {t}")
        print(f"  step {t}: G elements equal to the once-rounded exact sum: {frac:.4f}", flush=True)
    return W, G, tab


@pytest.mark.parametrize("T,V,D,gd,wd,steps", [
    (1, 1, 1, torch.bfloat16, torch.bfloat16, 2),        # degenerate: one token, one element
    (64, 256, 256, torch.bfloat16, torch.bfloat16, 2),   # one tile, one token step
    (200, 600, 520, torch.bfloat16, torch.bfloat16, 3),  # ragged rows, columns and tokens
    (130, 513, 264, torch.float32, torch.float32, 2),    # fp32 G and W
    (300, 1000, 72, torch.bfloat16, torch.float32, 2),   # narrow D, mixed dtypes
    (70, 300, 1001, torch.float32, torch.bfloat16, 2),   # D not a multiple of 8: partial chunks
    (256, 5000, 2048, torch.bfloat16, torch.bfloat16, 1),  # 160 tiles over the XCD mapping
])
def test_lmhead_step_matches_the_oracle(em, T, V, D, gd, wd, steps):
    run_steps(em, T, V, D, gd, wd, steps, seed=T + V + D)


@pytest.mark.parametrize("T,V,D,gd", [
    (1, 1, 1, torch.bfloat16),
    (64, 256, 256, torch.bfloat16),
    (200, 600, 520, torch.bfloat16),   # ragged rows, columns and tokens
    (130, 513, 264, torch.float32),
    (70, 300, 1001, torch.float32),    # D not a multiple of 8
    (300, 1000, 72, torch.bfloat16),
])
def test_lmhead_grad_exact_sums_are_bitwise_the_oracle(em, T, V, D, gd):
    """Entries k / 16 with integer |k| <= 32 (exact in bf16): every product is a
    multiple of 2^-8 of magnitude <= 4, so every fp32 partial sum of up to 300
    of them is exact, in any order.  The library's G is then the exact sum
    rounded once, which is what oracle.lmhead_grad computes: bit for bit."""
    print(f"lmhead exact sums T={T} V={V} D={D} G={gd}", flush=True)
    gen = torch.Generator().manual_seed(T * 7 + V + D)
    dY = _padded(T, V, torch.bfloat16, 1)
    H = _padded(T, D, torch.bfloat16, 2)
    dY.copy_((torch.randint(-32, 33, (T, V), generator=gen).float() / 16).to(DEV))
    H.copy_((torch.randint(-32, 33, (T, D), generator=gen).float() / 16).to(DEV))
    cfg = wl.Config("lmh_exact", V, D, torch.bfloat16, gd, 1, "logits", batch_tokens=T)
    W = _padded(V, D, torch.bfloat16, 1)
    W.copy_(wl.make_weights(cfg, seed=T, device=DEV))
    G = _padded(V, D, gd, 1)
    tab = em.EmberTable(V, D, device=DEV)
    em.ember_lmhead_step(W, dY, H, G, tab.r, tab.c, 1, LR, B2, EPS, False, tab.ws)
    torch.cuda.synchronize()
    want = oracle.lmhead_grad(host_bits(dY), host_bits(H), np.uint16 if gd == torch.bfloat16 else np.float32)
    got = host_bits(G)
    if gd == torch.float32:
        got, want = got.view(np.uint32), want.view(np.uint32)
    diff = got != want
    assert not diff.any(), (f"{int(diff.sum())} of {got.size} G elements differ from the exactly summed oracle; "
                            f"first at {np.argwhere(diff)[:3].tolist()}")


def test_padding_never_reaches_a_stored_value(em):
    run_steps(em, 100, 700, 300, torch.bfloat16, torch.bfloat16, 2, seed=9, ldy_pad=3, ldh_pad=5, nan_pad=True)


def test_no_tokens(em):
    V, D = 300, 64
    cfg = wl.Config("lmh0", V, D, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=0)
    W = wl.make_weights(cfg, seed=3, device=DEV)
    G = torch.full((V, D), 7.0, dtype=torch.bfloat16, device=DEV)
    tab = em.EmberTable(V, D, device=DEV)
    # one real step first so that r and c are nonzero
    dY, H = wl.make_lmhead_batch(cfg, 1, seed=3, device=DEV, T=50, ldy=304)
    em.ember_lmhead_step(W, dY, H, G, tab.r, tab.c, 1, LR, B2, EPS, False, tab.ws)
    torch.cuda.synchronize()
    W1, r1, c1 = W.clone(), tab.r.clone(), tab.c.clone()
    empty_y = torch.empty(0, V, dtype=torch.bfloat16, device=DEV)
    empty_h = torch.empty(0, D, dtype=torch.bfloat16, device=DEV)
    em.ember_lmhead_step(W, empty_y, empty_h, G, tab.r, tab.c, 2, LR, B2, EPS, False, tab.ws)
    torch.cuda.synchronize()
    assert not G.float().any()
    assert torch.equal(W.view(torch.int16), W1.view(torch.int16))
    assert torch.equal(tab.r, (torch.tensor(B2, dtype=torch.float32) * r1.cpu()).to(DEV))
    assert torch.equal(tab.c, (torch.tensor(B2, dtype=torch.float32) * c1.cpu()).to(DEV))


def test_bitwise_reproducible(em):
    T, V, D = 512, 2048, 1024
    cfg = wl.Config("lmh_det", V, D, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=T)
    dY, H = wl.make_lmhead_batch(cfg, 1, seed=5, device=DEV)
    outs = []
    for _ in range(2):
        W = wl.make_weights(cfg, seed=5, device=DEV)
        G = torch.empty(V, D, dtype=torch.bfloat16, device=DEV)
        tab = em.EmberTable(V, D, device=DEV)
        for t in (1, 2):
            em.ember_lmhead_step(W, dY, H, G, tab.r, tab.c, t, LR, B2, EPS, False, tab.ws)
        torch.cuda.synchronize()
        outs.append((host_bits(W), host_bits(G), tab.r.cpu().numpy(), tab.c.cpu().numpy()))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


@pytest.mark.timeout(900)
def test_full_lmhead128k_wgrad_step(em):
    """The benchmark's workload: 16384 tokens, 128256 x 4096 bf16.  G is checked
    on sampled rows (every column, tile edges included) against exact sums;
    the step in lockstep on the library's G, r and c on every element, W on
    the sampled rows."""
    cfg = wl.CONFIGS["lmhead128k_wgrad"]
    V, D, T = cfg.V, cfg.D, cfg.batch_tokens
    print(f"full LM-head step T={T} V={V} D={D}", flush=True)
    W = wl.make_weights(cfg, seed=11, device=DEV)
    G = torch.empty(V, D, dtype=torch.bfloat16, device=DEV)
    tab = em.EmberTable(V, D, device=DEV)
    rng = np.random.default_rng(11)
    rows = np.unique(np.concatenate([rng.choice(V, 300, replace=False), [0, 1, 255, 256, 257, 511, 512],
                                     np.arange(V - 260, V - 250), [V - 2, V - 1]])).astype(np.int64)
    rows_t = torch.from_numpy(rows).to(DEV)
    r_o = np.zeros(V, np.float32)
    c_o = np.zeros(D, np.float32)
    for t in (1, 2):
        dY, H = wl.make_lmhead_batch(cfg, t, seed=11, device=DEV)
        W_prev_rows = host_bits(W[rows_t])
        em.ember_lmhead_step(W, dY, H, G, tab.r, tab.c, t, LR, B2, EPS, False, tab.ws)
        torch.cuda.synchronize()
        dY_rows = as_f64(host_bits(dY.index_select(1, rows_t)))
        H_h = as_f64(host_bits(H))
        del dY
        G_h = host_bits(G)
        frac = check_grad(G_h[rows], dY_rows, H_h, f"G step {t} (sampled rows)")
        print(f"  step {t}: sampled G elements equal to the once-rounded exact sum: {frac:.4f}", flush=True)
        W_ref = np.empty((V, D), np.uint16)
        W_ref[rows] = W_prev_rows
        assert oracle.step(W_ref, G_h, r_o, c_o, t, w_rows=rows) == 0
        check_state(tab.r, r_o, f"r step {t}")
        check_state(tab.c, c_o, f"c step {t}")
        check_w(host_bits(W[rows_t]), W_ref[rows], W_prev_rows, f"W step {t}")
        del W_ref, G_h
    del W, G, tab
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_ragged_shape_with_many_tiles(em):
    # 79 x 4 tiles of which the last row and column tiles are partial, and a
    # partial last token step: every element of G is checked
    run_steps(em, 1000, 20001, 1000, torch.bfloat16, torch.bfloat16, 1, seed=21, ldy_pad=1)


def test_captured_step_replays_bitwise(em):
    """The fused step captured in a HIP graph and replayed on fresh inputs gives
    the bits of the same step run eagerly on a twin table, replay after replay."""
    T, V, D = 300, 3000, 512
    cfg = wl.Config("lmh_graph", V, D, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=T)
    ldy = (V + 7) // 8 * 8

    def table():
        return (wl.make_weights(cfg, seed=23, device=DEV), torch.empty(V, D, dtype=torch.bfloat16, device=DEV),
                em.EmberTable(V, D, device=DEV))

    W, G, tab = table()
    W2, G2, tab2 = table()
    dY_s = torch.empty(T, ldy, dtype=torch.bfloat16, device=DEV)[:, :V]
    H_s = torch.empty(T, D, dtype=torch.bfloat16, device=DEV)
    t_fixed = 4

    def step(W_, G_, tab_, dY, H):
        tab_.t = t_fixed - 1
        tab_.step_lmhead(W_, dY, H, G_)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dY0, H0 = wl.make_lmhead_batch(cfg, 1, seed=23, device=DEV, ldy=ldy)
        dY_s.copy_(dY0)
        H_s.copy_(H0)
        step(W, G, tab, dY_s, H_s)
        step(W2, G2, tab2, dY0, H0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(W, G, tab, dY_s, H_s)
    for rep in range(2, 5):
        dY, H = wl.make_lmhead_batch(cfg, rep, seed=23, device=DEV, ldy=ldy)
        dY_s.copy_(dY)
        H_s.copy_(H)
        graph.replay()
        step(W2, G2, tab2, dY, H)
        torch.cuda.synchronize()
        assert torch.equal(G.view(torch.int16), G2.view(torch.int16))
        assert torch.equal(W.view(torch.int16), W2.view(torch.int16))
        assert torch.equal(tab.r, tab2.r) and torch.equal(tab.c, tab2.c)


def test_ascent_and_zero_learning_rate(em):
    # maximize: the paper's literal ascent; lr = 0: the state advances and W
    # keeps every bit (the apply pass is skipped)
    run_steps(em, 120, 700, 300, torch.bfloat16, torch.float32, 2, seed=25, maximize=True)
    W, _, _ = run_steps(em, 120, 700, 300, torch.bfloat16, torch.bfloat16, 2, seed=26, lr=0.0)
    cfg = wl.Config("lmh", 700, 300, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=120)
    assert torch.equal(W.view(torch.int16), wl.make_weights(cfg, seed=26, device=DEV).view(torch.int16))
