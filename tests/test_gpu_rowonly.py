"""GPU parity of row-only Ember (Section 2.1: vtil_ij = rhat_i, state V) against
the oracle's row-only mode, through the C ABI.

Same lockstep protocol and tolerances as the canonical step (the docstring of
test_gpu_parity): r within 1e-5 relative (bit-exact where it only decays by
beta2), fp32 W within 1e-5 of max(|oracle|, |W before|), bf16 W within 1 ulp
or the cancellation bound, W rows outside idx bit-identical.  The shapes cover
each launch form of the fused kernel: rows held in registers with one or two
2 KiB slabs per wave (one or two 16-byte chunks per lane), and rows too long to
hold, which are read twice; and rows of up to 1024 chunks handled by one wave
each (D a multiple of the chunk width or not).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01455_amd import workloads as wl
from parity_checks import B2, DEV, EPS, LR, check_state, check_w, host_bits, sample_rows
from parity_checks import ld_for as _ld

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


class RowTable:
    def __init__(self, em, V, D):
        self.r = torch.empty(V, dtype=torch.float32, device=DEV)
        self.ws = torch.empty(em.ember_workspace_bytes(V, D), dtype=torch.uint8, device=DEV)
        em.ember_rowonly_init_state(self.r, D, self.ws)
        self.r_o = np.zeros(V, np.float32)


def dense_lockstep(em, cfg, seed=0, steps=None, rows=None, ld_pad=0, maximize=False,
                   lr=LR, beta2=B2, eps=EPS, all_rows_at=(1,)):
    steps = cfg.steps if steps is None else steps
    print(f"row-only dense {cfg.name} V={cfg.V} D={cfg.D} w={cfg.w_dtype} g={cfg.g_dtype} steps={steps}",
          flush=True)
    ldw = _ld(cfg.D, cfg.w_dtype, ld_pad) if ld_pad else None
    ldg = _ld(cfg.D, cfg.g_dtype, ld_pad) if ld_pad else None
    W = wl.make_weights(cfg, seed=seed, device=DEV, ld=ldw)
    scales = wl.row_scales(cfg, seed, DEV)
    tab = RowTable(em, cfg.V, cfg.D)
    rows_t = None if rows is None else torch.from_numpy(rows).to(DEV)
    for t in range(1, steps + 1):
        G = wl.make_dense_grad(cfg, t, seed=seed, device=DEV, scales=scales, ld=ldg)
        full = rows is None or t in all_rows_at
        W_prev = host_bits(W) if full else None
        prev_rows = None if full else host_bits(W[rows_t])
        pad_before = host_bits(W.as_strided((cfg.V, ldw - cfg.D), (ldw, 1), cfg.D)) if ld_pad else None
        em.ember_rowonly_step_dense(W, G, tab.r, t, lr, beta2, eps, maximize, tab.ws)
        torch.cuda.synchronize()
        if full:
            W_ref = W_prev.copy()
        else:
            W_ref = np.empty((cfg.V, cfg.D), dtype=prev_rows.dtype)
            W_ref[rows] = prev_rows
        assert oracle.step(W_ref, host_bits(G), tab.r_o, None, t, lr=lr, beta2=beta2, eps=eps,
                           maximize=maximize, w_rows=None if full else rows, row_only=True) == 0
        check_state(tab.r, tab.r_o, f"{cfg.name} r step {t}")
        if full:
            check_w(host_bits(W), W_ref, W_prev, f"{cfg.name} W step {t}")
        else:
            check_w(host_bits(W[rows_t]), W_ref[rows], prev_rows, f"{cfg.name} W step {t} (sampled rows)")
        if ld_pad:
            pad_after = host_bits(W.as_strided((cfg.V, ldw - cfg.D), (ldw, 1), cfg.D))
            assert np.array_equal(pad_before, pad_after), "row padding of W was written"
        del G, W_ref
    return W, tab


def sparse_lockstep(em, cfg, seed=0, steps=None, shuffle=False):
    steps = cfg.steps if steps is None else steps
    print(f"row-only sparse {cfg.name} V={cfg.V} D={cfg.D} steps={steps} shuffle={shuffle}", flush=True)
    W = wl.make_weights(cfg, seed=seed, device=DEV)
    tab = RowTable(em, cfg.V, cfg.D)
    for t in range(1, steps + 1):
        idx, Gr = wl.make_sparse_batch(cfg, t, seed=seed, device=DEV, shuffle=shuffle)
        W_prev = host_bits(W)
        r_prev = tab.r.cpu().numpy()
        em.ember_rowonly_step_sparse_rows(W, Gr, idx, tab.r, t, LR, B2, EPS, False, tab.ws)
        assert em.ember_get_error(tab.ws) == em.EMBER_OK
        idx_h = idx.cpu().numpy()
        touched = np.sort(idx_h)
        W_ref = W_prev.copy()
        assert oracle.step(W_ref, host_bits(Gr), tab.r_o, None, t, lr=LR, beta2=B2, eps=EPS,
                           idx=idx_h, w_rows=touched, row_only=True) == 0
        check_state(tab.r, tab.r_o, f"{cfg.name} r step {t}")
        W_gpu = host_bits(W)
        check_w(W_gpu[touched], W_ref[touched], W_prev[touched], f"{cfg.name} W step {t}")
        mask = np.ones(cfg.V, bool)
        mask[touched] = False
        assert np.array_equal(W_gpu[mask], W_prev[mask]), "a row outside idx changed"
        r_gpu = tab.r.cpu().numpy()
        assert np.array_equal(r_gpu[mask], np.float32(B2) * r_prev[mask]), "untouched r is not beta2 * r"
    return W, tab


# ---------------------------------------------------------------------------
# every element
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("V,D,wd,gd,pad", [
    (1024, 64, torch.float32, torch.float32, 0),       # one slab, one chunk per lane
    (3001, 896, torch.float32, torch.float32, 1),      # two slabs, padded rows
    (2049, 1001, torch.bfloat16, torch.bfloat16, 1),   # ragged last chunk (padded rows)
    (777, 4096, torch.bfloat16, torch.bfloat16, 2),    # four slabs of 2 KiB
    (515, 4096, torch.float32, torch.bfloat16, 0),     # fp32 W, bf16 G
    (600, 4096, torch.bfloat16, torch.float32, 0),     # bf16 W, fp32 G: eight slabs
    (37, 4100, torch.float32, torch.float32, 0),       # nine slabs: two per wave
    (70, 12000, torch.bfloat16, torch.bfloat16, 1),    # twelve slabs: two per wave
    (19, 8200, torch.float32, torch.float32, 0),       # 17 slabs: rows read twice
    (21, 20000, torch.bfloat16, torch.float32, 0),     # 40 slabs: rows read twice
    (45, 8192, torch.bfloat16, torch.bfloat16, 0),     # one wave per row, 16 chunks per lane
    (33, 4096, torch.float32, torch.float32, 1),       # the same in fp32
    (100, 1500, torch.bfloat16, torch.bfloat16, 1),    # one wave per row, ragged, 4 chunks per lane
    (1, 4096, torch.bfloat16, torch.bfloat16, 0),      # one row
    (17, 1, torch.float32, torch.float32, 3),          # one column, odd row count
    (9, 8, torch.bfloat16, torch.bfloat16, 0),         # one partial row block
])
def test_rowonly_small_shapes_every_element(em, V, D, wd, gd, pad):
    cfg = wl.Config(f"ro{V}x{D}", V, D, wd, gd, 3, "loguniform_rows")
    dense_lockstep(em, cfg, seed=V + D, ld_pad=pad)


def test_rowonly_maximize_and_hyperparameters(em):
    cfg = wl.Config("ro_hp", 1200, 256, torch.float32, torch.float32, 3, "normal")
    dense_lockstep(em, cfg, seed=3, maximize=True, lr=3e-4, beta2=0.9, eps=1e-6)


@pytest.mark.parametrize("scale,eps", [(1e-15, 0.0), (1e-15, 1e-8), (1e10, 1e-8), (1e10, 0.0)])
def test_rowonly_extreme_gradient_scales(em, scale, eps):
    cfg = wl.Config("ro_scale", 900, 192, torch.float32, torch.float32, 3, "loguniform_rows", g_std=scale)
    dense_lockstep(em, cfg, seed=21, eps=eps)


def test_rowonly_large_step_counter(em):
    cfg = wl.Config("ro_late", 600, 512, torch.bfloat16, torch.bfloat16, 2, "normal")
    W = wl.make_weights(cfg, seed=4, device=DEV)
    tab = RowTable(em, cfg.V, cfg.D)
    for t in (10000, 10001):
        G = wl.make_dense_grad(cfg, t, seed=4, device=DEV)
        W_prev = host_bits(W)
        em.ember_rowonly_step_dense(W, G, tab.r, t, LR, B2, EPS, False, tab.ws)
        W_ref = W_prev.copy()
        assert oracle.step(W_ref, host_bits(G), tab.r_o, None, t, row_only=True) == 0
        check_state(tab.r, tab.r_o, "r")
        check_w(host_bits(W), W_ref, W_prev, "W")


def test_rowonly_zero_gradient_and_zero_lr(em):
    cfg = wl.Config("ro_zero", 3000, 768, torch.bfloat16, torch.bfloat16, 2, "normal")
    W, tab = dense_lockstep(em, cfg, seed=7)
    W_prev = host_bits(W)
    r_prev = tab.r.cpu().numpy()
    G = torch.zeros(cfg.V, cfg.D, dtype=cfg.g_dtype, device=DEV)
    em.ember_rowonly_step_dense(W, G, tab.r, 3, LR, B2, EPS, False, tab.ws)
    assert np.array_equal(host_bits(W), W_prev)
    assert np.array_equal(tab.r.cpu().numpy(), np.float32(B2) * r_prev)
    # lr = 0: the weights keep their bits, r still follows the oracle
    tab.r_o[:] = tab.r.cpu().numpy()
    G = wl.make_dense_grad(cfg, 4, seed=7, device=DEV)
    em.ember_rowonly_step_dense(W, G, tab.r, 4, 0.0, B2, EPS, False, tab.ws)
    idx = torch.arange(0, 100, dtype=torch.int64, device=DEV)
    em.ember_rowonly_step_sparse_rows(W, G[:100].contiguous(), idx, tab.r, 5, 0.0, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    assert np.array_equal(host_bits(W), W_prev)
    W_ref = W_prev.copy()
    assert oracle.step(W_ref, host_bits(G), tab.r_o, None, 4, lr=0.0, row_only=True) == 0
    assert oracle.step(W_ref, host_bits(G[:100]), tab.r_o, None, 5, lr=0.0, idx=idx.cpu().numpy(),
                       row_only=True) == 0
    check_state(tab.r, tab.r_o, "r")


def test_rowonly_sparse_every_row(em):
    cfg = wl.Config("ro_sparse", 5000, 320, torch.bfloat16, torch.bfloat16, 4, "sparse_zipf",
                    batch_tokens=3000)
    sparse_lockstep(em, cfg, seed=5, shuffle=True)


def test_rowonly_sparse_long_rows(em):
    # rows too long for one wave: the block form of the fused kernel
    cfg = wl.Config("ro_sparse_long", 3000, 9000, torch.bfloat16, torch.bfloat16, 2, "sparse_zipf",
                    batch_tokens=1500)
    sparse_lockstep(em, cfg, seed=8, shuffle=True)


def test_rowonly_sparse_fp32_and_empty_index_list(em):
    cfg = wl.Config("ro_sparse_f32", 2000, 200, torch.float32, torch.float32, 2, "sparse_zipf",
                    batch_tokens=500)
    W, tab = sparse_lockstep(em, cfg, seed=6)
    W_prev = host_bits(W)
    r_prev = tab.r.cpu().numpy()
    empty_i = torch.zeros(0, dtype=torch.int64, device=DEV)
    empty_g = torch.zeros(0, cfg.D, dtype=cfg.g_dtype, device=DEV)
    em.ember_rowonly_step_sparse_rows(W, empty_g, empty_i, tab.r, 3, LR, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    assert np.array_equal(host_bits(W), W_prev)
    assert np.array_equal(tab.r.cpu().numpy(), np.float32(B2) * r_prev)


@pytest.mark.parametrize("bad", ["duplicate", "negative", "too_large"])
def test_rowonly_sparse_index_errors_leave_everything_untouched(em, bad):
    cfg = wl.Config("ro_err", 1000, 128, torch.bfloat16, torch.bfloat16, 1, "normal")
    W = wl.make_weights(cfg, seed=9, device=DEV)
    tab = RowTable(em, cfg.V, cfg.D)
    G = wl.make_dense_grad(cfg, 1, seed=9, device=DEV)
    W0 = host_bits(W)
    em.ember_rowonly_step_dense(W, G, tab.r, 1, LR, B2, EPS, False, tab.ws)
    assert oracle.step(W0, host_bits(G), tab.r_o, None, 1, row_only=True) == 0
    ids = {"duplicate": [3, 7, 500, 7], "negative": [3, -1, 9, 10], "too_large": [3, 1000, 9, 10]}[bad]
    idx = torch.tensor(ids, dtype=torch.int64, device=DEV)
    Gr = G[:4].contiguous()
    before = (host_bits(W), tab.r.cpu().numpy())
    em.ember_rowonly_step_sparse_rows(W, Gr, idx, tab.r, 2, LR, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_ERR_INDEX
    assert np.array_equal(host_bits(W), before[0])
    assert np.array_equal(tab.r.cpu().numpy(), before[1])
    # the next valid step (same t) works and reports OK: error bits and row marks were cleared
    idx_ok = torch.tensor([3, 7, 500, 8], dtype=torch.int64, device=DEV)
    W_prev = host_bits(W)
    em.ember_rowonly_step_sparse_rows(W, Gr, idx_ok, tab.r, 2, LR, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    W_ref = W_prev.copy()
    assert oracle.step(W_ref, host_bits(Gr), tab.r_o, None, 2, idx=idx_ok.cpu().numpy(), row_only=True) == 0
    check_w(host_bits(W), W_ref, W_prev, "W after recovery")
    check_state(tab.r, tab.r_o, "r after recovery")
    em.ember_rowonly_step_sparse_rows(W, Gr, idx, tab.r, 3, LR, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_ERR_INDEX
    em.ember_rowonly_step_dense(W, G, tab.r, 3, LR, B2, EPS, False, tab.ws)
    assert em.ember_get_error(tab.ws) == em.EMBER_OK


def test_rowonly_sparse_error_and_recovery_with_many_blocks(em):
    # ~1000 row blocks plus the decay blocks: every block counts itself in one
    # of the completion counters before the last one clears the error bits;
    # an index error, then valid steps, repeated, must each report correctly
    cfg = wl.Config("ro_err_big", 20000, 1024, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf",
                    batch_tokens=4000)
    W = wl.make_weights(cfg, seed=12, device=DEV)
    tab = em.EmberTable(cfg.V, cfg.D, device=DEV, row_only=True)
    twin_W = W.clone()
    twin = em.EmberTable(cfg.V, cfg.D, device=DEV, row_only=True)
    rng = np.random.default_rng(12)
    g = torch.Generator(device=DEV).manual_seed(12)
    for t in range(1, 4):
        n = 4000
        ids = rng.permutation(cfg.V)[:n].astype(np.int64)
        Gr = (torch.randn(n, cfg.D, generator=g, device=DEV) * 1e-3).to(torch.bfloat16)
        bad = ids.copy()
        bad[n - 1] = bad[0]                      # a repeated id in the last block
        before = (host_bits(W), tab.r.cpu().numpy())
        em.ember_rowonly_step_sparse_rows(W, Gr, torch.from_numpy(bad).to(DEV), tab.r, t, LR, B2, EPS, False, tab.ws)
        assert em.ember_get_error(tab.ws) == em.EMBER_ERR_INDEX
        assert np.array_equal(host_bits(W), before[0]) and np.array_equal(tab.r.cpu().numpy(), before[1])
        idx = torch.from_numpy(ids).to(DEV)
        em.ember_rowonly_step_sparse_rows(W, Gr, idx, tab.r, t, LR, B2, EPS, False, tab.ws)
        assert em.ember_get_error(tab.ws) == em.EMBER_OK
        # the twin takes only the valid steps: the same bits
        em.ember_rowonly_step_sparse_rows(twin_W, Gr, idx, twin.r, t, LR, B2, EPS, False, twin.ws)
        assert em.ember_get_error(twin.ws) == em.EMBER_OK
        assert torch.equal(W.view(torch.int16), twin_W.view(torch.int16)) and torch.equal(tab.r, twin.r)


def test_rowonly_bitwise_reproducible_and_table_binding(em):
    cfg = wl.Config("ro_det", 20000, 1024, torch.bfloat16, torch.bfloat16, 2, "sparse_zipf",
                    batch_tokens=4000)
    outs = []
    for rep in range(2):
        W = wl.make_weights(cfg, seed=10, device=DEV)
        tab = em.EmberTable(cfg.V, cfg.D, device=DEV, row_only=True)
        assert tab.c is None
        G = wl.make_dense_grad(cfg, 1, seed=10, device=DEV)
        tab.step(W, G)
        idx, Gr = wl.make_sparse_batch(cfg, 2, seed=10, device=DEV, shuffle=True)
        tab.step_sparse_rows(W, Gr, idx, check=True)
        assert tab.t == 2
        outs.append((host_bits(W), tab.r.cpu().numpy()))
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


# ---------------------------------------------------------------------------
# full-size workloads
# ---------------------------------------------------------------------------

@pytest.mark.timeout(600)
def test_rowonly_full_lmhead128k_bf16(em):
    cfg = wl.CONFIGS["lmhead128k"]
    dense_lockstep(em, cfg, seed=12, rows=sample_rows(cfg.V), all_rows_at=(1,))


@pytest.mark.timeout(600)
def test_rowonly_full_lmhead32k_fp32(em):
    cfg = wl.CONFIGS["lmhead32k"]
    dense_lockstep(em, cfg, seed=11, steps=4, rows=sample_rows(cfg.V), all_rows_at=(1,))


@pytest.mark.timeout(600)
def test_rowonly_full_embed128k_sparse_bf16(em):
    cfg = wl.CONFIGS["embed128k"]
    sparse_lockstep(em, cfg, seed=13, steps=4)


@pytest.mark.timeout(900)
def test_rowonly_full_wide262k_bf16(em):
    cfg = wl.CONFIGS["wide262k"]
    dense_lockstep(em, cfg, seed=15, steps=3, rows=sample_rows(cfg.V, 512), all_rows_at=())
