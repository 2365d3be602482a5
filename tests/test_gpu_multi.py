"""GPU tests of ember_step_multi: the canonical steps of several tables enqueued
as three launches in all.

Each table's W, r and c must equal, bit for bit, what its own
ember_step_dense / ember_step_sparse_rows call produces on the same inputs:
the multi-table launches give each table the same row blocks, slabs and
reduction orders as its own launches.  Those single-table calls are checked
against the oracle in test_gpu_parity; here one lockstep case also checks the
multi-table results against the oracle directly (tolerances as stated there).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01455_amd import workloads as wl
from parity_checks import B2, DEV, EPS, LR, check_state, check_w, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


def _bits_equal(a: torch.Tensor, b: torch.Tensor) -> bool:
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


class Spec:
    """One table of a test: shape, dtypes, step kind and scalars."""

    def __init__(self, name, V, D, dtype, sparse=False, batch_tokens=0, lr=LR, beta2=B2, eps=EPS,
                 maximize=False, empty=False, row_only=False):
        grad = "sparse_zipf" if sparse else "zipf_rows"
        self.cfg = wl.Config(name, V, D, dtype, dtype, 3, grad, batch_tokens=batch_tokens)
        self.sparse, self.empty, self.row_only = sparse, empty, row_only
        self.lr, self.beta2, self.eps, self.maximize = lr, beta2, eps, maximize


def _tables(em, spec, seed):
    """Two identical (table state, W) pairs: one for the multi-table call, one
    for the single-table calls."""
    out = []
    for _ in range(2):
        tab = em.EmberTable(spec.cfg.V, spec.cfg.D, device=DEV, lr=spec.lr, beta2=spec.beta2, eps=spec.eps,
                            maximize=spec.maximize, row_only=spec.row_only)
        out.append((tab, wl.make_weights(spec.cfg, seed=seed, device=DEV)))
    return out


def _grad(spec, t, seed, scales):
    if not spec.sparse:
        return wl.make_dense_grad(spec.cfg, t, seed=seed, device=DEV, scales=scales), None
    if spec.empty:
        return (torch.empty(0, spec.cfg.D, dtype=spec.cfg.g_dtype, device=DEV),
                torch.empty(0, dtype=torch.int64, device=DEV))
    idx, G = wl.make_sparse_batch(spec.cfg, t, seed=seed, device=DEV, shuffle=True)
    return G, idx


def _single(em, tab, W, G, idx):
    if idx is None:
        tab.step(W, G)
    else:
        tab.step_sparse_rows(W, G, idx)


def _run_against_single_calls(em, specs, steps, seed=0):
    print("multi vs single:", ", ".join(f"{s.cfg.name} {s.cfg.V}x{s.cfg.D}" for s in specs), flush=True)
    pairs = [_tables(em, s, seed + k) for k, s in enumerate(specs)]
    scales = [wl.row_scales(s.cfg, seed + k, DEV) if not s.sparse else None for k, s in enumerate(specs)]
    for t in range(1, steps + 1):
        grads = [_grad(s, t, seed + k, scales[k]) for k, s in enumerate(specs)]
        items = []
        for (multi, single), (G, idx) in zip(pairs, grads):
            items.append((multi[0], multi[1], G) if idx is None else (multi[0], multi[1], G, idx))
        em.step_tables(items)
        for (multi, single), (G, idx) in zip(pairs, grads):
            _single(em, single[0], single[1], G, idx)
        torch.cuda.synchronize()
        for s, (multi, single) in zip(specs, pairs):
            assert multi[0].t == single[0].t == t
            assert em.ember_get_error(multi[0].ws) == em.EMBER_OK
            what = f"{s.cfg.name} step {t}"
            assert _bits_equal(multi[1], single[1]), f"{what}: W differs from the single-table step"
            assert _bits_equal(multi[0].r, single[0].r), f"{what}: r differs"
            if not s.row_only:
                assert _bits_equal(multi[0].c, single[0].c), f"{what}: c differs"
    return pairs


def test_mixed_tables_match_single_table_steps_bitwise(em):
    # bf16 and fp32 tables (two launch groups), ragged widths, sparse tables with
    # shuffled ids and with no rows, per-table scalars, lr = 0 and ascent
    specs = [
        Spec("dense_bf16", 3000, 1000, torch.bfloat16),
        Spec("sparse_bf16", 5000, 4096, torch.bfloat16, sparse=True, batch_tokens=2048),
        Spec("dense_f32", 700, 260, torch.float32, beta2=0.99, maximize=True),
        Spec("sparse_f32_empty", 300, 64, torch.float32, sparse=True, empty=True),
        Spec("dense_bf16_lr0", 100, 64, torch.bfloat16, lr=0.0),
        Spec("sparse_f32", 2000, 96, torch.float32, sparse=True, batch_tokens=512, eps=1e-6),
    ]
    _run_against_single_calls(em, specs, steps=3)


def test_row_only_tables_match_single_table_steps_bitwise(em):
    # row-only tables (Section 2.1) beside canonical ones: dense and sparse, bf16
    # and fp32, shuffled ids, an empty sparse table, rows long enough for the
    # block-per-row kernel (D = 16384 bf16: 2048 chunks)
    specs = [
        Spec("ro_dense_bf16", 3000, 1000, torch.bfloat16, row_only=True),
        Spec("ro_sparse_bf16", 5000, 4096, torch.bfloat16, sparse=True, batch_tokens=2048, row_only=True),
        Spec("canon_dense_bf16", 2000, 512, torch.bfloat16),
        Spec("ro_sparse_f32_empty", 300, 64, torch.float32, sparse=True, empty=True, row_only=True),
        Spec("ro_dense_f32", 700, 260, torch.float32, beta2=0.99, maximize=True, row_only=True),
        Spec("ro_long_rows", 300, 16384, torch.bfloat16, sparse=True, batch_tokens=200, row_only=True),
        Spec("canon_sparse_bf16", 4000, 1024, torch.bfloat16, sparse=True, batch_tokens=900),
    ]
    _run_against_single_calls(em, specs, steps=3, seed=7)


def test_full_size_row_only_tables(em):
    """The benchmarked pair as row-only tables, bitwise against single calls."""
    specs = [Spec("ro_lmhead128k", 128256, 4096, torch.bfloat16, row_only=True),
             Spec("ro_embed128k", 128256, 4096, torch.bfloat16, sparse=True, batch_tokens=8 * 2048, row_only=True)]
    _run_against_single_calls(em, specs, steps=2, seed=9)


def test_eight_tables_in_one_call(em):
    specs = [Spec(f"t{k}", 64 * (k + 1) + 3, 8 * (k + 1) * 8, torch.bfloat16, sparse=(k % 3 == 1),
                  batch_tokens=50) for k in range(em.EMBER_MAX_TABLES)]
    _run_against_single_calls(em, specs, steps=2)


def test_multi_table_lockstep_with_oracle(em):
    """Dense and sparse bf16 tables in one call, every element against the
    oracle in lockstep (the oracle starts each step from the GPU's W)."""
    dense = wl.Config("dense", 2500, 1096, torch.bfloat16, torch.bfloat16, 3, "zipf_rows")
    sparse = wl.Config("sparse", 3000, 520, torch.bfloat16, torch.bfloat16, 3, "sparse_zipf", batch_tokens=1500)
    Wd = wl.make_weights(dense, seed=1, device=DEV)
    Ws = wl.make_weights(sparse, seed=2, device=DEV)
    td = em.EmberTable(dense.V, dense.D, device=DEV)
    ts = em.EmberTable(sparse.V, sparse.D, device=DEV)
    ro = {k: (np.zeros(c.V, np.float32), np.zeros(c.D, np.float32)) for k, c in (("d", dense), ("s", sparse))}
    scales = wl.row_scales(dense, 1, DEV)
    for t in (1, 2, 3):
        print(f"multi lockstep step {t}", flush=True)
        Gd = wl.make_dense_grad(dense, t, seed=1, device=DEV, scales=scales)
        idx, Gs = wl.make_sparse_batch(sparse, t, seed=2, device=DEV, shuffle=True)
        Wd_prev, Ws_prev = host_bits(Wd), host_bits(Ws)
        r_prev = ts.r.cpu().numpy()
        em.step_tables([(td, Wd, Gd), (ts, Ws, Gs, idx)])
        torch.cuda.synchronize()
        Wd_ref = Wd_prev.copy()
        assert oracle.step(Wd_ref, host_bits(Gd), ro["d"][0], ro["d"][1], t) == 0
        check_state(td.r, ro["d"][0], f"dense r step {t}")
        check_state(td.c, ro["d"][1], f"dense c step {t}")
        check_w(host_bits(Wd), Wd_ref, Wd_prev, f"dense W step {t}")
        idx_h = idx.cpu().numpy()
        Ws_ref = Ws_prev.copy()
        assert oracle.step(Ws_ref, host_bits(Gs), ro["s"][0], ro["s"][1], t, idx=idx_h) == 0
        check_state(ts.r, ro["s"][0], f"sparse r step {t}")
        check_state(ts.c, ro["s"][1], f"sparse c step {t}")
        got = host_bits(Ws)
        touched = np.sort(idx_h)
        check_w(got[touched], Ws_ref[touched], Ws_prev[touched], f"sparse W step {t}")
        mask = np.ones(sparse.V, bool)
        mask[touched] = False
        assert np.array_equal(got[mask], Ws_prev[mask]), "a row outside idx changed"
        assert np.array_equal(ts.r.cpu().numpy()[mask], np.float32(B2) * r_prev[mask])


def test_index_error_leaves_only_that_table_untouched(em):
    dense = Spec("dense", 900, 512, torch.bfloat16)
    sparse = Spec("sparse", 800, 512, torch.bfloat16, sparse=True, batch_tokens=300)
    (dm, ds), (sm, ss) = _tables(em, dense, 0), _tables(em, sparse, 1)
    for t in (1, 2):
        G, _ = _grad(dense, t, 0, None)
        Gs, idx = _grad(sparse, t, 1, None)
        bad = idx.clone()
        if t == 1:
            bad[-1] = bad[0]           # a repeated id: the sparse table must not step
        Ws_before, r_before, c_before = sm[1].clone(), sm[0].r.clone(), sm[0].c.clone()
        em.step_tables([(dm[0], dm[1], G), (sm[0], sm[1], Gs, bad)])
        _single(em, ds[0], ds[1], G, None)
        torch.cuda.synchronize()
        assert _bits_equal(dm[1], ds[1]) and _bits_equal(dm[0].r, ds[0].r) and _bits_equal(dm[0].c, ds[0].c)
        if t == 1:
            assert em.ember_get_error(sm[0].ws) == em.EMBER_ERR_INDEX
            assert _bits_equal(sm[1], Ws_before) and _bits_equal(sm[0].r, r_before)
            assert _bits_equal(sm[0].c, c_before)
            sm[0].t -= 1               # the caller does not advance t after an index error
        else:
            # the flag was cleared: a valid step after the failed one is the
            # first step of the single-table twin
            assert em.ember_get_error(sm[0].ws) == em.EMBER_OK
            _single(em, ss[0], ss[1], Gs, idx)
            torch.cuda.synchronize()
            assert _bits_equal(sm[1], ss[1]) and _bits_equal(sm[0].r, ss[0].r)
            assert _bits_equal(sm[0].c, ss[0].c)


def test_device_row_count_matches_the_single_call(em):
    sparse = Spec("sparse_devn", 4000, 1024, torch.bfloat16, sparse=True, batch_tokens=1200)
    dense = Spec("dense", 1000, 1024, torch.bfloat16)
    (sm, ss), (dm, ds) = _tables(em, sparse, 3), _tables(em, dense, 4)
    for t in (1, 2):
        Gs, idx = _grad(sparse, t, 3, None)
        G, _ = _grad(dense, t, 4, None)
        n = idx.numel()
        # the buffers hold more rows than the device count says
        idx_buf = torch.cat([idx, torch.full((37,), -1, dtype=torch.int64, device=DEV)])
        G_buf = torch.cat([Gs, torch.zeros(37, Gs.shape[1], dtype=Gs.dtype, device=DEV)])
        n_dev = torch.tensor([n], dtype=torch.int64, device=DEV)
        steps = [em.table_step(sm[1], G_buf, sm[0].r, sm[0].c, t, sm[0].ws, idx=idx_buf, n_idx_dev=n_dev),
                 em.table_step(dm[1], G, dm[0].r, dm[0].c, t, dm[0].ws)]
        em.ember_step_multi(steps, G)
        em.ember_step_sparse_rows_devn(ss[1], G_buf, idx_buf, n_dev, ss[0].r, ss[0].c, t, LR, B2, EPS, False,
                                       ss[0].ws)
        _single(em, ds[0], ds[1], G, None)
        torch.cuda.synchronize()
        assert em.ember_get_error(sm[0].ws) == em.EMBER_OK
        for a, b in ((sm[1], ss[1]), (sm[0].r, ss[0].r), (sm[0].c, ss[0].c), (dm[1], ds[1]), (dm[0].r, ds[0].r)):
            assert _bits_equal(a, b)


def test_full_size_lmhead_and_embedding_tables(em):
    """The benchmarked pair: the 128256 x 4096 bf16 LM head (dense) and input
    embedding (sparse rows, 8 x 2048 Zipf ids), two steps, bitwise against the
    single-table steps."""
    specs = [Spec("lmhead128k", 128256, 4096, torch.bfloat16),
             Spec("embed128k", 128256, 4096, torch.bfloat16, sparse=True, batch_tokens=8 * 2048)]
    _run_against_single_calls(em, specs, steps=2)


def test_captured_multi_step_replays_bitwise(em):
    """One HIP graph holding token -> coalesce and a multi-table call (dense
    LM head + device-count sparse embedding), replayed on fresh inputs; each
    replay must give the bits of single-table steps run eagerly on twins."""
    Vh, Dh, P = 8192, 512, 2048
    head_cfg = wl.Config("g_head", Vh, Dh, torch.bfloat16, torch.bfloat16, 1, "zipf_rows")
    emb_cfg = wl.Config("g_emb", Vh, Dh, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf", batch_tokens=P)
    print("graph capture of ember_step_multi", flush=True)

    def tables():
        return (wl.make_weights(head_cfg, seed=53, device=DEV), wl.make_weights(emb_cfg, seed=54, device=DEV),
                em.EmberTable(Vh, Dh, device=DEV), em.EmberTable(Vh, Dh, device=DEV),
                em.Coalescer(P, Vh, Dh, device=DEV))

    Wh, We, th, te, co = tables()
    Wh2, We2, th2, te2, co2 = tables()
    G_static = torch.empty(Vh, Dh, dtype=torch.bfloat16, device=DEV)
    tok_static = torch.empty(P, dtype=torch.int64, device=DEV)
    U_static = torch.empty(P, Dh, dtype=torch.bfloat16, device=DEV)
    t_fixed = 4   # the step counter is a launch argument: a captured step keeps its t

    def multi(G, tok, U):
        co.enqueue(tok, U)
        em.ember_step_multi([em.table_step(Wh, G, th.r, th.c, t_fixed, th.ws),
                             em.table_step(We, co.G_rows, te.r, te.c, t_fixed, te.ws, idx=co.idx,
                                           n_idx_dev=co.n_out)], G)

    def eager(G, tok, U):
        th2.t = te2.t = t_fixed - 1
        th2.step(Wh2, G)
        te2.step_tokens(We2, tok, U, co2)

    def check():
        assert em.ember_get_error(te.ws) == em.EMBER_OK and em.ember_get_error(co.ws) == em.EMBER_OK
        for a, b in ((Wh, Wh2), (th.r, th2.r), (th.c, th2.c), (We, We2), (te.r, te2.r), (te.c, te2.c)):
            assert _bits_equal(a, b)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        G0 = wl.make_dense_grad(head_cfg, 1, seed=55, device=DEV)
        tok0, U0 = wl.make_token_batch(emb_cfg, 1, seed=55, device=DEV)
        G_static.copy_(G0)
        tok_static.copy_(tok0)
        U_static.copy_(U0)
        multi(G_static, tok_static, U_static)
        eager(G0, tok0, U0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    check()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        multi(G_static, tok_static, U_static)
    for rep in range(2, 5):
        G = wl.make_dense_grad(head_cfg, rep, seed=55, device=DEV)
        tok, U = wl.make_token_batch(emb_cfg, rep, seed=55, device=DEV)
        G_static.copy_(G)
        tok_static.copy_(tok)
        U_static.copy_(U)
        graph.replay()
        eager(G, tok, U)
        torch.cuda.synchronize()
        check()
