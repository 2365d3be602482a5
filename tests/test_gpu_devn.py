"""GPU tests of the sparse steps whose row count lives in device memory, of the
token -> coalesce -> step path built on them, and of HIP-graph capture of the
steps.

* Parity: the step with a device count against the oracle's sparse step on
  the same (coalesced) rows, with the tolerances of test_gpu_parity.
* With the count equal to its maximum the result is bit-identical to the
  host-count step (same row partition).
* A count outside [0, max] and a coalescing index error (which writes n = -1)
  leave the table untouched and are reported by ember_get_error.
* Graph capture: a captured step replayed on fresh inputs gives the same bits
  as the same step run eagerly, replay after replay, with eager work and
  synchronisations in between.
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


def _tables_equal(a, b):
    assert torch.equal(a[0].view(torch.int16) if a[0].dtype == torch.bfloat16 else a[0],
                       b[0].view(torch.int16) if b[0].dtype == torch.bfloat16 else b[0])
    assert torch.equal(a[1], b[1])
    if a[2] is not None:
        assert torch.equal(a[2], b[2])


@pytest.mark.parametrize("row_only", [False, True])
def test_token_steps_match_the_oracle(em, row_only):
    cfg = wl.Config("devn", 5000, 320, torch.bfloat16, torch.bfloat16, 3, "sparse_zipf", batch_tokens=3000)
    print(f"tokens -> step, row_only={row_only}", flush=True)
    W = wl.make_weights(cfg, seed=40, device=DEV)
    tab = em.EmberTable(cfg.V, cfg.D, device=DEV, row_only=row_only)
    co = em.Coalescer(cfg.batch_tokens, cfg.V, cfg.D, device=DEV)
    r_o = np.zeros(cfg.V, np.float32)
    c_o = None if row_only else np.zeros(cfg.D, np.float32)
    for t in range(1, cfg.steps + 1):
        tok, U = wl.make_token_batch(cfg, t, seed=40, device=DEV)
        W_prev = host_bits(W)
        r_prev = tab.r.cpu().numpy()
        tab.step_tokens(W, tok, U, co)
        assert em.ember_get_error(co.ws) == em.EMBER_OK
        assert em.ember_get_error(tab.ws) == em.EMBER_OK
        n = int(co.n_out.item())
        idx_h = co.idx[:n].cpu().numpy()
        G_h = host_bits(co.G_rows[:n])
        # the coalesced rows are the oracle's up to rounding boundaries (see
        # test_gpu_coalesce); the step is checked on the rows it was given
        assert np.array_equal(idx_h, np.unique(tok.cpu().numpy()))
        W_ref = W_prev.copy()
        assert oracle.step(W_ref, G_h, r_o, c_o, t, idx=idx_h, w_rows=idx_h, row_only=row_only) == 0
        check_state(tab.r, r_o, f"r step {t}")
        if not row_only:
            check_state(tab.c, c_o, f"c step {t}")
        W_gpu = host_bits(W)
        check_w(W_gpu[idx_h], W_ref[idx_h], W_prev[idx_h], f"W step {t}")
        mask = np.ones(cfg.V, bool)
        mask[idx_h] = False
        assert np.array_equal(W_gpu[mask], W_prev[mask])
        assert np.array_equal(tab.r.cpu().numpy()[mask], np.float32(B2) * r_prev[mask])


@pytest.mark.parametrize("row_only", [False, True])
def test_full_count_is_bitwise_the_host_count_step(em, row_only):
    cfg = wl.Config("devn_eq", 20000, 1024, torch.bfloat16, torch.bfloat16, 2, "sparse_zipf", batch_tokens=4000)
    outs = []
    for use_dev in (False, True):
        W = wl.make_weights(cfg, seed=41, device=DEV)
        tab = em.EmberTable(cfg.V, cfg.D, device=DEV, row_only=row_only)
        for t in (1, 2):
            idx, Gr = wl.make_sparse_batch(cfg, t, seed=41, device=DEV, shuffle=True)
            if use_dev:
                n_dev = torch.tensor([idx.numel()], dtype=torch.int64, device=DEV)
                em.ember_step_sparse_rows_devn(W, Gr, idx, n_dev, tab.r, tab.c, t, LR, B2, EPS, False, tab.ws,
                                               row_only=row_only)
            else:
                tab.t = t - 1
                tab.step_sparse_rows(W, Gr, idx)
            assert em.ember_get_error(tab.ws) == em.EMBER_OK
        outs.append((W, tab.r, tab.c))
    _tables_equal(outs[0], outs[1])


def test_count_decides_the_form_on_the_device(em):
    # a maximum of 8192 rows, more than the one-launch form holds at D = 4096
    # bf16 (20 rows per block, 5120 in all): a count that fits takes that form
    # (marked in the workspace word after the status words), a larger one the
    # three launches; the result is the host-count step's, bit for bit, where
    # the partitions agree (a count that fits, or the maximum itself)
    V, D, max_rows = 20000, 4096, 8192
    cfg = wl.Config("devn_choice", V, D, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf", batch_tokens=max_rows)
    rng = np.random.default_rng(43)
    W_dev = wl.make_weights(cfg, seed=43, device=DEV)
    W_host = W_dev.clone()
    A = em.EmberTable(V, D, device=DEV)
    B = em.EmberTable(V, D, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(43)
    counts = [3000, max_rows, 100, 5120, 0, max_rows, 5121]
    for t, n in enumerate(counts, start=1):
        print(f"device-count step t={t} n={n} max={max_rows}", flush=True)
        ids = rng.permutation(V)[:max_rows].astype(np.int64)
        idx = torch.from_numpy(ids).to(DEV)
        Gr = (torch.randn(max_rows, D, generator=g, device=DEV) * 1e-3).to(torch.bfloat16)
        n_dev = torch.tensor([n], dtype=torch.int64, device=DEV)
        em.ember_step_sparse_rows_devn(W_dev, Gr, idx, n_dev, A.r, A.c, t, LR, B2, EPS, False, A.ws)
        assert em.ember_get_error(A.ws) == em.EMBER_OK
        taken = int(A.ws[28:32].view(torch.int32).item())
        assert taken == (1 if n <= 5120 else 0), f"n={n}: taken={taken}"
        em.ember_step_sparse_rows(W_host, Gr[:n], idx[:n], B.r, B.c, t, LR, B2, EPS, False, B.ws)
        assert em.ember_get_error(B.ws) == em.EMBER_OK
        if n <= 5120 or n == max_rows:
            _tables_equal((W_dev, A.r, A.c), (W_host, B.r, B.c))
        else:
            # other partitions of the same rows: the same step up to rounding
            assert torch.allclose(A.r, B.r, rtol=1e-5, atol=0)
            assert torch.allclose(A.c, B.c, rtol=1e-5, atol=0)
            assert torch.allclose(W_dev.float(), W_host.float(), rtol=1e-2, atol=1e-6)
    # a count outside [0, max]: the one-launch kernel takes it as a refused
    # step (the table is left alone, the index error reported), and the next
    # valid count steps normally
    before = (W_dev.clone(), A.r.clone(), A.c.clone())
    for bad in (-1, max_rows + 1):
        n_dev = torch.tensor([bad], dtype=torch.int64, device=DEV)
        em.ember_step_sparse_rows_devn(W_dev, Gr, idx, n_dev, A.r, A.c, len(counts) + 1, LR, B2, EPS, False, A.ws)
        assert em.ember_get_error(A.ws) == em.EMBER_ERR_INDEX
        assert int(A.ws[28:32].view(torch.int32).item()) == 1
        _tables_equal(before, (W_dev, A.r, A.c))
    n_dev = torch.tensor([2000], dtype=torch.int64, device=DEV)
    em.ember_step_sparse_rows_devn(W_dev, Gr, idx, n_dev, A.r, A.c, len(counts) + 1, LR, B2, EPS, False, A.ws)
    assert em.ember_get_error(A.ws) == em.EMBER_OK


@pytest.mark.parametrize("row_only", [False, True])
def test_bad_counts_and_coalescing_errors_leave_the_table_untouched(em, row_only):
    V, D = 1000, 128
    cfg = wl.Config("devn_err", V, D, torch.bfloat16, torch.bfloat16, 1, "normal")
    W = wl.make_weights(cfg, seed=42, device=DEV)
    tab = em.EmberTable(V, D, device=DEV, row_only=row_only)
    idx = torch.tensor([3, 7, 500, 8], dtype=torch.int64, device=DEV)
    Gr = (torch.randn(4, D, device=DEV) * 1e-3).to(torch.bfloat16)
    before = (W.clone(), tab.r.clone(), None if row_only else tab.c.clone())
    for bad in (5, -1):
        n_dev = torch.tensor([bad], dtype=torch.int64, device=DEV)
        em.ember_step_sparse_rows_devn(W, Gr, idx, n_dev, tab.r, tab.c, 1, LR, B2, EPS, False, tab.ws,
                                       row_only=row_only)
        assert em.ember_get_error(tab.ws) == em.EMBER_ERR_INDEX
        _tables_equal((W, tab.r, tab.c), before)
    # a token outside [0, V): coalescing reports it, writes n = -1, the step refuses it
    co = em.Coalescer(16, V, D, device=DEV)
    tok = torch.tensor([1, 2, V, 2], dtype=torch.int64, device=DEV)
    U = (torch.randn(4, D, device=DEV) * 1e-3).to(torch.bfloat16)
    tab.step_tokens(W, tok, U, co)
    assert em.ember_get_error(co.ws) == em.EMBER_ERR_INDEX
    assert em.ember_get_error(tab.ws) == em.EMBER_ERR_INDEX
    _tables_equal((W, tab.r, tab.c), before)
    # and the next good step goes through
    n_dev = torch.tensor([4], dtype=torch.int64, device=DEV)
    em.ember_step_sparse_rows_devn(W, Gr, idx, n_dev, tab.r, tab.c, 1, LR, B2, EPS, False, tab.ws, row_only=row_only)
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    assert not torch.equal(W.view(torch.int16), before[0].view(torch.int16))


@pytest.mark.parametrize("row_only", [False, True])
def test_captured_steps_replay_bitwise(em, row_only):
    """One HIP graph holding a dense step of an LM head and a token -> coalesce ->
    sparse step of an embedding, replayed on fresh inputs; each replay must give
    the bits of the same steps run eagerly on a twin set of tables."""
    Vh, Dh, P = 8192, 512, 2048
    head_cfg = wl.Config("g_head", Vh, Dh, torch.bfloat16, torch.bfloat16, 1, "zipf_rows")
    emb_cfg = wl.Config("g_emb", Vh, Dh, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf", batch_tokens=P)
    print(f"graph capture, row_only={row_only}", flush=True)

    def tables():
        return (wl.make_weights(head_cfg, seed=43, device=DEV), wl.make_weights(emb_cfg, seed=44, device=DEV),
                em.EmberTable(Vh, Dh, device=DEV, row_only=row_only),
                em.EmberTable(Vh, Dh, device=DEV, row_only=row_only),
                em.Coalescer(P, Vh, Dh, device=DEV))

    Wh, We, th, te, co = tables()
    Wh2, We2, th2, te2, co2 = tables()
    G_static = torch.empty(Vh, Dh, dtype=torch.bfloat16, device=DEV)
    tok_static = torch.empty(P, dtype=torch.int64, device=DEV)
    U_static = torch.empty(P, Dh, dtype=torch.bfloat16, device=DEV)
    t_fixed = 5   # the step counter is a launch argument: a captured step keeps its t

    def steps(Wh_, We_, th_, te_, co_, G, tok, U):
        th_.t = te_.t = t_fixed - 1
        th_.step(Wh_, G)
        te_.step_tokens(We_, tok, U, co_)

    # warm up on a side stream (first launches load the code objects), then capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        G0 = wl.make_dense_grad(head_cfg, 1, seed=45, device=DEV)
        tok0, U0 = wl.make_token_batch(emb_cfg, 1, seed=45, device=DEV)
        G_static.copy_(G0)
        tok_static.copy_(tok0)
        U_static.copy_(U0)
        steps(Wh, We, th, te, co, G_static, tok_static, U_static)
        steps(Wh2, We2, th2, te2, co2, G0, tok0, U0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    _tables_equal((Wh, th.r, th.c), (Wh2, th2.r, th2.c))
    _tables_equal((We, te.r, te.c), (We2, te2.r, te2.c))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        steps(Wh, We, th, te, co, G_static, tok_static, U_static)
    for rep in range(2, 5):
        G = wl.make_dense_grad(head_cfg, rep, seed=45, device=DEV)
        tok, U = wl.make_token_batch(emb_cfg, rep, seed=45, device=DEV)
        G_static.copy_(G)
        tok_static.copy_(tok)
        U_static.copy_(U)
        graph.replay()
        steps(Wh2, We2, th2, te2, co2, G, tok, U)   # eager twin
        torch.cuda.synchronize()
        assert em.ember_get_error(te.ws) == em.EMBER_OK and em.ember_get_error(co.ws) == em.EMBER_OK
        _tables_equal((Wh, th.r, th.c), (Wh2, th2.r, th2.c))
        _tables_equal((We, te.r, te.c), (We2, te2.r, te2.c))


def test_captured_count_choice_replays_bitwise(em):
    """A captured device-count step whose maximum (8192 rows at D = 4096 bf16)
    is beyond the one-launch form: each replay decides the form from the count
    it finds (3000 and 100 rows fit, 8192 and 5121 do not) and must give the
    bits of the same step run eagerly on a twin table."""
    V, D, max_rows = 20000, 4096, 8192
    cfg = wl.Config("g_choice", V, D, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf", batch_tokens=max_rows)
    W = wl.make_weights(cfg, seed=47, device=DEV)
    W2 = W.clone()
    A = em.EmberTable(V, D, device=DEV)
    B = em.EmberTable(V, D, device=DEV)
    idx_s = torch.empty(max_rows, dtype=torch.int64, device=DEV)
    G_s = torch.empty(max_rows, D, dtype=torch.bfloat16, device=DEV)
    n_s = torch.zeros(1, dtype=torch.int64, device=DEV)
    rng = np.random.default_rng(47)
    g = torch.Generator(device=DEV).manual_seed(47)
    t_fixed = 3   # the step counter is a launch argument: a captured step keeps its t

    def inputs(n):
        idx = torch.from_numpy(rng.permutation(V)[:max_rows].astype(np.int64)).to(DEV)
        G = (torch.randn(max_rows, D, generator=g, device=DEV) * 1e-3).to(torch.bfloat16)
        return idx, G, torch.tensor([n], dtype=torch.int64, device=DEV)

    def step(W_, T, idx, G, n):
        em.ember_step_sparse_rows_devn(W_, G, idx, n, T.r, T.c, t_fixed, LR, B2, EPS, False, T.ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        idx0, G0, n0 = inputs(3000)
        idx_s.copy_(idx0)
        G_s.copy_(G0)
        n_s.copy_(n0)
        step(W, A, idx_s, G_s, n_s)
        step(W2, B, idx0, G0, n0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    _tables_equal((W, A.r, A.c), (W2, B.r, B.c))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(W, A, idx_s, G_s, n_s)
    for n in (8192, 100, 5121, 3000, 8192):
        print(f"graph replay with n={n}", flush=True)
        idx, G, nd = inputs(n)
        idx_s.copy_(idx)
        G_s.copy_(G)
        n_s.copy_(nd)
        graph.replay()
        step(W2, B, idx, G, nd)   # eager twin
        torch.cuda.synchronize()
        assert em.ember_get_error(A.ws) == em.EMBER_OK and em.ember_get_error(B.ws) == em.EMBER_OK
        assert int(A.ws[28:32].view(torch.int32).item()) == (1 if n <= 5120 else 0)
        _tables_equal((W, A.r, A.c), (W2, B.r, B.c))
