"""The sparse step without a workspace (ember_step_sparse_rows_static): its
scratch is the library's own array.  Checked against ember_step_sparse_rows
(the same one-launch kernel with a caller workspace) on twin tables: W, r, c
and the status must be the same bits, on two calls in a row whose second
table is smaller than the first; then an index error and the call after it.
Host-side limits are checked without a GPU."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_01455_amd import workloads as wl


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


def _args(em, W, G, idx, r, c, status, V=None, D=None):
    Vw, Dw = W.shape
    return (W.data_ptr(), em.EMBER_BF16, Dw, G.data_ptr() if G.numel() else None, em.EMBER_BF16, Dw,
            idx.data_ptr() if idx.numel() else None, idx.numel(), r.data_ptr(), c.data_ptr(),
            Vw if V is None else V, Dw if D is None else D, 1, 1e-3, 0.999, 1e-8, 0, status, None)


def test_static_step_rejects_sizes_and_arguments_on_host(em):
    """Checks that run before anything is enqueued (no device is touched)."""
    W = torch.zeros(16, 64, dtype=torch.bfloat16)
    G = torch.zeros(4, 64, dtype=torch.bfloat16)
    idx = torch.zeros(4, dtype=torch.int64)
    r, c = torch.zeros(16), torch.zeros(64)
    st = ctypes.c_int32(0)
    status = ctypes.addressof(st)
    f = em.LIB.ember_step_sparse_rows_static
    # scratch: 4 V bytes of row marks alone exceed 16 MiB
    assert f(*_args(em, W, G, idx, r, c, status, V=5_000_000)) == em.EMBER_ERR_WORKSPACE
    # 1028 D bytes of partial sums and column factors exceed 16 MiB
    Ww = torch.zeros(16, 20000, dtype=torch.bfloat16)
    Gw = torch.zeros(4, 20000, dtype=torch.bfloat16)
    cw = torch.zeros(20000)
    assert f(*_args(em, Ww, Gw, idx, r, cw, status)) == em.EMBER_ERR_WORKSPACE
    assert f(*_args(em, W, G, idx, r, c, None)) == em.EMBER_ERR_ARG
    assert f(*_args(em, W, G, idx, r, c, status + 2)) == em.EMBER_ERR_ALIGN
    bad = list(_args(em, W, G, idx, r, c, status))
    bad[12] = 0   # t
    assert f(*bad) == em.EMBER_ERR_ARG


def _twin_tables(em, V, D, seed):
    cfg = wl.Config("noalloc", V, D, torch.bfloat16, torch.bfloat16, 1, "sparse_zipf", batch_tokens=3 * V // 4)
    W1 = wl.make_weights(cfg, seed=seed, device="cuda")
    W2 = W1.clone()
    tab = em.EmberTable(V, D, device="cuda")
    r = torch.zeros(V, device="cuda")
    c = torch.zeros(D, device="cuda")
    return cfg, W1, W2, tab, r, c


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.gpu
def test_static_step_matches_the_workspace_step(em):
    status = torch.full((1,), 77, dtype=torch.int32, device="cuda")
    for V, D, seed in ((20000, 1024, 61), (5000, 512, 62)):   # the second table is smaller
        print(f"static scratch step V={V} D={D}", flush=True)
        cfg, W1, W2, tab, r, c = _twin_tables(em, V, D, seed)
        for t in (1, 2):
            idx, G = wl.make_sparse_batch(cfg, t, seed=seed, device="cuda", shuffle=True)
            tab.step_sparse_rows(W1, G, idx)
            em.ember_step_sparse_rows_static(W2, G, idx, r, c, t, status)
            torch.cuda.synchronize()
            assert em.ember_get_error(tab.ws) == em.EMBER_OK
            assert int(status.item()) == 0
            assert torch.equal(_bits(W1), _bits(W2)), "W differs from the workspace step"
            assert torch.equal(_bits(tab.r), _bits(r)), "r differs from the workspace step"
            assert torch.equal(_bits(tab.c), _bits(c)), "c differs from the workspace step"
            assert not torch.equal(_bits(W2), _bits(wl.make_weights(cfg, seed=seed, device="cuda")))
    # an index error: nothing changes and the status says so; the next call is clean
    before = (W2.clone(), r.clone(), c.clone())
    idx_bad = torch.tensor([3, 7, 7], dtype=torch.int64, device="cuda")
    Gb = torch.ones(3, D, dtype=torch.bfloat16, device="cuda")
    em.ember_step_sparse_rows_static(W2, Gb, idx_bad, r, c, 3, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 2
    for a, b in zip((W2, r, c), before):
        assert torch.equal(_bits(a), _bits(b))
    idx_ok = torch.tensor([3, 7, 9], dtype=torch.int64, device="cuda")
    tab.step_sparse_rows(W1, Gb, idx_ok)
    em.ember_step_sparse_rows_static(W2, Gb, idx_ok, r, c, 3, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(_bits(W1), _bits(W2)) and torch.equal(_bits(tab.r), _bits(r))
