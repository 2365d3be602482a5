"""The failure path of the one-launch sparse step, forced from the host: with
the bound of its grid-barrier waits cut to one tick of the real-time counter
the blocks that wait time out (every wait still ends, every access stays in
bounds), the launch ends normally, and ember_get_error reports
EMBER_ERR_DEVICE until ember_init_state; after that the table steps exactly
as a fresh one does."""
import numpy as np
import pytest
import torch

from paper_2607_01455_amd import workloads as wl
from parity_checks import DEV, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


def _batch(V, D, n, seed):
    gen = torch.Generator().manual_seed(seed)
    idx = torch.randperm(V, generator=gen)[:n].sort().values
    G = (torch.randn(n, D, generator=gen) * 1e-3).to(torch.bfloat16)
    return idx.to(DEV), G.to(DEV)


def test_barrier_timeout_is_reported_and_cleared_by_init(em):
    V, D, n = 20000, 4096, 1500          # the one-launch form
    print(f"barrier timeout V={V} D={D} n={n}", flush=True)
    cfg = wl.Config("timeout", V, D, torch.bfloat16, torch.bfloat16, 3, "normal")
    W0 = wl.make_weights(cfg, seed=7, device=DEV)
    batches = [_batch(V, D, n, 7 + k) for k in range(3)]

    W = W0.clone()
    tab = em.EmberTable(V, D, device=DEV)
    tab.step_sparse_rows(W, *reversed(batches[0]))
    torch.cuda.synchronize()
    assert em.ember_get_error(tab.ws) == em.EMBER_OK

    em.ember_set_barrier_wait_ticks(1)
    try:
        tab.step_sparse_rows(W, *reversed(batches[1]))
        torch.cuda.synchronize()
    finally:
        em.ember_set_barrier_wait_ticks(0)
    assert em.ember_get_error(tab.ws) == em.EMBER_ERR_DEVICE
    # the report stays until the state is initialised again
    tab.step_sparse_rows(W, *reversed(batches[2]))
    torch.cuda.synchronize()
    assert em.ember_get_error(tab.ws) == em.EMBER_ERR_DEVICE

    # re-initialised, the table steps as a fresh one does
    em.ember_init_state(tab.r, tab.c, tab.ws)
    tab.t = 0
    W.copy_(W0)
    fresh_W = W0.clone()
    fresh = em.EmberTable(V, D, device=DEV)
    for b in batches:
        tab.step_sparse_rows(W, *reversed(b))
        fresh.step_sparse_rows(fresh_W, *reversed(b))
    torch.cuda.synchronize()
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    assert np.array_equal(host_bits(W), host_bits(fresh_W))
    assert torch.equal(tab.r, fresh.r) and torch.equal(tab.c, fresh.c)
