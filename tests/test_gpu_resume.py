"""Checkpoint and resume: the optimizer's state is r, c and t alone (Algorithm
1 initialises r_0 = 0, c_0 = 0, t = 0 and carries nothing else), and the
workspace holds nothing between steps that ember_init_state does not reset.
So saving (W, r, c, t) after step k, restoring it into fresh tensors with a
fresh workspace and continuing must give the bits of an uninterrupted run:
dense, sparse-row (one-launch and three-launch forms) and row-only steps."""
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


def _inputs(cfg, steps, seed, rows):
    if rows:
        # rows distinct ids per step (the count decides the one- or three-launch form)
        gen = torch.Generator().manual_seed(seed)
        out = []
        for _ in range(steps):
            idx = torch.randperm(cfg.V, generator=gen)[:rows].sort().values
            G = (torch.randn(rows, cfg.D, generator=gen) * 1e-3).to(torch.bfloat16)
            out.append((idx.to(DEV), G.to(DEV)))
        return out
    sc = wl.row_scales(cfg, seed, DEV)
    return [wl.make_dense_grad(cfg, t + 1, seed=seed, device=DEV, scales=sc) for t in range(steps)]


def _take(em, tab, W, inp, sparse):
    if sparse:
        idx, G = inp
        tab.step_sparse_rows(W, G, idx)
    else:
        tab.step(W, inp)


def _state(tab, W):
    return (host_bits(W), tab.r.cpu().numpy().copy(), None if tab.c is None else tab.c.cpu().numpy().copy(), tab.t)


@pytest.mark.parametrize("kind,V,D,rows", [
    ("dense", 3000, 512, 0),
    ("sparse", 20000, 4096, 1500),     # the one-launch form
    ("sparse", 20000, 4096, 6000),     # beyond its 5120 rows at this width: three launches
    ("row_only", 3000, 520, 0),
])
def test_resume_from_saved_state_gives_the_same_bits(em, kind, V, D, rows):
    sparse = kind == "sparse"
    row_only = kind == "row_only"
    cfg = wl.Config("resume", V, D, torch.bfloat16, torch.bfloat16, 6, "normal")
    print(f"resume {kind} V={V} D={D} rows={rows}", flush=True)
    inputs = _inputs(cfg, 6, seed=V + D, rows=rows)
    W0 = wl.make_weights(cfg, seed=V + D, device=DEV)

    # uninterrupted: six steps
    W = W0.clone()
    tab = em.EmberTable(V, D, device=DEV, row_only=row_only)
    for k in range(6):
        _take(em, tab, W, inputs[k], sparse)
    torch.cuda.synchronize()
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    want = _state(tab, W)

    # interrupted after three steps: save to host memory, drop everything
    W = W0.clone()
    tab = em.EmberTable(V, D, device=DEV, row_only=row_only)
    for k in range(3):
        _take(em, tab, W, inputs[k], sparse)
    torch.cuda.synchronize()
    saved = _state(tab, W)
    del W, tab
    torch.cuda.synchronize()

    # restore into fresh tensors and a fresh workspace, continue three steps
    W = torch.from_numpy(saved[0].view(np.int16)).to(DEV).view(torch.bfloat16)
    tab = em.EmberTable(V, D, device=DEV, row_only=row_only)
    tab.r.copy_(torch.from_numpy(saved[1]))
    if saved[2] is not None:
        tab.c.copy_(torch.from_numpy(saved[2]))
    tab.t = saved[3]
    for k in range(3, 6):
        _take(em, tab, W, inputs[k], sparse)
    torch.cuda.synchronize()
    assert em.ember_get_error(tab.ws) == em.EMBER_OK
    got = _state(tab, W)

    assert got[3] == want[3] == 6
    assert np.array_equal(got[0], want[0]), "W differs after resuming"
    assert np.array_equal(got[1].view(np.uint32), want[1].view(np.uint32)), "r differs after resuming"
    if want[2] is not None:
        assert np.array_equal(got[2].view(np.uint32), want[2].view(np.uint32)), "c differs after resuming"
