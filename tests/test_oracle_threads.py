"""The oracle's loops may run on several threads (row ranges, column ranges);
every float64 sum keeps its order, so the results must be the same bits for
any thread count.  Checked at 1 thread and at every core, on dense, sparse
and row-only steps in fp32 and bf16, and on the LM-head gradient."""
import os

import numpy as np
import pytest

import oracle


def _bits(a):
    return a.view(np.uint32) if a.dtype == np.float32 else a


def _inputs(rng, V, D, dtype):
    if dtype == np.float32:
        W = (rng.standard_normal((V, D)) * 0.02).astype(np.float32)
        G = (rng.standard_normal((V, D)) * 1e-3 * rng.lognormal(0, 2, (V, 1))).astype(np.float32)
    else:
        W = (rng.standard_normal((V, D)).astype(np.float32) * 0.02).view(np.uint32)
        W = (W >> 16).astype(np.uint16)
        G = (rng.standard_normal((V, D)).astype(np.float32) * 1e-3).view(np.uint32)
        G = (G >> 16).astype(np.uint16)
    return W, G


def _run(threads, W, G, steps, idx=None, row_only=False):
    oracle.set_threads(threads)
    W = W.copy()
    V, D = W.shape
    r = np.zeros(V, np.float32)
    c = None if row_only else np.zeros(D, np.float32)
    for t in range(1, steps + 1):
        Gt = G if idx is None else G[: len(idx)]
        assert oracle.step(W, Gt, r, c, t, idx=idx, row_only=row_only) == 0
    return W, r, c


@pytest.fixture(autouse=True)
def _restore_threads():
    n = oracle.set_threads(0)
    yield
    oracle.set_threads(n)


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
@pytest.mark.parametrize("kind", ["dense", "sparse", "row_only"])
def test_results_do_not_depend_on_the_thread_count(dtype, kind):
    rng = np.random.default_rng(7)
    V, D = 1537, 333          # ragged against every chunk the loops use
    W, G = _inputs(rng, V, D, dtype)
    idx = rng.permutation(V)[:400].astype(np.int64) if kind == "sparse" else None
    many = max(2, os.cpu_count() or 2)
    one = _run(1, W, G, 3, idx=idx, row_only=kind == "row_only")
    all_ = _run(many, W, G, 3, idx=idx, row_only=kind == "row_only")
    for a, b in zip(one, all_):
        if a is not None:
            assert np.array_equal(_bits(a), _bits(b))


def test_lmhead_gradient_does_not_depend_on_the_thread_count():
    rng = np.random.default_rng(8)
    T, V, D = 37, 301, 67
    dY = (rng.standard_normal((T, V)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    H = (rng.standard_normal((T, D)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    oracle.set_threads(1)
    g1 = oracle.lmhead_grad(dY, H)
    oracle.set_threads(max(2, os.cpu_count() or 2))
    gn = oracle.lmhead_grad(dY, H)
    assert np.array_equal(g1, gn)
