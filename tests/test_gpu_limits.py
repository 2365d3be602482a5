"""GPU parity at the size limits of the C ABI: the largest row count (V =
EMBER_MAX_V), element offsets beyond 2^31, the widest rows (D = EMBER_MAX_D)
and the largest token batch of the coalescing step.  These catch 32-bit index
arithmetic and grid-size overflows that small shapes cannot show.

Checks follow the tolerances of test_gpu_parity; at these sizes W is compared
on the touched or sampled rows and the state on every element, chunk by
chunk.
"""
import numpy as np
import pytest
import torch

import oracle
from parity_checks import B2, DEV, EPS, LR, as_f64, check_coalesced_rows, check_w, host_bits

pytestmark = pytest.mark.gpu

MAX_V = 0x7FFFFFFE
MAX_D = 1 << 22


@pytest.fixture(scope="module")
def em():
    from paper_2607_01455_amd import ember
    return ember


def _fill_normal(t: torch.Tensor, std: float, seed: int, rows_per_chunk: int = 1 << 24):
    g = torch.Generator(device=DEV).manual_seed(seed)
    for r0 in range(0, t.shape[0], rows_per_chunk):
        r1 = min(t.shape[0], r0 + rows_per_chunk)
        t[r0:r1] = (torch.randn(r1 - r0, t.shape[1], generator=g, device=DEV) * std).to(t.dtype)


def _check_state_chunked(got: torch.Tensor, want: np.ndarray, what: str, chunk: int = 1 << 26):
    for i0 in range(0, want.size, chunk):
        g = got[i0:i0 + chunk].cpu().numpy().astype(np.float64)
        w = want[i0:i0 + chunk].astype(np.float64)
        bad = ~(np.abs(g - w) <= 1e-5 * np.abs(w))
        assert not bad.any(), f"{what}: {bad.sum()} elements out of 1e-5 near offset {i0}"


def _free():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("row_only", [False, True])
def test_sparse_step_at_the_largest_row_count(em, row_only):
    # V = 2^31 - 2 rows of 8 bf16 columns: W 34 GB; two sparse steps whose ids
    # include 0 and V - 1, so the decay pass, the row marks and the scatter all
    # reach the last row
    V, D = MAX_V, 8
    print(f"sparse step at V={V} D={D} row_only={row_only}", flush=True)
    W = torch.empty(V, D, dtype=torch.bfloat16, device=DEV)
    _fill_normal(W, 0.02, 1)
    r = torch.empty(V, dtype=torch.float32, device=DEV)
    c = None if row_only else torch.empty(D, dtype=torch.float32, device=DEV)
    ws = torch.empty(em.ember_workspace_bytes(V, D), dtype=torch.uint8, device=DEV)
    if row_only:
        em.ember_rowonly_init_state(r, D, ws)
    else:
        em.ember_init_state(r, c, ws)
    r_o = np.zeros(V, np.float32)
    c_o = None if row_only else np.zeros(D, np.float32)
    rng = np.random.default_rng(2)
    sets = [np.unique(np.concatenate([[0, V - 1, V // 2], rng.integers(0, V, 3000)])),
            np.unique(np.concatenate([[V - 1, 1], rng.integers(V - 5000, V, 2000)]))]
    for t, ids in enumerate(sets, start=1):
        ids = rng.permutation(ids).astype(np.int64)
        idx = torch.from_numpy(ids).to(DEV)
        Gr = (torch.randn(ids.size, D, generator=torch.Generator(device=DEV).manual_seed(t), device=DEV)
              * 1e-3).to(torch.bfloat16)
        rows = np.sort(ids)
        rows_t = torch.from_numpy(rows).to(DEV)
        prev = host_bits(W[rows_t])
        if row_only:
            em.ember_rowonly_step_sparse_rows(W, Gr, idx, r, t, LR, B2, EPS, False, ws)
        else:
            em.ember_step_sparse_rows(W, Gr, idx, r, c, t, LR, B2, EPS, False, ws)
        assert em.ember_get_error(ws) == em.EMBER_OK
        W_ref = np.empty((V, D), np.uint16)      # only the touched rows are written
        W_ref[rows] = prev
        assert oracle.step(W_ref, host_bits(Gr), r_o, c_o, t, idx=ids, w_rows=rows, row_only=row_only) == 0
        check_w(host_bits(W[rows_t]), W_ref[rows], prev, f"W step {t}")
        del W_ref
        _check_state_chunked(r, r_o, f"r step {t}")
        if not row_only:
            _check_state_chunked(c, c_o, f"c step {t}")
    del W, r, c, ws
    _free()


@pytest.mark.timeout(900)
def test_dense_step_with_element_offsets_beyond_2_31(em):
    # 600M x 4 fp32: offsets up to 2.4e9 elements
    V, D = 600_000_000, 4
    print(f"dense step at V={V} D={D}", flush=True)
    W = torch.empty(V, D, dtype=torch.float32, device=DEV)
    G = torch.empty(V, D, dtype=torch.float32, device=DEV)
    _fill_normal(W, 0.02, 3)
    _fill_normal(G, 1e-3, 4)
    r = torch.empty(V, dtype=torch.float32, device=DEV)
    c = torch.empty(D, dtype=torch.float32, device=DEV)
    ws = torch.empty(em.ember_workspace_bytes(V, D), dtype=torch.uint8, device=DEV)
    em.ember_init_state(r, c, ws)
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, V - 1], rng.integers(0, V, 4000), np.arange(V - 100, V)]))
    rows_t = torch.from_numpy(rows).to(DEV)
    prev = host_bits(W[rows_t])
    em.ember_step_dense(W, G, r, c, 1, LR, B2, EPS, False, ws)
    torch.cuda.synchronize()
    G_h = G.cpu().numpy()
    del G
    r_o, c_o = np.zeros(V, np.float32), np.zeros(D, np.float32)
    W_ref = np.empty((V, D), np.float32)
    W_ref[rows] = prev
    assert oracle.step(W_ref, G_h, r_o, c_o, 1, w_rows=rows) == 0
    del G_h
    check_w(host_bits(W[rows_t]), W_ref[rows], prev, "W")
    _check_state_chunked(r, r_o, "r")
    _check_state_chunked(c, c_o, "c")
    del W, r, c, ws, W_ref
    _free()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("row_only", [False, True])
def test_widest_rows_every_element(em, dtype, row_only):
    V, D = 5, MAX_D
    print(f"dense step at V={V} D={D} {dtype} row_only={row_only}", flush=True)
    W = torch.empty(V, D, dtype=dtype, device=DEV)
    G = torch.empty(V, D, dtype=dtype, device=DEV)
    _fill_normal(W, 0.02, 6)
    _fill_normal(G, 1e-3, 7)
    r = torch.empty(V, dtype=torch.float32, device=DEV)
    c = None if row_only else torch.empty(D, dtype=torch.float32, device=DEV)
    ws = torch.empty(em.ember_workspace_bytes(V, D), dtype=torch.uint8, device=DEV)
    if row_only:
        em.ember_rowonly_init_state(r, D, ws)
    else:
        em.ember_init_state(r, c, ws)
    r_o = np.zeros(V, np.float32)
    c_o = None if row_only else np.zeros(D, np.float32)
    for t in (1, 2):
        prev = host_bits(W)
        if row_only:
            em.ember_rowonly_step_dense(W, G, r, t, LR, B2, EPS, False, ws)
        else:
            em.ember_step_dense(W, G, r, c, t, LR, B2, EPS, False, ws)
        torch.cuda.synchronize()
        W_ref = prev.copy()
        assert oracle.step(W_ref, host_bits(G), r_o, c_o, t, row_only=row_only) == 0
        check_w(host_bits(W), W_ref, prev, f"W step {t}")
        _check_state_chunked(r, r_o, f"r step {t}")
        if not row_only:
            _check_state_chunked(c, c_o, f"c step {t}")
    del W, G, r, c, ws
    _free()


@pytest.mark.timeout(900)
def test_coalesce_the_largest_token_batch(em):
    # 2^26 token ids (Zipf over 128256 rows) with 8-wide bf16 signal rows
    P, V, D = 1 << 26, 128256, 8
    print(f"coalesce P={P} V={V} D={D}", flush=True)
    rng = np.random.default_rng(8)
    p = 1.0 / np.arange(1, V + 1) ** 1.1
    tok_h = rng.choice(V, P, p=p / p.sum()).astype(np.int64)
    U = torch.empty(P, D, dtype=torch.bfloat16, device=DEV)
    _fill_normal(U, 1e-3, 9)
    co = em.Coalescer(P, V, D, dtype=torch.bfloat16, device=DEV)
    idx, G = co(torch.from_numpy(tok_h).to(DEV), U)
    U_h = host_bits(U)
    st, idx_o, G_o = oracle.coalesce(tok_h, U_h, V, out_dtype=np.uint16)
    assert st == oracle.OK
    assert np.array_equal(idx.cpu().numpy(), idx_o)
    n_diff = check_coalesced_rows(host_bits(G), G_o, tok_h, as_f64(U_h), "largest batch")
    print(f"largest batch: n={idx.numel()}, elements at a rounding boundary: {n_diff}", flush=True)
    del U, co, idx, G
    _free()
