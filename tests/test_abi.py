"""C-ABI tests that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments on the host with the documented
status codes before touching the device."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ember.h")


@pytest.fixture(scope="module")
def em():
    lib_path = os.path.join(ROOT, "paper_2607_01455_amd", "libember.so")
    if not os.path.exists(lib_path):
        from paper_2607_01455_amd import build
        build.build()
    from paper_2607_01455_amd import ember
    return ember


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(ember_\w+)\s*\(", text, re.M)))


def test_header_declares_the_entry_points():
    names = _declared_functions()
    for required in ("ember_workspace_bytes", "ember_init_state", "ember_step_dense",
                     "ember_step_sparse_rows", "ember_rowonly_init_state", "ember_rowonly_step_dense",
                     "ember_rowonly_step_sparse_rows", "ember_get_error", "ember_strerror"):
        assert required in names


def test_library_exports_every_declared_function(em):
    names = _declared_functions()
    assert sorted(em.EXPORTED) == names
    for name in names:
        assert hasattr(em.LIB, name), name


def test_strerror_covers_every_status(em):
    for st in range(0, -9, -1):
        assert em.ember_strerror(st) and em.ember_strerror(st) != "unknown status"
    assert em.ember_strerror(12345) == "unknown status"


def test_workspace_bytes(em):
    out = ctypes.c_size_t(0)
    assert em.LIB.ember_workspace_bytes(0, 4, ctypes.byref(out)) == em.EMBER_ERR_SHAPE
    assert em.LIB.ember_workspace_bytes(4, 0, ctypes.byref(out)) == em.EMBER_ERR_SHAPE
    assert em.LIB.ember_workspace_bytes(4, 4, None) == em.EMBER_ERR_ARG
    assert em.LIB.ember_workspace_bytes(2 ** 31, 4, ctypes.byref(out)) == em.EMBER_ERR_SHAPE
    sizes = {}
    for V, D in [(1, 1), (1024, 64), (128256, 4096), (262144, 8192)]:
        assert em.LIB.ember_workspace_bytes(V, D, ctypes.byref(out)) == em.EMBER_OK
        assert out.value % 256 == 0
        # at least: slot table, per-slab row sums, per-block column partials
        assert out.value >= 4 * V + 4 * V * math.ceil(D / 4096) + 4 * D
        sizes[(V, D)] = out.value
    # partial buffers: per-block (or per-256-row tile) column sums and per-slab
    # (or per-256-column tile) row sums, a few tens of MB at the largest shape
    # (V D / 32 bytes from the tile partials: 1/64 of a bf16 gradient)
    assert sizes[(262144, 8192)] < 80 * 2 ** 20


# Fake, suitably aligned addresses: every call below must fail validation on
# the host, so none of them is ever dereferenced or passed to the device.
A = 1 << 20
W_, G_, R_, C_, WS_, IDX_ = A, 2 * A, 3 * A, 4 * A, 5 * A, 6 * A


def _ws_bytes(em, V, D):
    out = ctypes.c_size_t(0)
    em.LIB.ember_workspace_bytes(V, D, ctypes.byref(out))
    return out.value


def _dense(em, **kw):
    a = dict(W=W_, wd=1, ldw=64, G=G_, gd=1, ldg=64, r=R_, c=C_, V=10, D=64, t=1,
             lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.LIB.ember_step_dense(a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"], a["r"], a["c"],
                                   a["V"], a["D"], a["t"], a["lr"], a["b2"], a["eps"], a["mx"],
                                   a["ws"], a["wsb"], None)


def _sparse(em, **kw):
    a = dict(W=W_, wd=1, ldw=64, G=G_, gd=1, ldg=64, idx=IDX_, n=3, r=R_, c=C_, V=10, D=64, t=1,
             lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.LIB.ember_step_sparse_rows(a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"], a["idx"],
                                         a["n"], a["r"], a["c"], a["V"], a["D"], a["t"], a["lr"], a["b2"],
                                         a["eps"], a["mx"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(V=0), "SHAPE"), (dict(D=0), "SHAPE"), (dict(ldw=63), "SHAPE"), (dict(ldg=32), "SHAPE"),
    (dict(V=2 ** 31), "SHAPE"), (dict(D=2 ** 22 + 8, ldw=2 ** 22 + 8, ldg=2 ** 22 + 8), "SHAPE"),
    (dict(W=None), "ARG"), (dict(G=None), "ARG"), (dict(r=None), "ARG"), (dict(c=None), "ARG"),
    (dict(ws=None), "ARG"),
    (dict(W=W_ + 8), "ALIGN"), (dict(G=G_ + 2), "ALIGN"), (dict(ldw=68, D=60), "ALIGN"),
    (dict(wd=0, ldw=66, D=66), "ALIGN"), (dict(r=R_ + 2), "ALIGN"), (dict(ws=WS_ + 128), "ALIGN"),
    (dict(wd=2), "DTYPE"), (dict(gd=-1), "DTYPE"),
    (dict(wsb=1024), "WORKSPACE"),
    (dict(t=0), "ARG"), (dict(t=-5), "ARG"), (dict(b2=1.0), "ARG"), (dict(b2=-0.5), "ARG"),
    (dict(b2=float("nan")), "ARG"), (dict(lr=-1e-3), "ARG"), (dict(lr=float("inf")), "ARG"),
    (dict(eps=-1.0), "ARG"), (dict(eps=float("nan")), "ARG"),
])
def test_dense_step_rejects_bad_arguments_on_host(em, kw, status):
    assert _dense(em, **kw) == getattr(em, "EMBER_ERR_" + status)


@pytest.mark.parametrize("kw,status", [
    (dict(n=-1), "SHAPE"), (dict(n=11), "SHAPE"), (dict(idx=None), "ARG"), (dict(idx=IDX_ + 4), "ALIGN"),
    (dict(G=None), "ARG"), (dict(W=None), "ARG"), (dict(gd=3), "DTYPE"), (dict(t=0), "ARG"),
    (dict(wsb=0), "WORKSPACE"), (dict(V=0), "SHAPE"),
])
def test_sparse_step_rejects_bad_arguments_on_host(em, kw, status):
    assert _sparse(em, **kw) == getattr(em, "EMBER_ERR_" + status)


def _rowonly_dense(em, **kw):
    a = dict(W=W_, wd=1, ldw=64, G=G_, gd=1, ldg=64, r=R_, V=10, D=64, t=1,
             lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.LIB.ember_rowonly_step_dense(a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"], a["r"],
                                           a["V"], a["D"], a["t"], a["lr"], a["b2"], a["eps"], a["mx"],
                                           a["ws"], a["wsb"], None)


def _rowonly_sparse(em, **kw):
    a = dict(W=W_, wd=1, ldw=64, G=G_, gd=1, ldg=64, idx=IDX_, n=3, r=R_, V=10, D=64, t=1,
             lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.LIB.ember_rowonly_step_sparse_rows(a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"],
                                                 a["idx"], a["n"], a["r"], a["V"], a["D"], a["t"], a["lr"],
                                                 a["b2"], a["eps"], a["mx"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(V=0), "SHAPE"), (dict(D=0), "SHAPE"), (dict(ldw=63), "SHAPE"), (dict(ldg=32), "SHAPE"),
    (dict(V=2 ** 31), "SHAPE"), (dict(D=2 ** 22 + 8, ldw=2 ** 22 + 8, ldg=2 ** 22 + 8), "SHAPE"),
    (dict(W=None), "ARG"), (dict(G=None), "ARG"), (dict(r=None), "ARG"), (dict(ws=None), "ARG"),
    (dict(W=W_ + 8), "ALIGN"), (dict(G=G_ + 2), "ALIGN"), (dict(r=R_ + 2), "ALIGN"),
    (dict(ws=WS_ + 128), "ALIGN"), (dict(wd=2), "DTYPE"), (dict(wsb=1024), "WORKSPACE"),
    (dict(t=0), "ARG"), (dict(b2=1.0), "ARG"), (dict(lr=-1e-3), "ARG"), (dict(eps=float("inf")), "ARG"),
])
def test_rowonly_dense_step_rejects_bad_arguments_on_host(em, kw, status):
    assert _rowonly_dense(em, **kw) == getattr(em, "EMBER_ERR_" + status)


@pytest.mark.parametrize("kw,status", [
    (dict(n=-1), "SHAPE"), (dict(n=11), "SHAPE"), (dict(idx=None), "ARG"), (dict(idx=IDX_ + 4), "ALIGN"),
    (dict(G=None), "ARG"), (dict(r=None), "ARG"), (dict(gd=3), "DTYPE"), (dict(t=0), "ARG"),
    (dict(wsb=0), "WORKSPACE"), (dict(V=0), "SHAPE"),
])
def test_rowonly_sparse_step_rejects_bad_arguments_on_host(em, kw, status):
    assert _rowonly_sparse(em, **kw) == getattr(em, "EMBER_ERR_" + status)


def _coalesce(em, **kw):
    a = dict(tok=IDX_, P=100, U=G_, ud=1, ldu=64, V=1000, D=64, idx=IDX_ + A, G=W_, gd=1, ldg=64,
             n=R_, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        out = ctypes.c_size_t(0)
        em.LIB.ember_coalesce_workspace_bytes(max(a["P"], 0), max(a["V"], 1), max(a["D"], 1), ctypes.byref(out))
        a["wsb"] = out.value
    return em.LIB.ember_coalesce_rows(a["tok"], a["P"], a["U"], a["ud"], a["ldu"], a["V"], a["D"], a["idx"],
                                      a["G"], a["gd"], a["ldg"], a["n"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(P=-1), "SHAPE"), (dict(P=2 ** 26 + 1), "SHAPE"), (dict(V=0), "SHAPE"), (dict(D=0), "SHAPE"),
    (dict(ldu=32), "SHAPE"), (dict(ldg=63), "SHAPE"),
    (dict(tok=None), "ARG"), (dict(U=None), "ARG"), (dict(idx=None), "ARG"), (dict(G=None), "ARG"),
    (dict(n=None), "ARG"), (dict(ws=None), "ARG"),
    (dict(tok=IDX_ + 4), "ALIGN"), (dict(idx=IDX_ + A + 2), "ALIGN"), (dict(n=R_ + 4), "ALIGN"),
    (dict(U=G_ + 2), "ALIGN"), (dict(ws=WS_ + 64), "ALIGN"), (dict(ud=5), "DTYPE"), (dict(gd=-1), "DTYPE"),
    (dict(wsb=256), "WORKSPACE"),
])
def test_coalesce_rejects_bad_arguments_on_host(em, kw, status):
    assert _coalesce(em, **kw) == getattr(em, "EMBER_ERR_" + status)


def test_coalesce_workspace_bytes(em):
    out = ctypes.c_size_t(0)
    assert em.LIB.ember_coalesce_workspace_bytes(-1, 10, 10, ctypes.byref(out)) == em.EMBER_ERR_SHAPE
    assert em.LIB.ember_coalesce_workspace_bytes(10, 10, 10, None) == em.EMBER_ERR_ARG
    sizes = []
    for P in (0, 1, 16384, 1 << 20):
        assert em.LIB.ember_coalesce_workspace_bytes(P, 128256, 4096, ctypes.byref(out)) == em.EMBER_OK
        assert out.value % 256 == 0
        sizes.append(out.value)
    assert sizes == sorted(sizes)
    # sort buffers grow with the batch; the float64 partial rows stay bounded
    assert sizes[-1] < 2 * (1 << 25) * 8 + 64 * (1 << 20)


def _devn(em, row_only=False, **kw):
    a = dict(W=W_, wd=1, ldw=64, G=G_, gd=1, ldg=64, idx=IDX_, ndev=IDX_ + A, mx_rows=3, r=R_, c=C_, V=10, D=64,
             t=1, lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    if row_only:
        return em.LIB.ember_rowonly_step_sparse_rows_devn(
            a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"], a["idx"], a["ndev"], a["mx_rows"], a["r"],
            a["V"], a["D"], a["t"], a["lr"], a["b2"], a["eps"], a["mx"], a["ws"], a["wsb"], None)
    return em.LIB.ember_step_sparse_rows_devn(
        a["W"], a["wd"], a["ldw"], a["G"], a["gd"], a["ldg"], a["idx"], a["ndev"], a["mx_rows"], a["r"], a["c"],
        a["V"], a["D"], a["t"], a["lr"], a["b2"], a["eps"], a["mx"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("row_only", [False, True])
@pytest.mark.parametrize("kw,status", [
    (dict(mx_rows=-1), "SHAPE"), (dict(mx_rows=11), "SHAPE"), (dict(ndev=None), "ARG"),
    (dict(idx=None), "ARG"), (dict(ndev=IDX_ + A + 4), "ALIGN"), (dict(idx=IDX_ + 2), "ALIGN"),
    (dict(G=None), "ARG"), (dict(W=None), "ARG"), (dict(r=None), "ARG"), (dict(gd=7), "DTYPE"),
    (dict(t=0), "ARG"), (dict(wsb=0), "WORKSPACE"), (dict(V=0), "SHAPE"),
])
def test_device_count_steps_reject_bad_arguments_on_host(em, row_only, kw, status):
    assert _devn(em, row_only=row_only, **kw) == getattr(em, "EMBER_ERR_" + status)


DY_, H_ = 7 * A, 8 * A


def _lmhead(em, **kw):
    a = dict(W=W_, wd=1, ldw=64, dY=DY_, ldy=16, H=H_, ldh=64, T=32, G=G_, gd=1, ldg=64, r=R_, c=C_,
             V=10, D=64, t=1, lr=1e-3, b2=0.999, eps=1e-8, mx=0, ws=WS_, wsb=None)
    a.update(kw)
    if a["wsb"] is None:
        a["wsb"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.LIB.ember_lmhead_step(a["W"], a["wd"], a["ldw"], a["dY"], a["ldy"], a["H"], a["ldh"], a["T"],
                                    a["G"], a["gd"], a["ldg"], a["r"], a["c"], a["V"], a["D"], a["t"],
                                    a["lr"], a["b2"], a["eps"], a["mx"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(T=-1), "SHAPE"), (dict(T=2 ** 30 + 1), "SHAPE"), (dict(ldy=8), "SHAPE"), (dict(ldh=56), "SHAPE"),
    (dict(ldy=2 ** 24, V=2 ** 24 - 8), "SHAPE"), (dict(ldh=2 ** 24, D=64), "SHAPE"),
    (dict(V=0), "SHAPE"), (dict(ldw=32), "SHAPE"),
    (dict(dY=None), "ARG"), (dict(H=None), "ARG"), (dict(G=None), "ARG"), (dict(W=None), "ARG"),
    (dict(c=None), "ARG"), (dict(ws=None), "ARG"),
    (dict(dY=DY_ + 2), "ALIGN"), (dict(H=H_ + 8), "ALIGN"), (dict(ldy=12), "ALIGN"), (dict(G=G_ + 4), "ALIGN"),
    (dict(ws=WS_ + 64), "ALIGN"),
    (dict(wd=5), "DTYPE"), (dict(gd=2), "DTYPE"),
    (dict(wsb=256), "WORKSPACE"),
    (dict(t=0), "ARG"), (dict(b2=1.5), "ARG"), (dict(lr=float("nan")), "ARG"),
])
def test_lmhead_step_rejects_bad_arguments_on_host(em, kw, status):
    assert _lmhead(em, **kw) == getattr(em, "EMBER_ERR_" + status)


def test_lmhead_step_accepts_no_tokens_without_operands(em):
    # T = 0 lets dY and H be NULL; a bad scalar still fails on the host, so
    # nothing is launched here
    assert _lmhead(em, T=0, dY=None, H=None, t=0) == em.EMBER_ERR_ARG
    assert _lmhead(em, T=0, dY=None, H=None, wsb=0) == em.EMBER_ERR_WORKSPACE


def test_init_state_and_get_error_reject_bad_arguments(em):
    wsb = _ws_bytes(em, 10, 64)
    assert em.LIB.ember_init_state(R_, C_, 0, 64, WS_, wsb, None) == em.EMBER_ERR_SHAPE
    assert em.LIB.ember_init_state(None, C_, 10, 64, WS_, wsb, None) == em.EMBER_ERR_ARG
    assert em.LIB.ember_init_state(R_, C_, 10, 64, WS_, 8, None) == em.EMBER_ERR_WORKSPACE
    assert em.LIB.ember_init_state(R_, C_, 10, 64, WS_ + 4, wsb, None) == em.EMBER_ERR_ALIGN
    assert em.LIB.ember_rowonly_init_state(R_, 0, 64, WS_, wsb, None) == em.EMBER_ERR_SHAPE
    assert em.LIB.ember_rowonly_init_state(None, 10, 64, WS_, wsb, None) == em.EMBER_ERR_ARG
    assert em.LIB.ember_rowonly_init_state(R_, 10, 64, WS_, 8, None) == em.EMBER_ERR_WORKSPACE
    assert em.LIB.ember_rowonly_init_state(R_, 10, 64, WS_ + 4, wsb, None) == em.EMBER_ERR_ALIGN
    st = ctypes.c_int(0)
    assert em.LIB.ember_get_error(None, None, ctypes.byref(st)) == em.EMBER_ERR_ARG
    assert em.LIB.ember_get_error(WS_, None, None) == em.EMBER_ERR_ARG
    assert em.LIB.ember_get_error(WS_ + 16, None, ctypes.byref(st)) == em.EMBER_ERR_ALIGN


def test_binding_marshals_dtypes_and_strides(em):
    import torch
    assert em._dtype(torch.zeros(1, dtype=torch.float32)) == em.EMBER_F32
    assert em._dtype(torch.zeros(1, dtype=torch.bfloat16)) == em.EMBER_BF16
    assert em._dtype(torch.zeros(1, dtype=torch.float16)) not in (em.EMBER_F32, em.EMBER_BF16)
    x = torch.zeros(5, 72)[:, :64]
    assert em._ld(x) == 72
    # one row: a stride that keeps rows 16-byte aligned (never used to step rows)
    assert em._ld(torch.zeros(1, 5)) == 8
    assert em._ld(torch.zeros(1, 5, dtype=torch.bfloat16)) == 8
    assert em._ld(torch.zeros(1, 4096, dtype=torch.bfloat16)) == 4096
    with pytest.raises(TypeError):
        em._ld(torch.zeros(5, 8).t())


# ---------------------------------------------------------------------------
# ember_step_multi: host checks (fake addresses again: every call must fail)
# ---------------------------------------------------------------------------

def _table(em, base=0, **kw):
    """A TableStep of a 10 x 64 bf16 table whose buffers start at base + the
    fake addresses above (base = k * 16 A keeps tables apart)."""
    a = dict(W=W_ + base, w_dtype=1, ldw=64, G=G_ + base, g_dtype=1, ldg=64, sparse=0, idx=None, n_idx=0,
             n_idx_dev=None, r=R_ + base, c=C_ + base, V=10, D=64, t=1, lr=1e-3, beta2=0.999, eps=1e-8,
             maximize=0, ws=WS_ + base, ws_bytes=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = _ws_bytes(em, max(a["V"], 1), max(a["D"], 1))
    return em.TableStep(**a)


def _multi(em, tables, n=None):
    arr = (em.TableStep * max(len(tables), 1))(*tables)
    return em.LIB.ember_step_multi(arr, len(tables) if n is None else n, None)


@pytest.mark.parametrize("kw,status", [
    (dict(V=0), "SHAPE"), (dict(ldw=32), "SHAPE"), (dict(W=None), "ARG"), (dict(G=G_ + 16 * A + 2), "ALIGN"),
    (dict(w_dtype=5), "DTYPE"), (dict(ws_bytes=64), "WORKSPACE"), (dict(t=0), "ARG"), (dict(beta2=1.0), "ARG"),
    (dict(sparse=2), "ARG"),
    (dict(sparse=1, idx=IDX_ + 16 * A, n_idx=11), "SHAPE"), (dict(sparse=1, idx=None, n_idx=3), "ARG"),
    (dict(sparse=1, idx=IDX_ + 16 * A + 4, n_idx=3), "ALIGN"),
    (dict(sparse=1, idx=IDX_ + 16 * A, n_idx=3, n_idx_dev=IDX_ + 16 * A + 4), "ALIGN"),
    (dict(sparse=1, idx=IDX_ + 16 * A, n_idx=-1, n_idx_dev=IDX_ + 17 * A), "SHAPE"),
    (dict(row_only=2), "ARG"), (dict(row_only=1, r=None), "ARG"), (dict(row_only=1, ws_bytes=64), "WORKSPACE"),
    (dict(row_only=1, sparse=1, idx=None, n_idx=3), "ARG"),
])
def test_multi_step_checks_every_table(em, kw, status):
    # the first table is valid; the second fails its own call's check
    good = _table(em)
    assert _multi(em, [good, _table(em, base=16 * A, **kw)]) == getattr(em, "EMBER_ERR_" + status)


def test_multi_step_rejects_table_counts_and_overlaps(em):
    good = _table(em)
    assert _multi(em, [good], n=0) == em.EMBER_ERR_ARG
    assert _multi(em, [good] * 9) == em.EMBER_ERR_ARG
    assert em.LIB.ember_step_multi(None, 1, None) == em.EMBER_ERR_ARG
    # two tables sharing a workspace, an r/c vector or a weight matrix
    assert _multi(em, [good, _table(em, base=16 * A, ws=WS_)]) == em.EMBER_ERR_ARG
    assert _multi(em, [good, _table(em, base=16 * A, r=C_)]) == em.EMBER_ERR_ARG
    assert _multi(em, [good, _table(em, base=16 * A, W=W_ + 128)]) == em.EMBER_ERR_ARG
    assert _multi(em, [good, _table(em, base=16 * A, c=WS_ + 256)]) == em.EMBER_ERR_ARG
    assert _multi(em, [good, good]) == em.EMBER_ERR_ARG
    # one table's written memory over another table's gradient, id list or row count
    assert _multi(em, [good, _table(em, base=16 * A, W=G_)]) == em.EMBER_ERR_ARG
    assert _multi(em, [good, _table(em, base=16 * A, G=W_ + 256)]) == em.EMBER_ERR_ARG
    sparse = dict(sparse=1, idx=IDX_ + 16 * A, n_idx=3)
    assert _multi(em, [good, _table(em, base=16 * A, **dict(sparse, idx=R_))]) == em.EMBER_ERR_ARG
    assert _multi(em, [_table(em, base=16 * A, **sparse), _table(em, r=IDX_ + 16 * A + 8)]) == em.EMBER_ERR_ARG
    devn = dict(sparse, n_idx_dev=IDX_ + 17 * A)
    assert _multi(em, [_table(em, base=16 * A, **devn), _table(em, c=IDX_ + 17 * A)]) == em.EMBER_ERR_ARG


def test_stream_probe_rejects_bad_arguments_on_host(em):
    P = em.LIB.ember_stream_probe
    assert P(3, W_, G_, None, 64, None) == em.EMBER_ERR_ARG
    assert P(-1, W_, G_, None, 64, None) == em.EMBER_ERR_ARG
    assert P(1, None, G_, None, 64, None) == em.EMBER_ERR_ARG
    assert P(1, W_, None, None, 64, None) == em.EMBER_ERR_ARG
    assert P(2, W_, G_, None, 64, None) == em.EMBER_ERR_ARG
    assert P(1, W_, G_, None, 40, None) == em.EMBER_ERR_SHAPE
    assert P(1, W_ + 8, G_, None, 64, None) == em.EMBER_ERR_ALIGN
    assert P(2, W_, G_, R_ + 4, 64, None) == em.EMBER_ERR_ALIGN


def test_table_step_struct_matches_the_header(em):
    """The binding's TableStep has the fields of ember_table_step, in order and
    with C types of the same size (a mismatch would hand the library wrong
    pointers)."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct \{(.*?)\}\s*ember_table_step;", text, re.S).group(1)
    fields = re.findall(r"^\s*(.+?)\s*\b(\w+);", body, re.M)
    sizes = {"void*": 8, "const void*": 8, "int": 4, "int64_t": 8, "const int64_t*": 8, "float*": 8,
             "float": 4, "size_t": 8}
    assert [name for _, name in fields] == [f[0] for f in em.TableStep._fields_]
    for (ctype, name), (pname, ptype) in zip(fields, em.TableStep._fields_):
        assert ctypes.sizeof(ptype) == sizes[ctype.replace(" *", "*")], (name, ctype, ptype)
    # natural alignment, as the C compiler lays the struct out
    off = 0
    for (ctype, name), (pname, ptype) in zip(fields, em.TableStep._fields_):
        sz = sizes[ctype.replace(" *", "*")]
        off = (off + sz - 1) // sz * sz
        assert getattr(em.TableStep, pname).offset == off, name
        off += sz
    assert ctypes.sizeof(em.TableStep) == (off + 7) // 8 * 8


def test_barrier_wait_bound_checks_its_argument(em):
    assert em.LIB.ember_set_barrier_wait_ticks(-1) == em.EMBER_ERR_ARG
    assert em.LIB.ember_set_barrier_wait_ticks(1000) == em.EMBER_OK
    assert em.LIB.ember_set_barrier_wait_ticks(0) == em.EMBER_OK   # the default again
