"""Python binding of libember.so: argument marshalling only.

Each function has the name of the C entry point it calls (include/ember.h) and
passes torch tensors as raw device pointers plus sizes, on the current torch
stream.  Every step of the Ember update runs in the library's HIP kernels;
there is no other implementation here.  Importing this module fails loudly if
the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libember.so")

EMBER_F32 = 0
EMBER_BF16 = 1

EMBER_OK = 0
EMBER_ERR_ARG = -1
EMBER_ERR_SHAPE = -2
EMBER_ERR_ALIGN = -3
EMBER_ERR_DTYPE = -4
EMBER_ERR_WORKSPACE = -5
EMBER_ERR_INDEX = -6
EMBER_ERR_HIP = -7
EMBER_ERR_DEVICE = -8

# Every function the C header declares, checked by the CPU test suite.
EXPORTED = ("ember_workspace_bytes", "ember_init_state", "ember_step_dense",
            "ember_step_sparse_rows", "ember_rowonly_init_state", "ember_rowonly_step_dense",
            "ember_rowonly_step_sparse_rows", "ember_step_sparse_rows_devn",
            "ember_rowonly_step_sparse_rows_devn", "ember_coalesce_workspace_bytes", "ember_coalesce_rows",
            "ember_lmhead_step", "ember_step_multi", "ember_get_error", "ember_strerror",
            "ember_profile_enable", "ember_profile_collect", "ember_stream_probe",
            "ember_set_barrier_wait_ticks",
            "ember_step_sparse_rows_static")


class EmberError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {ember_strerror(status)} (status {status})")
        self.status = status


EMBER_MAX_TABLES = 8


class TableStep(ctypes.Structure):
    """One table of ember_step_multi (the C struct ember_table_step)."""
    _fields_ = [("W", ctypes.c_void_p), ("w_dtype", ctypes.c_int), ("ldw", ctypes.c_int64),
                ("G", ctypes.c_void_p), ("g_dtype", ctypes.c_int), ("ldg", ctypes.c_int64),
                ("sparse", ctypes.c_int), ("row_only", ctypes.c_int), ("idx", ctypes.c_void_p),
                ("n_idx", ctypes.c_int64),
                ("n_idx_dev", ctypes.c_void_p), ("r", ctypes.c_void_p), ("c", ctypes.c_void_p),
                ("V", ctypes.c_int64), ("D", ctypes.c_int64), ("t", ctypes.c_int64),
                ("lr", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("maximize", ctypes.c_int), ("ws", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t)]


class _KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


def _load(path: str = _LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_01455_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i64, f32, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int, ctypes.c_size_t
    lib.ember_workspace_bytes.argtypes = [i64, i64, ctypes.POINTER(sz)]
    lib.ember_init_state.argtypes = [vp, vp, i64, i64, vp, sz, vp]
    lib.ember_step_dense.argtypes = [vp, i32, i64, vp, i32, i64, vp, vp, i64, i64, i64,
                                     f32, f32, f32, i32, vp, sz, vp]
    lib.ember_step_sparse_rows.argtypes = [vp, i32, i64, vp, i32, i64, vp, i64, vp, vp, i64, i64, i64,
                                           f32, f32, f32, i32, vp, sz, vp]
    lib.ember_rowonly_init_state.argtypes = [vp, i64, i64, vp, sz, vp]
    lib.ember_rowonly_step_dense.argtypes = [vp, i32, i64, vp, i32, i64, vp, i64, i64, i64,
                                             f32, f32, f32, i32, vp, sz, vp]
    lib.ember_rowonly_step_sparse_rows.argtypes = [vp, i32, i64, vp, i32, i64, vp, i64, vp, i64, i64, i64,
                                                   f32, f32, f32, i32, vp, sz, vp]
    lib.ember_step_sparse_rows_devn.argtypes = [vp, i32, i64, vp, i32, i64, vp, vp, i64, vp, vp, i64, i64, i64,
                                                f32, f32, f32, i32, vp, sz, vp]
    lib.ember_rowonly_step_sparse_rows_devn.argtypes = [vp, i32, i64, vp, i32, i64, vp, vp, i64, vp, i64, i64,
                                                        i64, f32, f32, f32, i32, vp, sz, vp]
    lib.ember_coalesce_workspace_bytes.argtypes = [i64, i64, i64, ctypes.POINTER(sz)]
    lib.ember_coalesce_rows.argtypes = [vp, i64, vp, i32, i64, i64, i64, vp, vp, i32, i64, vp, vp, sz, vp]
    lib.ember_lmhead_step.argtypes = [vp, i32, i64, vp, i64, vp, i64, i64, vp, i32, i64, vp, vp, i64, i64, i64,
                                      f32, f32, f32, i32, vp, sz, vp]
    lib.ember_step_multi.argtypes = [ctypes.POINTER(TableStep), i32, vp]
    lib.ember_get_error.argtypes = [vp, vp, ctypes.POINTER(i32)]
    lib.ember_strerror.argtypes = [i32]
    lib.ember_strerror.restype = ctypes.c_char_p
    lib.ember_profile_enable.argtypes = [i32]
    lib.ember_set_barrier_wait_ticks.argtypes = [ctypes.c_int64]
    lib.ember_profile_collect.argtypes = [ctypes.POINTER(_KernelStat), i32, ctypes.POINTER(i32)]
    lib.ember_stream_probe.argtypes = [i32, vp, vp, vp, sz, vp]
    lib.ember_step_sparse_rows_static.argtypes = [vp, i32, i64, vp, i32, i64, vp, i64, vp, vp, i64, i64, i64,
                                                  f32, f32, f32, i32, vp, vp]
    for name in EXPORTED:
        if name != "ember_strerror":
            getattr(lib, name).restype = i32
    return lib


LIB = _load()


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return EMBER_F32
    if t.dtype == torch.bfloat16:
        return EMBER_BF16
    return 99  # rejected by the library with EMBER_ERR_DTYPE


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or (t.size(1) > 1 and t.stride(1) != 1):
        raise TypeError("a 2-D tensor with unit column stride is required")
    if t.size(0) > 1:
        return t.stride(0)
    # one row: the stride is never used to address a second row; give the
    # smallest one that keeps the library's 16-byte row rule
    q = max(1, 16 // t.element_size())
    return (t.size(1) + q - 1) // q * q


def _ptr(t):
    return None if t is None or t.numel() == 0 else t.data_ptr()


def _stream(t: torch.Tensor):
    return torch.cuda.current_stream(t.device).cuda_stream


def _check(status: int, where: str) -> None:
    if status != EMBER_OK:
        raise EmberError(status, where)


def ember_strerror(status: int) -> str:
    return LIB.ember_strerror(int(status)).decode()


def ember_workspace_bytes(V: int, D: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.ember_workspace_bytes(int(V), int(D), ctypes.byref(out)), "ember_workspace_bytes")
    return out.value


def ember_init_state(r: torch.Tensor, c: torch.Tensor, ws: torch.Tensor) -> None:
    _check(LIB.ember_init_state(_ptr(r), _ptr(c), r.numel(), c.numel(), _ptr(ws),
                                ws.numel() * ws.element_size(), _stream(r)), "ember_init_state")


def ember_step_dense(W: torch.Tensor, G: torch.Tensor, r: torch.Tensor, c: torch.Tensor, t: int,
                     lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                     maximize: bool = False, ws: torch.Tensor | None = None) -> None:
    V, D = W.shape
    _check(LIB.ember_step_dense(_ptr(W), _dtype(W), _ld(W), _ptr(G), _dtype(G), _ld(G),
                                _ptr(r), _ptr(c), V, D, int(t), float(lr), float(beta2), float(eps),
                                int(bool(maximize)), _ptr(ws), ws.numel() * ws.element_size(),
                                _stream(W)), "ember_step_dense")


def ember_step_sparse_rows(W: torch.Tensor, G_rows: torch.Tensor, idx: torch.Tensor,
                           r: torch.Tensor, c: torch.Tensor, t: int,
                           lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                           maximize: bool = False, ws: torch.Tensor | None = None) -> None:
    V, D = W.shape
    n = idx.numel()
    if idx.dtype != torch.int64:
        raise TypeError("idx must be int64")
    ldg = _ld(G_rows) if G_rows.numel() else D
    _check(LIB.ember_step_sparse_rows(_ptr(W), _dtype(W), _ld(W), _ptr(G_rows), _dtype(G_rows), ldg,
                                      _ptr(idx), n, _ptr(r), _ptr(c), V, D, int(t), float(lr),
                                      float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream(W)),
           "ember_step_sparse_rows")


def ember_step_sparse_rows_static(W: torch.Tensor, G_rows: torch.Tensor, idx: torch.Tensor,
                                  r: torch.Tensor, c: torch.Tensor, t: int, status: torch.Tensor,
                                  lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                                  maximize: bool = False) -> None:
    """Sparse-row step whose scratch is the library's own array (no workspace);
    status: a device int32 tensor of one element that receives the error bits."""
    V, D = W.shape
    n = idx.numel()
    if idx.dtype != torch.int64 or status.dtype != torch.int32:
        raise TypeError("idx must be int64 and status int32")
    ldg = _ld(G_rows) if G_rows.numel() else D
    _check(LIB.ember_step_sparse_rows_static(_ptr(W), _dtype(W), _ld(W), _ptr(G_rows), _dtype(G_rows), ldg,
                                             _ptr(idx), n, _ptr(r), _ptr(c), V, D, int(t), float(lr),
                                             float(beta2), float(eps), int(bool(maximize)), status.data_ptr(),
                                             _stream(W)), "ember_step_sparse_rows_static")


def ember_rowonly_init_state(r: torch.Tensor, D: int, ws: torch.Tensor) -> None:
    _check(LIB.ember_rowonly_init_state(_ptr(r), r.numel(), int(D), _ptr(ws),
                                        ws.numel() * ws.element_size(), _stream(r)),
           "ember_rowonly_init_state")


def ember_rowonly_step_dense(W: torch.Tensor, G: torch.Tensor, r: torch.Tensor, t: int,
                             lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                             maximize: bool = False, ws: torch.Tensor | None = None) -> None:
    V, D = W.shape
    _check(LIB.ember_rowonly_step_dense(_ptr(W), _dtype(W), _ld(W), _ptr(G), _dtype(G), _ld(G),
                                        _ptr(r), V, D, int(t), float(lr), float(beta2), float(eps),
                                        int(bool(maximize)), _ptr(ws), ws.numel() * ws.element_size(),
                                        _stream(W)), "ember_rowonly_step_dense")


def ember_rowonly_step_sparse_rows(W: torch.Tensor, G_rows: torch.Tensor, idx: torch.Tensor,
                                   r: torch.Tensor, t: int,
                                   lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                                   maximize: bool = False, ws: torch.Tensor | None = None) -> None:
    V, D = W.shape
    n = idx.numel()
    if idx.dtype != torch.int64:
        raise TypeError("idx must be int64")
    ldg = _ld(G_rows) if G_rows.numel() else D
    _check(LIB.ember_rowonly_step_sparse_rows(_ptr(W), _dtype(W), _ld(W), _ptr(G_rows), _dtype(G_rows),
                                              ldg, _ptr(idx), n, _ptr(r), V, D, int(t), float(lr),
                                              float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
                                              ws.numel() * ws.element_size(), _stream(W)),
           "ember_rowonly_step_sparse_rows")


def ember_step_sparse_rows_devn(W: torch.Tensor, G_rows: torch.Tensor, idx: torch.Tensor, n_dev: torch.Tensor,
                                r: torch.Tensor, c, t: int, lr: float = 1e-3, beta2: float = 0.999,
                                eps: float = 1e-8, maximize: bool = False, ws: torch.Tensor | None = None,
                                row_only: bool = False) -> None:
    """Sparse step whose row count n is the int64 in device tensor n_dev; G_rows
    and idx hold the maximum count of rows (their first dimension)."""
    V, D = W.shape
    if idx.dtype != torch.int64 or n_dev.dtype != torch.int64:
        raise TypeError("idx and n_dev must be int64")
    max_rows = idx.numel()
    ldg = _ld(G_rows) if G_rows.numel() else D
    if row_only:
        st = LIB.ember_rowonly_step_sparse_rows_devn(
            _ptr(W), _dtype(W), _ld(W), _ptr(G_rows), _dtype(G_rows), ldg, _ptr(idx), n_dev.data_ptr(), max_rows,
            _ptr(r), V, D, int(t), float(lr), float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(W))
    else:
        st = LIB.ember_step_sparse_rows_devn(
            _ptr(W), _dtype(W), _ld(W), _ptr(G_rows), _dtype(G_rows), ldg, _ptr(idx), n_dev.data_ptr(), max_rows,
            _ptr(r), _ptr(c), V, D, int(t), float(lr), float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(W))
    _check(st, "ember_step_sparse_rows_devn")


def ember_coalesce_workspace_bytes(max_tokens: int, V: int, D: int) -> int:
    out = ctypes.c_size_t(0)
    _check(LIB.ember_coalesce_workspace_bytes(int(max_tokens), int(V), int(D), ctypes.byref(out)),
           "ember_coalesce_workspace_bytes")
    return out.value


def ember_coalesce_rows(tok: torch.Tensor, U: torch.Tensor, V: int, idx: torch.Tensor, G_rows: torch.Tensor,
                        n_out: torch.Tensor, ws: torch.Tensor) -> None:
    """Enqueue the coalescing of (tok, U) into (idx, G_rows, n_out) on the current
    stream; n_out is a device int64 tensor of one element."""
    if tok.dtype != torch.int64 or idx.dtype != torch.int64 or n_out.dtype != torch.int64:
        raise TypeError("tok, idx and n_out must be int64")
    P = tok.numel()
    D = U.shape[1]
    ldu = _ld(U) if P else D
    ldg = _ld(G_rows) if G_rows.numel() else D
    _check(LIB.ember_coalesce_rows(_ptr(tok), P, _ptr(U), _dtype(U), ldu, int(V), D, _ptr(idx),
                                   _ptr(G_rows), _dtype(G_rows), ldg, n_out.data_ptr(), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(n_out)), "ember_coalesce_rows")


class Coalescer:
    """Workspace and outputs for coalescing batches of up to max_tokens token
    gradients of a V-row, D-column table."""

    def __init__(self, max_tokens: int, V: int, D: int, dtype=torch.bfloat16, device="cuda"):
        self.max_tokens, self.V, self.D = int(max_tokens), int(V), int(D)
        n = max(self.max_tokens, 1)
        q = 16 // torch.empty(0, dtype=dtype).element_size()
        ld = (self.D + q - 1) // q * q   # rows start on 16-byte boundaries
        self.idx = torch.empty(n, dtype=torch.int64, device=device)
        self.G_rows = torch.empty(n, ld, dtype=dtype, device=device)[:, :self.D]
        self.n_out = torch.zeros(1, dtype=torch.int64, device=device)
        nbytes = ember_coalesce_workspace_bytes(self.max_tokens, self.V, self.D)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=device)

    def enqueue(self, tok: torch.Tensor, U: torch.Tensor) -> None:
        """Coalesce one batch on the current stream without reading n back:
        self.idx, self.G_rows and self.n_out then feed a step with a device
        row count (EmberTable.step_tokens)."""
        if tok.numel() > self.max_tokens:
            raise ValueError("batch larger than max_tokens")
        ember_coalesce_rows(tok, U, self.V, self.idx, self.G_rows, self.n_out, self.ws)

    def __call__(self, tok: torch.Tensor, U: torch.Tensor):
        """Coalesce one batch; synchronises to read n.  Returns (idx, G_rows)
        views of the first n rows."""
        if tok.numel() > self.max_tokens:
            raise ValueError("batch larger than max_tokens")
        ember_coalesce_rows(tok, U, self.V, self.idx, self.G_rows, self.n_out, self.ws)
        _check(ember_get_error(self.ws), "ember_coalesce_rows (device)")
        n = int(self.n_out.item())
        return self.idx[:n], self.G_rows[:n]


def ember_lmhead_step(W: torch.Tensor, dY: torch.Tensor, H: torch.Tensor, G: torch.Tensor,
                      r: torch.Tensor, c: torch.Tensor, t: int,
                      lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
                      maximize: bool = False, ws: torch.Tensor | None = None) -> None:
    """LM-head step: G = dY^T H (dY: T x V logits gradient, H: T x D hidden
    states, both bf16) written to G, and the dense Ember step on W with it."""
    V, D = W.shape
    T = dY.shape[0]
    if dY.dim() != 2 or H.dim() != 2 or dY.shape[1] != V or H.shape[0] != T or H.shape[1] != D:
        raise ValueError(f"shapes: dY {tuple(dY.shape)}, H {tuple(H.shape)} for W {tuple(W.shape)}")
    if tuple(G.shape) != (V, D):
        raise ValueError(f"G must be {V} x {D}")
    if T and (dY.dtype != torch.bfloat16 or H.dtype != torch.bfloat16):
        raise TypeError("dY and H must be bfloat16")
    ldy = _ld(dY) if T else V
    ldh = _ld(H) if T else D
    _check(LIB.ember_lmhead_step(_ptr(W), _dtype(W), _ld(W), _ptr(dY), ldy, _ptr(H), ldh, T,
                                 _ptr(G), _dtype(G), _ld(G), _ptr(r), _ptr(c), V, D, int(t), float(lr),
                                 float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
                                 ws.numel() * ws.element_size(), _stream(W)), "ember_lmhead_step")


def table_step(W: torch.Tensor, G: torch.Tensor | None, r: torch.Tensor, c: torch.Tensor | None, t: int,
               ws: torch.Tensor, idx: torch.Tensor | None = None, n_idx_dev: torch.Tensor | None = None,
               lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
               maximize: bool = False, row_only: bool = False) -> TableStep:
    """One entry of ember_step_multi: a dense step when idx is None, else a
    sparse-row step on the rows idx lists (with n_idx_dev: the row count in
    device memory, idx.numel() its maximum); row_only: the row-only step (c
    unused).  The tensors must stay alive until the step has run."""
    V, D = W.shape
    sparse = idx is not None
    if sparse and idx.dtype != torch.int64:
        raise TypeError("idx must be int64")
    n = idx.numel() if sparse else 0
    ldg = _ld(G) if G is not None and G.numel() else D
    return TableStep(_ptr(W), _dtype(W), _ld(W), _ptr(G), _dtype(G) if G is not None else _dtype(W), ldg,
                     int(sparse), int(bool(row_only)), _ptr(idx) if sparse else None, n, _ptr(n_idx_dev),
                     _ptr(r), _ptr(c),
                     V, D, int(t), float(lr), float(beta2), float(eps), int(bool(maximize)), _ptr(ws),
                     ws.numel() * ws.element_size())


def ember_step_multi(steps, stream_of: torch.Tensor) -> None:
    """Enqueue the steps of several tables (TableStep entries) on the current
    stream of stream_of's device, in shared launches (a sparse table whose
    rows fit on chip takes its one-launch step)."""
    arr = (TableStep * len(steps))(*steps)
    _check(LIB.ember_step_multi(arr, len(steps), _stream(stream_of)), "ember_step_multi")


def step_tables(items) -> None:
    """Ember steps of several tables in one call.  items: tuples (EmberTable,
    W, G) for a dense step or (EmberTable, W, G_rows, idx) for a sparse-row
    step; each table takes its canonical or row-only step; every table
    advances t by one."""
    steps = []
    for it in items:
        tab, W, G = it[0], it[1], it[2]
        idx = it[3] if len(it) > 3 else None
        steps.append(table_step(W, G, tab.r, tab.c, tab.t + 1, tab.ws, idx=idx, lr=tab.lr, beta2=tab.beta2,
                                eps=tab.eps, maximize=tab.maximize, row_only=tab.row_only))
    ember_step_multi(steps, items[0][1])
    for it in items:
        it[0].t += 1


def ember_get_error(ws: torch.Tensor) -> int:
    """Device status of the last step on this workspace (synchronises the stream)."""
    st = ctypes.c_int(0)
    _check(LIB.ember_get_error(_ptr(ws), _stream(ws), ctypes.byref(st)), "ember_get_error")
    return st.value


def ember_set_barrier_wait_ticks(ticks: int) -> None:
    """Bound of the one-launch sparse step's grid-barrier waits in 100 MHz
    ticks (diagnostics; 0 restores the default of about one second)."""
    _check(LIB.ember_set_barrier_wait_ticks(int(ticks)), "ember_set_barrier_wait_ticks")


def ember_profile_enable(enable: bool) -> None:
    _check(LIB.ember_profile_enable(int(bool(enable))), "ember_profile_enable")


def ember_profile_collect() -> dict:
    """{kernel name: (launches, total milliseconds)} since the last collect."""
    buf = (_KernelStat * 16)()
    n = ctypes.c_int(0)
    _check(LIB.ember_profile_collect(buf, 16, ctypes.byref(n)), "ember_profile_collect")
    return {buf[k].name.decode(): (buf[k].launches, buf[k].total_ms) for k in range(n.value)}


def ember_stream_probe(mode: int, dst: torch.Tensor, a: torch.Tensor, b: torch.Tensor | None = None) -> None:
    """Streaming probe over a's bytes: 0 read a, 1 copy a to dst, 2 dst = a + b
    (32-bit integer lanes)."""
    nbytes = a.numel() * a.element_size()
    _check(LIB.ember_stream_probe(int(mode), _ptr(dst), _ptr(a), _ptr(b), nbytes, _stream(a)),
           "ember_stream_probe")


class EmberTable:
    """Ember state of one V x D token table on one device: r, c, workspace, t.

    A convenience holder around the C entry points (Algorithm 1: r_0 = 0,
    c_0 = 0, t = 0, then t += 1 before each update).  ``row_only`` selects the
    row-only variant of Section 2.1 (no c).
    """

    def __init__(self, V: int, D: int, device="cuda", lr: float = 1e-3, beta2: float = 0.999,
                 eps: float = 1e-8, maximize: bool = False, row_only: bool = False):
        self.V, self.D = int(V), int(D)
        self.lr, self.beta2, self.eps, self.maximize = lr, beta2, eps, maximize
        self.row_only = bool(row_only)
        self.r = torch.empty(self.V, dtype=torch.float32, device=device)
        self.c = None if self.row_only else torch.empty(self.D, dtype=torch.float32, device=device)
        nbytes = ember_workspace_bytes(self.V, self.D)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.t = 0
        if self.row_only:
            ember_rowonly_init_state(self.r, self.D, self.ws)
        else:
            ember_init_state(self.r, self.c, self.ws)

    def step(self, W: torch.Tensor, G: torch.Tensor) -> None:
        if self.row_only:
            ember_rowonly_step_dense(W, G, self.r, self.t + 1, self.lr, self.beta2, self.eps,
                                     self.maximize, self.ws)
        else:
            ember_step_dense(W, G, self.r, self.c, self.t + 1, self.lr, self.beta2, self.eps,
                             self.maximize, self.ws)
        self.t += 1

    def step_lmhead(self, W: torch.Tensor, dY: torch.Tensor, H: torch.Tensor, G: torch.Tensor) -> None:
        """LM-head step from the logits gradient dY [T, V] and hidden states
        H [T, D] (bf16): G = dY^T H is written to G and the step takes its
        statistics from the GEMM's epilogue (canonical Ember only)."""
        if self.row_only:
            raise ValueError("the fused LM-head step is the canonical (row and column) step")
        ember_lmhead_step(W, dY, H, G, self.r, self.c, self.t + 1, self.lr, self.beta2, self.eps,
                          self.maximize, self.ws)
        self.t += 1

    def step_tokens(self, W: torch.Tensor, tok: torch.Tensor, U: torch.Tensor, coalescer: "Coalescer") -> None:
        """Sparse step from token ids and per-position gradient rows: coalescing
        and the step are enqueued back to back with the row count kept in
        device memory (no host synchronisation; capturable in a HIP graph).
        Index errors of either call show in ember_get_error of its workspace."""
        coalescer.enqueue(tok, U)
        ember_step_sparse_rows_devn(W, coalescer.G_rows, coalescer.idx, coalescer.n_out, self.r, self.c,
                                    self.t + 1, self.lr, self.beta2, self.eps, self.maximize, self.ws,
                                    row_only=self.row_only)
        self.t += 1

    def step_sparse_rows(self, W: torch.Tensor, G_rows: torch.Tensor, idx: torch.Tensor,
                         check: bool = False) -> None:
        """Sparse-row step.  With check=True the index status is read back (a
        stream sync) and t advances only if idx was valid."""
        if self.row_only:
            ember_rowonly_step_sparse_rows(W, G_rows, idx, self.r, self.t + 1, self.lr, self.beta2,
                                           self.eps, self.maximize, self.ws)
        else:
            ember_step_sparse_rows(W, G_rows, idx, self.r, self.c, self.t + 1, self.lr, self.beta2,
                                   self.eps, self.maximize, self.ws)
        if check:
            _check(ember_get_error(self.ws), "ember_step_sparse_rows (device)")
        self.t += 1
