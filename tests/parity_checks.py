"""Comparison helpers shared by the GPU parity tests (tolerances are stated in
the docstring of test_gpu_parity)."""
import numpy as np
import torch

DEV = "cuda"
B2 = 0.999
LR = 1e-3
EPS = 1e-8


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Host copy of a device tensor: float32 values or bf16 bit patterns."""
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return t.contiguous().cpu().numpy()


def bf16_values(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def ordered16(b: np.ndarray) -> np.ndarray:
    b = b.astype(np.int64)
    return np.where(b & 0x8000, 0x8000 - (b & 0x7FFF), 0x8000 + b)


def check_w(got: np.ndarray, want: np.ndarray, prev: np.ndarray, what: str) -> None:
    if got.dtype == np.uint16:
        d = np.abs(ordered16(got) - ordered16(want))
        bad = d > 1
        if bad.any():
            gv, wv, pv = (bf16_values(x[bad]) for x in (got, want, prev))
            cancel_ok = np.abs(gv - wv) <= 1e-5 * np.maximum(np.abs(wv), np.abs(pv))
            assert cancel_ok.all(), (
                f"{what}: {(~cancel_ok).sum()} bf16 elements differ by > 1 ulp outside cancellation "
                f"(max {d.max()} ulp); first: got {gv[~cancel_ok][:3]} want {wv[~cancel_ok][:3]} prev {pv[~cancel_ok][:3]}")
    else:
        tol = 1e-5 * np.maximum(np.abs(want), np.abs(prev))
        err = np.abs(got.astype(np.float64) - want.astype(np.float64))
        bad = ~(err <= tol)
        assert not bad.any(), f"{what}: {bad.sum()} fp32 elements out of tolerance (max err {err.max()})"


def check_state(got: torch.Tensor, want: np.ndarray, what: str) -> None:
    g = got.cpu().numpy().astype(np.float64)
    w = want.astype(np.float64)
    err = np.abs(g - w)
    bad = ~(err <= 1e-5 * np.abs(w))
    assert not bad.any(), f"{what}: {bad.sum()} of {w.size} out of 1e-5 (max rel {np.max(err / np.maximum(np.abs(w), 1e-300))})"


def sample_rows(V: int, n: int = 1024, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(V, size=min(n, V), replace=False).tolist())
    rows |= set(range(min(32, V))) | {V - 1, V // 2}
    return np.array(sorted(rows), dtype=np.int64)


def ld_for(D, dtype, pad):
    """Row stride with `pad` extra 16-byte chunks (keeps rows 16-byte aligned)."""
    q = 8 if dtype == torch.bfloat16 else 4
    return ((D + q - 1) // q + pad) * q


# --- coalescing: rows are exact float64 sums rounded once, in two fixed orders
# (the oracle's and the library's); see the docstring of test_gpu_coalesce.

def as_f64(bits: np.ndarray) -> np.ndarray:
    if bits.dtype == np.uint16:
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return bits.astype(np.float64)


def _ordered(bits: np.ndarray) -> np.ndarray:
    if bits.dtype == np.uint16:
        b = bits.astype(np.int64)
        return np.where(b & 0x8000, 0x8000 - (b & 0x7FFF), 0x8000 + b)
    b = bits.view(np.uint32).astype(np.int64)
    return np.where(b & 0x80000000, 0x80000000 - (b & 0x7FFFFFFF), 0x80000000 + b)


def check_coalesced_rows(got: np.ndarray, want: np.ndarray, tok: np.ndarray, U64: np.ndarray, what: str):
    """got/want: [n, D] in the row dtype (fp32 values or bf16 bits); returns the
    number of elements that differ (each at a rounding boundary)."""
    if np.array_equal(got.view(np.uint32) if got.dtype == np.float32 else got,
                      want.view(np.uint32) if want.dtype == np.float32 else want):
        return 0
    ids, inv, counts = np.unique(tok, return_inverse=True, return_counts=True)
    S = np.zeros(want.shape, np.float64)
    A = np.zeros(want.shape, np.float64)
    np.add.at(S, inv, U64)
    np.add.at(A, inv, np.abs(U64))
    diff = (got.view(np.uint32) != want.view(np.uint32)) if got.dtype == np.float32 else (got != want)
    rows, cols = np.nonzero(diff)
    d_ulp = np.abs(_ordered(got[rows, cols]) - _ordered(want[rows, cols]))
    assert (d_ulp == 1).all(), f"{what}: {int((d_ulp > 1).sum())} elements differ by more than 1 ulp"
    assert (counts[rows] > 1).all(), f"{what}: a single-occurrence row is not a copy"
    mid = 0.5 * (as_f64(got[rows, cols]) + as_f64(want[rows, cols]))
    bound = 2.0 * (counts[rows] - 1) * 2.0 ** -53 * A[rows, cols]
    ok = np.abs(S[rows, cols] - mid) <= bound
    assert ok.all(), f"{what}: {int((~ok).sum())} elements differ away from a rounding boundary"
    return int(diff.sum())
