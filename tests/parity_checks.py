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


# W bars.  The library's update term g / (sqrt(rhat chat / s) + eps) uses its
# own r and c, which agree with the oracle's to 1e-5 (check_state), so the
# term itself may differ by ~1e-5 of its size; the fp32 arithmetic around it
# adds ~2^-23 of |W_prev|.  Hence:
# * fp32: |W - W_ref| <= 1e-5 max(|W_ref|, |W_prev - W_ref|), the update's
#   size standing in when the update cancels most of W_prev; elements that
#   pass only through the update's size are counted and printed.
# * bf16: within one ulp of W_ref (the final rounding dominates), except where
#   the update cancelled the previous weight, |W_ref| < 2^-7 |W_prev| (the
#   error above reaches one bf16 ulp only far below that), and then within
#   1e-5 max(|W_ref|, |W_prev - W_ref|).  These elements are counted and
#   capped: at most CANCEL_CAP of the checked elements per call, with a floor
#   of CANCEL_FLOOR elements for small samples (at the ~1e-6 rate seen over
#   whole tables, 5 or more in 3e5 elements has a chance of about 1e-4).
# Session totals are printed at the end of the run.
CANCEL_RATIO_BF16 = 2.0 ** -7
CANCEL_CAP = 2e-6
CANCEL_FLOOR = 4
cancel_tally = {"bf16": [0, 0, 0], "fp32": [0, 0, 0]}   # calls, checked, through the update bar


def check_w(got: np.ndarray, want: np.ndarray, prev: np.ndarray, what: str) -> int:
    """W against the oracle by the bars above; returns the number of elements
    that passed through the update-size bar."""
    if got.dtype == np.uint16:
        beyond = np.abs(ordered16(got) - ordered16(want)) > 1
        gv, wv, pv = (bf16_values(x[beyond]) for x in (got, want, prev))
        upd_ok = np.abs(gv - wv) <= 1e-5 * np.maximum(np.abs(wv), np.abs(pv - wv))
        ok = (np.abs(wv) < CANCEL_RATIO_BF16 * np.abs(pv)) & upd_ok
        assert ok.all(), (
            f"{what}: {(~ok).sum()} bf16 elements beyond one ulp without cancellation; "
            f"first: got {gv[~ok][:3]} want {wv[~ok][:3]} prev {pv[~ok][:3]}")
        cap = max(CANCEL_FLOOR, int(np.ceil(CANCEL_CAP * got.size)))
    else:
        g64, w64, p64 = got.astype(np.float64), want.astype(np.float64), prev.astype(np.float64)
        err = np.abs(g64 - w64)
        ok = err <= 1e-5 * np.maximum(np.abs(w64), np.abs(p64 - w64))
        assert ok.all(), (f"{what}: {(~ok).sum()} fp32 elements beyond 1e-5 of max(|W_ref|, |update|); "
                          f"max err {err.max()}")
        beyond = ~(err <= 1e-5 * np.abs(w64))
        cap = None
    k = int(beyond.sum())
    tally = cancel_tally["bf16" if got.dtype == np.uint16 else "fp32"]
    tally[0] += 1
    tally[1] += int(got.size)
    tally[2] += k
    if k:
        print(f"  {what}: {k} of {got.size} elements passed through the update-size bar"
              + (f" (cap {cap})" if cap is not None else ""), flush=True)
    if cap is not None:
        assert k <= cap, f"{what}: {k} cancellation elements of {got.size}, above the cap of {cap}"
    return k


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
