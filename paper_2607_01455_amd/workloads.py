"""Seeded synthetic workloads for the Ember step.  No Ember arithmetic here.

The paper trains on FineWeb, Alpaca, Countdown and LlamaGen data with
pretrained models; none of that is used.  These generators stand in for them
with the shapes of the paper's token tables (vocabularies of 32k to 262k rows,
widths 896 to 8192) and the gradient structure its analysis describes:
heavy-tailed per-token gradient scale (row norm proportional to token
frequency, Section 2.2 and the appendix on the LM head) and one-hot embedding
gradients that touch only the tokens of a batch (appendix "Decomposing the
Squared Gradient").

Both the HIP library and the CPU oracle receive the same materialised
tensors, so any seeded generator would do; these use torch generators on the
target device so that gigabyte-sized inputs are made in milliseconds.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Config:
    name: str
    V: int
    D: int
    w_dtype: torch.dtype
    g_dtype: torch.dtype
    steps: int
    grad: str          # "normal" | "loguniform_rows" | "zipf_rows" | "sparse_zipf" | "logits"
    w_std: float = 0.02
    g_std: float = 1e-3
    batch_tokens: int = 0  # sparse: token ids per step


CONFIGS = {
    # 1024 x 64 fp32, 3 steps: small enough for the oracle to check every element
    "tiny": Config("tiny", 1024, 64, torch.float32, torch.float32, 3, "normal"),
    # 32000 x 4096 fp32 LM head, per-row gradient scale log-uniform in [1e-2, 1e2]
    "lmhead32k": Config("lmhead32k", 32000, 4096, torch.float32, torch.float32, 10, "loguniform_rows"),
    # 128256 x 4096 bf16 LM head, per-row scale from Zipf(1.1) token frequencies
    "lmhead128k": Config("lmhead128k", 128256, 4096, torch.bfloat16, torch.bfloat16, 10, "zipf_rows"),
    # 128256 x 4096 bf16 input embedding, 8 x 2048 Zipf(1.1) token ids per step
    "embed128k": Config("embed128k", 128256, 4096, torch.bfloat16, torch.bfloat16, 10, "sparse_zipf",
                        batch_tokens=8 * 2048),
    # 128256 x 4096 bf16 LM head whose gradient is formed from 8 x 2048 tokens:
    # logits gradient [16384, 128256] and hidden states [16384, 4096], bf16
    "lmhead128k_wgrad": Config("lmhead128k_wgrad", 128256, 4096, torch.bfloat16, torch.bfloat16, 3, "logits",
                               batch_tokens=8 * 2048),
    # tied 151936 x 896 fp32 table
    "tied152k": Config("tied152k", 151936, 896, torch.float32, torch.float32, 5, "normal"),
    # 262144 x 8192 bf16 table
    "wide262k": Config("wide262k", 262144, 8192, torch.bfloat16, torch.bfloat16, 5, "normal"),
}

ZIPF_EXPONENT = 1.1


def _gen(device, *seed_parts: int) -> torch.Generator:
    g = torch.Generator(device=device)
    s = 0x9E3779B1
    for p in seed_parts:
        s = (s * 1000003 + int(p) + 1) % (2 ** 63 - 1)
    g.manual_seed(s)
    return g


def zipf_probs(V: int, exponent: float = ZIPF_EXPONENT, device="cpu") -> torch.Tensor:
    """p_i proportional to (i + 1)^-exponent: row i is the token of frequency rank i + 1."""
    ranks = torch.arange(1, V + 1, dtype=torch.float64, device=device)
    w = ranks.pow(-exponent)
    return w / w.sum()


def row_scales(cfg: Config, seed: int, device) -> torch.Tensor | None:
    """Per-row gradient scale (float32 [V]) or None for a flat scale."""
    if cfg.grad == "loguniform_rows":
        u = torch.rand(cfg.V, generator=_gen(device, seed, 1 << 20), device=device, dtype=torch.float64)
        return torch.pow(10.0, 4.0 * u - 2.0).float()
    if cfg.grad == "zipf_rows":
        # V * p_i: mean 1, from ~17000 (most frequent token) down to ~0.04
        return (zipf_probs(cfg.V, device=device) * cfg.V).float()
    return None


def make_weights(cfg: Config, seed: int = 0, device="cuda", ld: int | None = None) -> torch.Tensor:
    """W ~ N(0, w_std) in the table's dtype; optional padded row stride ld >= D."""
    ld = cfg.D if ld is None else ld
    out = torch.empty(cfg.V, ld, dtype=cfg.w_dtype, device=device)
    g = _gen(device, seed, 0)
    for r0 in range(0, cfg.V, 16384):
        r1 = min(cfg.V, r0 + 16384)
        out[r0:r1] = (torch.randn(r1 - r0, ld, generator=g, device=device) * cfg.w_std).to(cfg.w_dtype)
    return out[:, :cfg.D]


def make_dense_grad(cfg: Config, step: int, seed: int = 0, device="cuda", scales=None,
                    ld: int | None = None) -> torch.Tensor:
    """Dense G at step t: N(0, g_std) per element, times the row scale if any."""
    ld = cfg.D if ld is None else ld
    out = torch.empty(cfg.V, ld, dtype=cfg.g_dtype, device=device)
    g = _gen(device, seed, 2 + step)
    for r0 in range(0, cfg.V, 16384):
        r1 = min(cfg.V, r0 + 16384)
        x = torch.randn(r1 - r0, ld, generator=g, device=device) * cfg.g_std
        if scales is not None:
            x *= scales[r0:r1, None]
        out[r0:r1] = x.to(cfg.g_dtype)
    return out[:, :cfg.D]


def make_sparse_batch(cfg: Config, step: int, seed: int = 0, device="cuda", shuffle: bool = False):
    """(idx int64 [n], G_rows [n, D]) for one step of the embedding table.

    batch_tokens ids are drawn with replacement from Zipf(1.1) over the V rows;
    idx holds the distinct ids (ascending, or shuffled).  The gradient of a row
    that occurs k times is the sum of k independent N(0, g_std) vectors, drawn
    here directly as sqrt(k) * N(0, g_std), which has the same distribution.
    """
    # ids on the CPU generator: its multinomial and randperm are reproducible
    # for a given seed, which the device versions are not
    gc = _gen("cpu", seed, 1000 + step)
    p = zipf_probs(cfg.V).float()
    ids = torch.multinomial(p, cfg.batch_tokens, replacement=True, generator=gc)
    uniq, counts = torch.unique(ids, sorted=True, return_counts=True)
    if shuffle:
        perm = torch.randperm(uniq.numel(), generator=gc)
        uniq, counts = uniq[perm], counts[perm]
    g = _gen(device, seed, 1000 + step)
    x = torch.randn(uniq.numel(), cfg.D, generator=g, device=device) * cfg.g_std
    x *= counts.to(device=device, dtype=torch.float32).sqrt()[:, None]
    return uniq.to(device=device, dtype=torch.int64).contiguous(), x.to(cfg.g_dtype)


def make_token_batch(cfg: Config, step: int, seed: int = 0, device="cuda", dtype=None, ld: int | None = None):
    """(tok int64 [P], U [P, D]) for one step of the embedding table before
    coalescing: batch_tokens ids drawn with replacement from Zipf(1.1) over the
    V rows, in batch order, and one back-propagated signal N(0, g_std) per
    position (the per-position gradient rows whose per-id sums the sparse step
    takes)."""
    gc = _gen("cpu", seed, 2000 + step)
    p = zipf_probs(cfg.V).float()
    tok = torch.multinomial(p, cfg.batch_tokens, replacement=True, generator=gc)
    ld = cfg.D if ld is None else ld
    dtype = cfg.g_dtype if dtype is None else dtype
    g = _gen(device, seed, 2000 + step)
    U = torch.empty(cfg.batch_tokens, ld, dtype=dtype, device=device)
    for r0 in range(0, cfg.batch_tokens, 16384):
        r1 = min(cfg.batch_tokens, r0 + 16384)
        U[r0:r1] = (torch.randn(r1 - r0, ld, generator=g, device=device) * cfg.g_std).to(dtype)
    return tok.to(device=device, dtype=torch.int64).contiguous(), U[:, :cfg.D]


def make_lmhead_batch(cfg: Config, step: int, seed: int = 0, device="cuda", T: int | None = None,
                      ldy: int | None = None, ldh: int | None = None):
    """(dY [T, V], H [T, D]), both bf16, for one step of an LM head whose
    weight gradient is G = dY^T H (appendix "The LM Head Factorizes Like the
    Embedding Table").

    H: hidden states N(0, 1) per coordinate (after the final normalisation).
    Targets y_m: Zipf(1.1) over the V rows.  Logits z_mi = log p_i + N(0, 1),
    so the softmax background follows the token frequencies, as in the
    appendix's decomposition of G into a frequency term and a target-count
    term.  dY = (softmax(z_m) - onehot(y_m)) / T, the gradient of the mean
    cross-entropy over the T positions.  Optional padded row strides.
    """
    T = cfg.batch_tokens if T is None else T
    V, D = cfg.V, cfg.D
    ldy = V if ldy is None else ldy
    ldh = D if ldh is None else ldh
    gc = _gen("cpu", seed, 3000 + step)
    p = zipf_probs(V)
    y = torch.multinomial(p.float(), max(T, 1), replacement=True, generator=gc)[:T].to(device)
    logp = p.log().float().to(device)
    g = _gen(device, seed, 3000 + step)
    H = torch.empty(T, ldh, dtype=torch.bfloat16, device=device)
    dY = torch.empty(T, ldy, dtype=torch.bfloat16, device=device)
    for m0 in range(0, T, 1024):
        m1 = min(T, m0 + 1024)
        H[m0:m1] = torch.randn(m1 - m0, ldh, generator=g, device=device).to(torch.bfloat16)
        z = torch.randn(m1 - m0, V, generator=g, device=device) + logp[None, :]
        q = torch.softmax(z, dim=1)
        q[torch.arange(m1 - m0, device=device), y[m0:m1]] -= 1.0
        dY[m0:m1, :V] = (q / T).to(torch.bfloat16)
        if ldy > V:
            dY[m0:m1, V:] = torch.randn(m1 - m0, ldy - V, generator=g, device=device).to(torch.bfloat16)
    return dY[:, :V], H[:, :D]


def lmhead_flops(T: int, V: int, D: int) -> int:
    """Multiply-adds of G = dY^T H, counted as two flops each."""
    return 2 * T * V * D


def coalesce_bytes(P: int, n: int, D: int, u_size: int, g_size: int) -> int:
    """HBM bytes coalescing must move: the token ids and per-position rows read
    once, the distinct ids and summed rows written once."""
    return 8 * P + P * D * u_size + 8 * n + n * D * g_size


def algorithmic_bytes(V: int, D: int, w_size: int, g_size: int, rows: int | None = None) -> int:
    """HBM bytes one step must move: G read twice, W read and written once on
    the `rows` rows that carry gradient (all V if dense), r read and written,
    c read and written.  The sparse step also reads its int64 index list."""
    rows = V if rows is None else rows
    b = rows * D * (2 * g_size + 2 * w_size) + 8 * (V + D)
    if rows != V:
        b += 8 * rows
    return b


def rowonly_algorithmic_bytes(V: int, D: int, w_size: int, g_size: int, rows: int | None = None) -> int:
    """HBM bytes one row-only step must move: each row's statistic depends on
    that row alone, so G is read once; W read and written once on the rows with
    gradient, r read and written, plus the sparse step's int64 index list."""
    rows = V if rows is None else rows
    b = rows * D * (g_size + 2 * w_size) + 8 * V
    if rows != V:
        b += 8 * rows
    return b
