"""CPU checks of the synthetic inputs: they have the structure of the paper's
workloads that the recipe claims (the generators run on the CPU here)."""
import torch

from paper_2607_01455_amd import workloads as wl


def _bf16_to_f64(t):
    return t.to(torch.float64)


def test_lmhead_batch_is_a_cross_entropy_gradient():
    # appendix "The LM Head Factorizes Like the Embedding Table": dY = q - onehot(y)
    # (here over T for a mean loss): each row sums to zero, holds one negative
    # entry (the target) and a positive softmax background
    cfg = wl.Config("lmh_cpu", 500, 64, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=40)
    dY, H = wl.make_lmhead_batch(cfg, 1, seed=3, device="cpu")
    assert dY.shape == (40, 500) and H.shape == (40, 64)
    assert dY.dtype == torch.bfloat16 and H.dtype == torch.bfloat16
    y = _bf16_to_f64(dY) * 40
    assert torch.all((y < 0).sum(dim=1) == 1)
    # row sums vanish up to the bf16 rounding of each entry (relative 2^-8)
    assert torch.all(y.sum(dim=1).abs() <= 2.0 ** -8 * y.abs().sum(dim=1))
    assert torch.all(y.min(dim=1).values < -0.5)
    # hidden states: unit scale per coordinate
    h = _bf16_to_f64(H)
    assert 0.8 < h.std().item() < 1.2 and abs(h.mean().item()) < 0.1


def test_lmhead_targets_follow_the_token_frequencies():
    # targets are Zipf(1.1) over the V rows: the most frequent ids dominate
    cfg = wl.Config("lmh_cpu", 1000, 8, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=4000)
    dY, _ = wl.make_lmhead_batch(cfg, 1, seed=4, device="cpu")
    tgt = torch.argmin(dY.to(torch.float32), dim=1)
    counts = torch.bincount(tgt, minlength=1000).to(torch.float64)
    p = wl.zipf_probs(1000)
    assert abs(counts[0].item() / 4000 - p[0].item()) < 0.03
    assert counts[:10].sum() > counts[500:].sum()
    # the softmax background of a row also decreases with the rank on average
    q = dY.to(torch.float64).clamp(min=0).mean(dim=0)
    assert q[:10].mean() > 5 * q[500:].mean()


def test_lmhead_batches_are_reproducible_and_padding_is_separate():
    cfg = wl.Config("lmh_cpu", 300, 40, torch.bfloat16, torch.bfloat16, 1, "logits", batch_tokens=20)
    a = wl.make_lmhead_batch(cfg, 2, seed=5, device="cpu")
    b = wl.make_lmhead_batch(cfg, 2, seed=5, device="cpu")
    c = wl.make_lmhead_batch(cfg, 3, seed=5, device="cpu")
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    assert not torch.equal(a[0], c[0])
    d, h = wl.make_lmhead_batch(cfg, 2, seed=5, device="cpu", ldy=312, ldh=48)
    assert d.stride(0) == 312 and h.stride(0) == 48
    assert d.shape == (20, 300) and h.shape == (20, 40)


def test_lmhead_flops():
    assert wl.lmhead_flops(16384, 128256, 4096) == 17214228922368
