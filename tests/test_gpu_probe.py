"""GPU test of the streaming probe kernels (the reference rates the benchmark reports
beside the Ember passes): copy and two-operand add are checked element by
element against torch, over sizes with a ragged grid-stride tail."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n16", [1, 37, 4096 * 4 * 256 + 17])
def test_stream_probe_copy_and_add(n16):
    from paper_2607_01455_amd import ember
    print(f"stream probe, {n16} chunks of 16 bytes", flush=True)
    g = torch.Generator(device="cuda").manual_seed(n16)
    a = torch.randint(-2 ** 31, 2 ** 31 - 1, (n16 * 4,), generator=g, device="cuda", dtype=torch.int32)
    b = torch.randint(-2 ** 31, 2 ** 31 - 1, (n16 * 4,), generator=g, device="cuda", dtype=torch.int32)
    dst = torch.zeros_like(a)
    ember.ember_stream_probe(1, dst, a)
    torch.cuda.synchronize()
    assert torch.equal(dst, a)
    ember.ember_stream_probe(2, dst, a, b)
    torch.cuda.synchronize()
    want = (a.to(torch.int64) + b.to(torch.int64) + 2 ** 31) % 2 ** 32 - 2 ** 31   # 32-bit wrap-around
    assert torch.equal(dst.to(torch.int64), want)
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    ember.ember_stream_probe(0, sink, a)
    torch.cuda.synchronize()
