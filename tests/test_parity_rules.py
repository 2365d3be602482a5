"""The W comparison rule of the GPU parity tests (parity_checks.check_w),
checked on planted cases on the CPU: one bf16 ulp passes, two fail unless the
update cancelled the previous weight, cancellation elements are counted and
capped, and the fp32 bar is relative to the larger of the reference value and
the update."""
import numpy as np
import pytest

import parity_checks as pc


@pytest.fixture(autouse=True)
def keep_tally():
    # planted cases stay out of the session's count of real comparisons
    saved = {k: list(v) for k, v in pc.cancel_tally.items()}
    yield
    pc.cancel_tally.update(saved)


def bf16_bits(x):
    b = np.asarray(x, np.float32).view(np.uint32)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def step_ulps(bits, k):
    return (bits.astype(np.int64) + k).astype(np.uint16)   # positive values only


def test_bf16_one_ulp_passes_two_fail_without_cancellation():
    want = bf16_bits(np.linspace(0.5, 1.5, 1000))
    prev = bf16_bits(np.full(1000, 1.0))
    assert pc.check_w(step_ulps(want, 1), want, prev, "one ulp") == 0
    got = want.copy()
    got[7] = step_ulps(want[7:8], 2)[0]
    with pytest.raises(AssertionError, match="without cancellation"):
        pc.check_w(got, want, prev, "two ulps")


def test_bf16_cancellation_element_is_counted_and_capped():
    n = 10000
    prev = bf16_bits(np.full(n, 1.0))
    want = bf16_bits(np.full(n, 1.0))
    # element 3: the update cancelled W_prev down to ~1e-6 (|W_ref| < 2^-7 |W_prev|)
    want[3] = bf16_bits(np.float32(1e-6))
    got = want.copy()
    got[3] = step_ulps(want[3:4], 5)[0]           # 5 ulps of 1e-6: ~2e-8 << 1e-5 |W_prev|
    assert pc.check_w(got, want, prev, "cancel") == 1
    # more cancellation elements than the cap (max(4, 2e-6 n) = 4 here)
    for i in (4, 5, 6, 8):
        want[i] = want[3]
        got[i] = got[3]
    with pytest.raises(AssertionError, match="above the cap"):
        pc.check_w(got, want, prev, "over cap")


def test_bf16_cancellation_is_bounded_by_the_previous_weight():
    prev = bf16_bits(np.full(4, 1.0))
    want = bf16_bits(np.full(4, 1e-3))            # cancelled (|W_ref| < 2^-7)
    got = bf16_bits(np.full(4, 1e-3 + 5e-5))      # off by 5e-5 > 1e-5 |W_prev|
    with pytest.raises(AssertionError, match="without cancellation"):
        pc.check_w(got, want, prev, "too far")


def test_fp32_bar_is_relative_to_the_reference_or_the_update():
    prev = np.full(100, 1.0, np.float32)
    want = np.full(100, 0.999, np.float32)        # a small update (1e-3)
    got = want * np.float32(1 + 5e-6)
    assert pc.check_w(got, want, prev, "inside") == 0
    got = want.copy()
    got[0] = np.float32(0.999 * (1 + 3e-5))       # 3e-5 of W_ref, far beyond 1e-5 of the update
    with pytest.raises(AssertionError, match="beyond 1e-5"):
        pc.check_w(got, want, prev, "outside")
    want[1] = np.float32(1e-3)                    # the update cancelled W_prev: |update| ~ 1
    got = want.copy()
    got[1] = np.float32(1e-3 + 2e-6)              # 2e-3 of W_ref, 2e-6 of the update
    assert pc.check_w(got, want, prev, "cancelled") == 1
    got[1] = np.float32(1e-3 + 2e-5)              # 2e-5 of the update
    with pytest.raises(AssertionError, match="beyond 1e-5"):
        pc.check_w(got, want, prev, "too far")
