"""The router's storage format (three bf16 planes per fp32 weight) pinned on
the CPU: hi = bf16(w), mid = bf16(w - hi), lo = bf16(w - hi - mid), each
rounded to nearest even, sum back to w exactly for every normal fp32 weight
whose remainders stay normal (|w| above about 1e-33) and whose bf16 rounding
stays finite (|w| below about 3.39e38, the largest bf16), and the sum is
exact in fp32 in the order the kernel rebuilds it ((hi + mid) + lo).  Written from the
formats' definitions; nothing here comes from the GPU path."""
import numpy as np


def bf16_rne(x):
    b = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint32)
    return (r << 16).view(np.float32)


def planes(w):
    w = np.asarray(w, np.float32)
    hi = bf16_rne(w)
    r1 = (w - hi).astype(np.float32)
    mid = bf16_rne(r1)
    lo = bf16_rne((r1 - mid).astype(np.float32))
    return hi, mid, lo


def test_bf16_rne_reference_values():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1) wins; 1 + 3*2^-8 rounds up
    x = np.array([1.0, 1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -2.5, 0.0], np.float32)
    assert bf16_rne(x).tolist() == [1.0, 1.0, 1 + 2.0 ** -6, -2.5, 0.0]


def test_three_planes_rebuild_exactly():
    rng = np.random.default_rng(0)
    n = 2_000_000
    normal = rng.normal(0, 0.02, n).astype(np.float32)                    # router-weight scale
    wide = (rng.normal(0, 1, n) * 2.0 ** rng.integers(-100, 100, n)).astype(np.float32)
    wide = wide[np.abs(wide) > 2.0 ** -100]
    for w in (normal, wide, np.array([1e30, -3.3e38, 1.17549435e-38 * 2 ** 20, 7.0], np.float32)):
        hi, mid, lo = planes(w)
        rebuilt = ((hi + mid).astype(np.float32) + lo).astype(np.float32)  # the kernel's fp32 order
        assert np.array_equal(rebuilt, w)
        assert np.array_equal(hi.astype(np.float64) + mid + lo, w.astype(np.float64))


def test_weights_past_the_largest_bf16_overflow():
    # the format's upper limit: hi rounds to infinity (the kernel's rounding does the same)
    with np.errstate(invalid="ignore"):  # inf - inf in the remainders
        hi, _, _ = planes(np.array([3.4e38, -3.4e38], np.float32))
    assert np.isinf(hi).all()


def test_small_weights_lose_under_2_pow_minus_125():
    # below the normal range of the remainders the split may lose bits, never more than 2^-125
    rng = np.random.default_rng(1)
    w = (rng.uniform(1, 2, 200_000) * 2.0 ** rng.integers(-126, -100, 200_000)).astype(np.float32)
    hi, mid, lo = planes(w)
    err = np.abs(hi.astype(np.float64) + mid + lo - w.astype(np.float64))
    assert err.max() < 2.0 ** -125
