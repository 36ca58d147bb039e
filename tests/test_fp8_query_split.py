"""The exactness claim behind scoring fp8 keys on the fp8 matrix cores, checked on the CPU.

The fine stage (Eq. 1 / Eq. 11) multiplies bf16 queries by e4m3 key codes. On the fp8 matrix
cores each bf16 query element x of a head, scaled by a power of two so that the head's largest
magnitude lies in [2^7, 2^8), is written as hi + lo with hi = e4m3(x) and lo = e4m3(x - hi), both
rounded to nearest even. Claimed: hi + lo == x exactly whenever |x| >= 2^-2 (every bf16 element
within 2^10 of its head's largest), and |hi + lo - x| <= 2^-10 below that. Checked here for every
bf16 value in [0, 2^8) and its negative, with torch's e4m3fn cast as the rounding routine.
"""
import numpy as np
import torch


def _all_bf16_below_256():
    bits = np.arange(0, 0x4380, dtype=np.uint32)            # +0 .. 255.0 (0x4380 is 256.0)
    x = (bits << 16).view(np.float32)
    x = x[np.isfinite(x)]
    return np.concatenate([x, -x]).astype(np.float32)


def _e4m3(v: np.ndarray) -> np.ndarray:
    return torch.from_numpy(v).to(torch.float8_e4m3fn).to(torch.float32).numpy()


def test_split_is_exact_within_2_pow_10_of_the_largest():
    x = _all_bf16_below_256()
    hi = _e4m3(x)
    lo = _e4m3((x - hi).astype(np.float32))        # x - hi is exact in float32 (x has 8 bits)
    assert np.array_equal((x.astype(np.float64) - hi) , (x - hi).astype(np.float64))
    err = np.abs(hi.astype(np.float64) + lo - x)
    big = np.abs(x) >= 0.25
    assert big.sum() > 2000
    assert np.all(err[big] == 0.0), x[big][err[big] > 0][:8]
    assert err[~big].max() <= 2.0 ** -10
    assert err[~big].max() > 0                      # the bound is reached: the claim is not vacuous


def test_scaled_head_maximum_fits_e4m3():
    """The largest element after scaling lies below 256, whose rounding stays finite (448 max)."""
    x = _all_bf16_below_256()
    top = x[np.abs(x) >= 128.0]
    assert np.all(np.isfinite(_e4m3(top))) and np.abs(_e4m3(top)).max() <= 256.0
