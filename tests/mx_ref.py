"""An MX (e4m3 elements, one E8M0 scale per 32 columns) quantiser written from the OCP formats,
the reference of the fp8-MFMA variant's activation quantisation in the tests: the scale of a
block with largest magnitude m is the smallest 2^e with m / 2^e <= 448 (the largest e4m3 value),
and each element x / 2^e rounds to the nearest e4m3 value, ties to the even code."""
import numpy as np


def _e4m3_values():
    """Magnitudes of the e4m3fn codes 0x00..0x7E (0x7F is NaN), ascending."""
    v = []
    for c in range(0x7F):
        e, m = c >> 3, c & 7
        v.append(m / 8.0 * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7))
    return np.array(v)


E4M3 = _e4m3_values()


def e4m3_rne(v: np.ndarray) -> np.ndarray:
    """Codes of |v| <= 448 rounded to the nearest e4m3 value, ties to the even code; the sign in bit 7."""
    a = np.abs(v)
    assert np.all(a <= 448.0)
    hi = np.clip(np.searchsorted(E4M3, a, side="left"), 0, len(E4M3) - 1)
    lo = np.maximum(hi - 1, 0)
    d_hi, d_lo = E4M3[hi] - a, a - E4M3[lo]
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(E4M3[hi] == a, hi, np.where(pick_hi, hi, lo)).astype(np.uint8)
    return code | np.where(np.signbit(v), 0x80, 0).astype(np.uint8)


def mx_quantise(x: np.ndarray):
    """x [T][H] (exact float values) -> (codes [T][H], scale bytes [T][H / 32])."""
    T, H = x.shape
    blk = x.reshape(T, H // 32, 32)
    amax = np.abs(blk).max(axis=2)
    mant, ex = np.frexp(amax)  # amax = mant 2^ex, mant in [0.5, 1)
    ea = ex - 1                # amax = (2 mant) 2^ea, 2 mant in [1, 2)
    e = ea - 8 + (2 * mant > 1.75)
    s = np.where(amax == 0, 127, np.clip(e + 127, 0, 253)).astype(np.int64)
    scaled = blk * np.ldexp(1.0, (127 - s))[:, :, None]
    return e4m3_rne(scaled).reshape(T, H), s.astype(np.uint8)
