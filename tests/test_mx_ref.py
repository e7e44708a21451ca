"""Pins of the test-side MX quantiser (tests/mx_ref.py) on values the e4m3 format fixes."""
import numpy as np

from tests.mx_ref import E4M3, e4m3_rne, mx_quantise


def test_e4m3_codes_and_scale():
    # The encoder here, on values whose codes follow from the format: exact values, the
    # midpoint ties (to the even code), the largest value, subnormals and zero.
    assert E4M3[-1] == 448.0 and E4M3[1] == 2.0 ** -9 and E4M3[8] == 2.0 ** -6
    np.testing.assert_array_equal(e4m3_rne(np.array([1.0, 1.125, 1.0625, 1.1875, 448.0, -2.0, 2.0 ** -10, 0.0])),
                                  [0x38, 0x39, 0x38, 0x3A, 0x7E, 0xC0, 0x00, 0x00])
    q, s = mx_quantise(np.r_[np.full(31, 0.5), 1.75 * 2.0 ** 3][None, :])  # amax 14 = 1.75 2^3: e = -5
    assert s[0, 0] == 127 - 5 and q[0, 31] == 0x7E
