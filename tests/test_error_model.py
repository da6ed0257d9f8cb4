"""CPU pins of the MFMA error-model helpers used as GEMM tolerances."""

import numpy as np

from gpu_util import e4m3_exponent, mfma_dot_bound


def test_e4m3_exponent_values():
    codes = np.array([0x00, 0x80, 0x01, 0x07, 0x08, 0x38, 0x7E, 0xFE], np.uint8)
    assert np.array_equal(e4m3_exponent(codes), [-np.inf, -np.inf, -6, -6, -6, 0, 8, 8])


def test_dot_bound_hand_worked():
    # one K-group; a = 448 at k=0 (exponent 8), 1.0 elsewhere (exponent 0) in span 0;
    # b = 1.0 everywhere (exponent 0). Span 0 (k < 16): 2^(8+0); spans 1..7: 2^(0+0).
    a = np.full((1, 128), 0x38, np.uint8)
    a[0, 0] = 0x7E
    b = np.full((128, 128), 0x38, np.uint8)
    bound = mfma_dot_bound(a, b)
    assert len(bound) == 1 and bound[0].shape == (1, 128)
    want = 16 * 2.0 ** -13 * (2.0 ** 8 + 7 * 1.0)
    assert np.all(bound[0] == want)
    # zero spans contribute nothing
    a[0, :] = 0
    assert np.all(mfma_dot_bound(a, b)[0] == 0)
