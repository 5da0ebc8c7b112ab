"""Pins of the oracle's max pooling (the pooling layers between the
convolution blocks of the networks in Sec. 5.2), against facts fixed outside
the oracle: a hand-computed example, special cases with known answers, brute
force on tiny inputs, and scipy.ndimage's maximum filter."""
import itertools

import numpy as np
import pytest
from scipy import ndimage

import oracle


def test_hand_computed_example():
    # 1 image, 1 channel, 4x4, 2x2 windows, stride 2: the max of each quadrant
    x = np.array([[1, 5, 2, 0],
                  [3, -1, 7, 4],
                  [0, 0, -2, -3],
                  [9, 1, -4, -1]], np.float32).reshape(1, 1, 4, 4)
    y = oracle.maxpool2d(x, 2, 2, 2, 0, "NCHW")
    assert y.tolist() == [[[[5.0, 7.0], [9.0, -1.0]]]]
    # 3x3 window, stride 1, pad 1: the max over each 3x3 neighbourhood inside the image
    y = oracle.maxpool2d(x, 3, 3, 1, 1, "NCHW")
    assert y[0, 0].tolist() == [[5, 7, 7, 7], [5, 7, 7, 7], [9, 9, 7, 7], [9, 9, 1, -1]]


def test_unit_window_is_identity_and_full_window_is_global_max():
    rng = np.random.Generator(np.random.PCG64(8))
    x = rng.standard_normal((3, 4, 6, 7)).astype(np.float32)
    assert np.array_equal(oracle.maxpool2d(x, 1, 1, 1, 0, "NCHW"), x)
    g = oracle.maxpool2d(x, 6, 7, 1, 0, "NCHW")
    assert g.shape == (3, 4, 1, 1)
    assert np.array_equal(g[:, :, 0, 0], x.max(axis=(2, 3)))


def _brute(x, R, S, sh, sw, ph, pw):
    N, C, H, W = x.shape
    Ho, Wo = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    y = np.empty((N, C, Ho, Wo), np.float32)
    for b, c, oh, ow in itertools.product(range(N), range(C), range(Ho), range(Wo)):
        vals = [x[b, c, oh * sh + r - ph, ow * sw + s - pw] for r in range(R) for s in range(S)
                if 0 <= oh * sh + r - ph < H and 0 <= ow * sw + s - pw < W]
        y[b, c, oh, ow] = max(vals)
    return y


@pytest.mark.parametrize("R,S,sh,sw,ph,pw", [(2, 2, 2, 2, 0, 0), (3, 3, 2, 2, 1, 1), (3, 2, 1, 2, 1, 0),
                                             (3, 3, 2, 2, 0, 0), (5, 3, 3, 1, 2, 1)])
def test_brute_force_tiny(R, S, sh, sw, ph, pw):
    rng = np.random.Generator(np.random.PCG64(R * 10 + S))
    x = rng.standard_normal((2, 3, 9, 8)).astype(np.float32)
    y = oracle.maxpool2d(x, R, S, (sh, sw), (ph, pw), "NCHW")
    assert np.array_equal(y, _brute(x, R, S, sh, sw, ph, pw))
    # HWCN is the same logical operation
    xh = np.ascontiguousarray(np.transpose(x, (2, 3, 1, 0)))
    yh = oracle.maxpool2d(xh, R, S, (sh, sw), (ph, pw), "HWCN")
    assert np.array_equal(np.transpose(yh, (3, 2, 0, 1)), y)


@pytest.mark.parametrize("R,sh,ph", [(3, 2, 1), (2, 2, 0), (3, 1, 1), (3, 2, 0)])
def test_matches_scipy_maximum_filter(R, sh, ph):
    rng = np.random.Generator(np.random.PCG64(100 + R))
    x = rng.standard_normal((2, 2, 15, 12)).astype(np.float32)
    y = oracle.maxpool2d(x, R, R, sh, ph, "NCHW")
    # maximum over the window anchored at (oh*sh - ph, ow*sw - pw), padding -inf
    xp = np.pad(x, ((0, 0), (0, 0), (ph, ph), (ph, ph)), constant_values=-np.inf)
    f = ndimage.maximum_filter(xp, size=(1, 1, R, R), mode="constant", cval=-np.inf,
                               origin=(0, 0, -(R // 2), -(R // 2)))
    Ho, Wo = y.shape[2:]
    ref = f[:, :, (np.arange(Ho) * sh)[:, None], (np.arange(Wo) * sh)[None, :]]
    assert np.array_equal(y, ref)


def test_nan_propagates():
    x = np.zeros((1, 1, 4, 4), np.float32)
    x[0, 0, 1, 2] = np.nan
    y = oracle.maxpool2d(x, 2, 2, 2, 0, "NCHW")
    assert np.isnan(y[0, 0, 0, 1]) and not np.isnan(y[0, 0, 0, 0]) and not np.isnan(y[0, 0, 1, :]).any()
