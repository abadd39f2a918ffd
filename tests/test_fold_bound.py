"""CPU checks of the folded layout's accuracy bound (no GPU).

The folded-scale kernel writes each group scale's grid code A (an integer up
to 127 * (1 + 255 + 255^2)) as three balanced base-255 digits and combines
the three exact integer sums in fp32.  The bound of the accuracy guard in
fgq_prepare_weights rests on two facts checked here: the digits' weighted
magnitudes never exceed 3 A, for every code A; and the per-scale limit plus
the fp32 combination bound stay below the 1e-5 tolerance.  The constants are
read from the library's internal header so that the code and this check
cannot drift apart.
"""
import os
import re

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "paper_1705_01462_amd", "csrc", "fgq_internal.h")
KAMAX = 127 * (1 + 255 + 255 * 255)
U = 2.0 ** -24


def constant(name):
    m = re.search(rf"constexpr double {name} = ([0-9.eE+-]+);", open(HEADER).read())
    assert m, name
    return float(m.group(1))


def balanced_digits(A):
    """Three balanced base-255 digits in [-127, 127] of codes A >= 0."""
    r, out = A.copy(), []
    for _ in range(3):
        d = r % 255
        d = np.where(d > 127, d - 255, d)
        out.append(d)
        r = (r - d) // 255
    assert (r == 0).all()
    return out


def test_digits_reconstruct_and_stay_int8():
    A = np.arange(0, KAMAX + 1, dtype=np.int64)
    d = balanced_digits(A)
    assert all(np.abs(x).max() <= 127 for x in d)
    np.testing.assert_array_equal(d[0] + 255 * d[1] + 65025 * d[2], A)


def test_weighted_digit_magnitude_below_three_codes():
    A = np.arange(1, KAMAX + 1, dtype=np.int64)
    d = balanced_digits(A)
    tot = np.abs(d[0]) + 255 * np.abs(d[1]) + 65025 * np.abs(d[2])
    assert (tot < 3 * A).all()
    assert (tot / A).max() > 2.99  # the factor is tight (A = 32513)


def test_guard_constants_meet_the_tolerance():
    max_rel = constant("kFoldMaxRel")
    combine = constant("kFoldCombineRel")
    # three conversions, c0 and two coefficients rounded (3 roundings on each
    # of the three terms, each term at most 3 A |P| in weight), the two fused
    # multiply-adds (3 A |P| and A |P|): 3 * 3 + 3 + 1 = 13 roundings
    assert 13 * U <= combine
    assert max_rel + combine * (1 + max_rel) < 1e-5


def test_grid_step_keeps_the_largest_code():
    # the step rule of the preparation: the smallest fp32 h with amax / h <= KAMAX
    r = np.random.default_rng(1705)
    for amax in np.concatenate([r.uniform(1e-6, 10, 2000), [1.0, 2.0 ** -20, 3.0]]).astype(np.float32):
        h = np.float32(np.float64(amax) / KAMAX)
        if float(h) * KAMAX < float(amax):
            h = np.nextafter(h, np.float32(np.inf))
        assert np.rint(float(amax) / float(h)) <= KAMAX
        # and it is the smallest: one fp32 step down exceeds the range
        lo = np.nextafter(h, np.float32(0))
        assert float(amax) / float(lo) > KAMAX
