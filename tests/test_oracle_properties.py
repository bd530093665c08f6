"""Property-based pins of the CPU oracle (hypothesis, derandomized): the same
independent references as pins.py, over drawn shapes and values instead of
fixed cases.

* encode == brute-force enumeration of the 16 root-to-leaf paths, with
  values drawn to include exact ties, signed zeros, infinities and NaN;
* lut_accumulate's int32 sums == the one-hot encoder output times the
  stacked, shifted code table in int64 (the dense form of the gather-sum);
* y == the single fp32 rounding of acc 2^e_min + bias32, in exact rationals,
  when the offsets' double sum is exact.
"""
from fractions import Fraction

import numpy as np
import pytest

hyp = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

import pins  # noqa: E402

K = pins.K
SETTINGS = settings(max_examples=120, deadline=None, derandomize=True)


@st.composite
def encode_case(draw):
    N = draw(st.integers(0, 24))
    D = draw(st.integers(1, 12))
    C = draw(st.integers(1, 9))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    rng = np.random.default_rng(seed)
    thr = (rng.standard_normal((C, 15)) * 2).astype(np.float32)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan], dtype=np.float32)
    A = (rng.standard_normal((N, D)) * 2).astype(np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    if N:
        # a third of the entries: a threshold of the row's codebooks exactly,
        # or a special value
        mask = rng.random((N, D)) < 0.33
        picks = np.concatenate([thr.ravel(), specials])
        A[mask] = rng.choice(picks, size=int(mask.sum()))
    if draw(st.booleans()):
        thr[rng.random(thr.shape) < 0.1] = 0.0
    return A, split, thr


@SETTINGS
@given(encode_case())
def test_encode_is_the_brute_force_leaf(orc, case):
    A, split, thr = case
    idx = orc.encode(A, split, thr)
    assert idx.shape == (A.shape[0], split.shape[0])
    assert np.array_equal(idx, pins.brute_force_leaf(A, split, thr))


@st.composite
def accumulate_case(draw):
    N = draw(st.integers(0, 30))
    C = draw(st.integers(1, 24))
    M = draw(st.integers(1, 17))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    maxsh = draw(st.integers(0, 12))
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    lut = rng.integers(-128, 128, size=(C, K, M)).astype(np.int8)
    e = rng.integers(-4, -4 + maxsh + 1, size=C)
    scale = np.ldexp(np.float32(1), e.astype(np.int32)).astype(np.float32)
    offset = rng.integers(-2 ** 16, 2 ** 16, size=C).astype(np.float32)   # double sum exact
    return idx, lut, scale, offset


@SETTINGS
@given(accumulate_case())
def test_accumulate_is_the_one_hot_product(orc, case):
    idx, lut, scale, offset = case
    C = lut.shape[0]
    acc, _ = orc.lut_accumulate(idx, lut, scale, offset)
    ex = pins.exponents(scale)
    Q = (lut.astype(np.int64) * (2 ** (ex - ex.min()))[:, None, None]).reshape(C * K, lut.shape[2])
    assert np.array_equal(acc.astype(np.int64), pins.one_hot(idx) @ Q)


@SETTINGS
@given(accumulate_case())
def test_output_is_one_rounding(orc, case):
    idx, lut, scale, offset = case
    acc, y = orc.lut_accumulate(idx, lut, scale, offset)
    emin = int(pins.exponents(scale).min())
    bias = pins.rne32(sum(Fraction(float(o)) for o in offset))
    N, M = acc.shape
    for n in range(min(N, 6)):
        for m in range(M):
            want = pins.rne32(Fraction(int(acc[n, m])) * Fraction(2) ** emin + Fraction(bias))
            assert float(y[n, m]) == want
