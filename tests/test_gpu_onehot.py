"""The one-hot product accumulate (int8 tables, C % 16 == 0, 48 <= C <= 128,
M % 4 == 0, M >= 128, 16,384 rows and more) against the oracle: int32 sums and outputs
bit-exact.  The cases cover the two instantiations (64 and 128 staged
codebooks), codebook counts that leave padded codebooks, column counts that
leave a ragged last slice, row counts with a ragged last tile, codes of
-128, and block exponents whose spread needs one, two and three shift groups
(one-hot entries must fit int8: 2^0 .. 2^6 per group)."""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def codes(C, M, seed, max_shift, with_min=False):
    lut, scale, offset = W.random_codes(C, M, seed=seed, max_shift=max_shift)
    if with_min:   # -128 in a tenth of the entries
        rng = np.random.default_rng(seed + 7)
        lut[rng.random(lut.shape) < 0.1] = -128
    e = np.frexp(scale)[1]
    assert 128 * int(np.sum(2.0 ** (e - e.min()))) <= 2 ** 31   # the documented no-overflow bound
    return lut, scale, offset


def sample_rows(N, seed, n=512):
    if N <= 20000:
        return np.arange(N)
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(128), np.arange(N - 128, N), rng.integers(0, N, n)]))


CASES = [  # (N, C, M, max_shift, want_acc, -128 codes)
    (16384, 64, 512, 1, False, False),        # dense_hidden's table shape
    (16384 + 37, 64, 512, 6, True, True),     # one group at its widest, ragged last tile
    (16500, 48, 160, 3, True, False),         # 16 padded codebooks, ragged last slice
    (17000, 48, 128, 0, False, True),         # one slice exactly
    (16411, 80, 132, 7, True, False),         # 128 staged codebooks (48 padded), two shift groups
    (16384, 128, 128, 13, True, True),        # two groups, the second at its widest
    (16390, 64, 132, 2, True, False),         # a last slice of four columns
    (18000, 96, 200, 16, False, False),       # three shift groups
    (40000, 128, 1000, 1, True, False),       # wide_layer's codebooks, sampled rows
]


@pytest.mark.parametrize("N,C,M,max_shift,want_acc,with_min", CASES,
                         ids=[f"N{c[0]}-C{c[1]}-M{c[2]}-sh{c[3]}" for c in CASES])
def test_onehot_accumulate(orc, N, C, M, max_shift, want_acc, with_min):
    seed = N + 7 * C + M + max_shift
    idx = W.random_indices(N, C, seed=seed)
    lut, scale, offset = codes(C, M, seed + 1, max_shift, with_min)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=want_acc)
    r = sample_rows(N, seed)
    racc, ry = orc.lut_accumulate(idx[r], lut, scale, offset)
    assert np.array_equal(host(y)[r], ry)
    if want_acc:
        assert np.array_equal(host(acc)[r], racc)


def test_onehot_sums_only(orc):
    """int32 sums without outputs (y not requested)."""
    N, C, M = 16400, 64, 256
    idx = W.random_indices(N, C, seed=5)
    lut, scale, offset = codes(C, M, 6, 9)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, want_y=False)
    assert y is None
    racc, _ = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)


@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_onehot_layer_output(orc, act):
    """The second launch of a fused call whose table exceeds the single-launch
    kernels (128 codebooks), with the layer output in its epilogue (the
    softmax as a pass after it)."""
    N, D, C, M = 16500, 256, 128, 256
    rng = np.random.default_rng(31)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = codes(C, M, 32, 2)
    bias = rng.standard_normal(M).astype(np.float32)
    y = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                            col_bias=dev(bias), act=act))
    r = sample_rows(N, 33, n=1024)
    _, _, ry = orc.matmul(A[r], split, thr, lut, scale, offset)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    ref = orc.sigma(ry, bias, code)
    if act != "softmax":
        assert np.array_equal(y[r].astype(np.float64), ref)
        return
    z = orc.sigma(ry, bias, 1)
    d = z - z.max(axis=1, keepdims=True)
    tol = 1.01 * (np.abs(d) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(y[r].astype(np.float64) - ref) <= tol)


def test_onehot_repeat_and_smaller_call(orc):
    """Two calls in a row into the same outputs, the second over fewer rows:
    each equal to the oracle (nothing carried over between calls)."""
    C, M = 64, 512
    lut, scale, offset = codes(C, M, 41, 3)
    y = torch.full((30000, M), 5.0, dtype=torch.float32, device=DEV)
    for N, seed in ((30000, 42), (16385, 43)):
        idx = W.random_indices(N, C, seed=seed)
        mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), y_out=y[:N])
        r = sample_rows(N, seed)
        assert np.array_equal(host(y[:N])[r], orc.lut_accumulate(idx[r], lut, scale, offset)[1])
