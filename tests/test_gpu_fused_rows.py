"""Parity of the row-streaming fused kernel with the oracle.

The fused entry points take that kernel for int8 tables of 64 codebooks with
16 <= M <= 512 columns (M % 16 == 0), too large for the gather-fused kernel,
and calls of at least 98304 rows: the dense hidden layer's shape.  It encodes
and sums in one launch when the 16-bit field sums fit (255 sum_c 2^sh <=
65535); otherwise it only encodes (into idx_out, or into the first bytes of
each output row) and the row-uniform accumulate that always follows it sums
with 32-bit accumulators.  Both branches are covered here, with row strides,
ragged row counts, column counts below one tile, the field bound exactly,
every layer output, and the optional index and int32 outputs.  Given an
8-byte aligned index array, calls of at least 128 columns whose table the
one-hot product takes run faster as encode + that product (the index-size
query asks for the array there); so the kernel itself is reached here through
the allocation-free entry point without an index array, or with one at a
4-byte offset, and the routed call is checked beside it.  Bar: indices, int32
sums and fp32 outputs bit-exact; softmax within the bound of the sigma
tests."""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
N0 = 98304          # fewest rows that take the kernel


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def layer(N, D, M, seed, pad=0, max_shift=0, shifts=None, code=None):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, D + pad), dtype=np.float32)
    split = rng.integers(0, D, size=(64, 4)).astype(np.int32)
    thr = rng.standard_normal((64, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(64, M, seed=seed + 1, max_shift=max_shift)
    if shifts is not None:
        scale = np.ldexp(np.float32(1.0), np.asarray(shifts, np.int32) - 20).astype(np.float32)
    if code is not None:
        lut = np.full((64, 16, M), code, np.int8)
    return A, split, thr, lut, scale, offset


def rows_sample(N, seed=0):
    rng = np.random.default_rng(seed)
    return np.unique(np.r_[0:1500, N - 1500:N, rng.integers(0, N, size=3000)])


def offset_index_array(N):
    """An [N, 64] index array 4 bytes past an 8-byte boundary: the one-hot
    product does not take it, so a fused call keeps the row-streaming kernel."""
    flat = torch.empty(N * 64 + 4, dtype=torch.uint8, device=DEV)
    return flat[4:].view(N, 64)


def run_and_check(orc, A, D, split, thr, lut, scale, offset, rows=None, with_idx=True, with_acc=True):
    """Fused call on A[:, :D] (row stride A.shape[1]) through the row-streaming
    kernel, and as the library routes it by default; both against the oracle."""
    N, M = A.shape[0], lut.shape[2]
    Ad = dev(A)[:, :D]
    args = (Ad, dev(split), dev(thr), dev(lut), dev(scale), dev(offset))
    assert mdn.matmul_index_bytes(Ad, 64, M) == (N * 64 if M >= 128 else 0)
    y = torch.empty((N, M), dtype=torch.float32, device=DEV)
    acc = torch.empty((N, M), dtype=torch.int32, device=DEV) if with_acc else None
    idx = offset_index_array(N) if with_idx else None
    mdn.matmul_noalloc(*args, y_out=y, acc_out=acc, idx_out=idx)
    rows = np.arange(N) if rows is None else rows
    ridx, racc, ry = orc.matmul(A[rows, :D], split, thr, lut, scale, offset)
    r = torch.from_numpy(rows).to(DEV)
    routed = mdn.matmul(*args, want_acc=with_acc, want_idx=with_idx, validate=True)
    for yy, aa, ii in ((y, acc, idx), routed):
        if with_idx:
            assert np.array_equal(host(ii[r]), ridx)
            assert int(ii.max()) < 16
        if with_acc:
            assert np.array_equal(host(aa[r]), racc)
        assert np.array_equal(host(yy[r]), ry)
    return y


@pytest.mark.parametrize("extra", [0, 1, 1234, 11])
def test_dense_hidden_layer(orc, extra):
    """The dense hidden layer (D 512, C 64, M 512, its own trees and table)
    at N0 + extra rows, every row compared."""
    p = W.make("dense_hidden", N=N0 + extra)
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    run_and_check(orc, p.A, p.D, p.split, p.thr, rl, rs, ro, with_idx=(extra != 11), with_acc=(extra != 1))


@pytest.mark.parametrize("M,max_shift,pad", [(512, 0, 0), (512, 2, 3), (256, 1, 0), (128, 0, 1), (496, 2, 0),
                                             (80, 0, 0)])
def test_random_layers(orc, M, max_shift, pad):
    """Random trees over 200 columns (row stride 200 + pad), random codes with
    per-codebook shifts up to max_shift (16-bit fields), M below and at one
    tile; sampled rows."""
    N = N0 + 3 * M + 5
    A, split, thr, lut, scale, offset = layer(N, 200, M, seed=M + max_shift + pad, pad=pad, max_shift=max_shift)
    run_and_check(orc, A, 200, split, thr, lut, scale, offset, rows=rows_sample(N, M))


@pytest.mark.parametrize("code", [127, -128])
def test_field_bound_exactly(orc, code):
    """sum_c 2^sh = 257 (shifts 7, 6, 1, 1, 1, then 0): the largest table the
    16-bit fields take, with every code at an extreme."""
    shifts = [7, 6, 1, 1, 1] + [0] * 59
    assert sum(2 ** s for s in shifts) == 257
    A, split, thr, lut, scale, offset = layer(N0 + 50, 96, 512, seed=5, shifts=shifts, code=code)
    run_and_check(orc, A, 96, split, thr, lut, scale, offset, rows=rows_sample(N0 + 50, 1))


@pytest.mark.parametrize("with_idx", [True, False])
def test_wide_exponents_take_the_32bit_sums(orc, with_idx):
    """sum_c 2^sh > 257: the kernel only encodes (into idx_out, or into the
    output rows themselves) and the row-uniform accumulate sums in int32."""
    shifts = [9, 3] + [0] * 62
    A, split, thr, lut, scale, offset = layer(N0 + 333, 128, 512, seed=9, shifts=shifts)
    lut = np.random.default_rng(3).integers(-128, 128, size=lut.shape).astype(np.int8)
    run_and_check(orc, A, 128, split, thr, lut, scale, offset, rows=rows_sample(N0 + 333, 2), with_idx=with_idx)


@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_layer_outputs(orc, act):
    """The layer output fused in the retire step: bias and ReLU bit-exact,
    the row softmax within the bound of the sigma tests."""
    p = W.make("dense_hidden", N=N0 + 77)
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    bias = np.random.default_rng(4).standard_normal(512).astype(np.float32)
    args = (dev(p.A), dev(p.split), dev(p.thr), dev(rl), dev(rs), dev(ro))
    assert mdn.matmul_index_bytes(args[0], 64, 512, act=act) == (0 if act == "softmax" else p.N * 64)
    rows = rows_sample(p.N, 3)
    _, _, yr = orc.matmul(p.A[rows], p.split, p.thr, rl, rs, ro)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    ref = orc.sigma(yr, bias, code)
    # the row-streaming kernel (index array off 8-byte alignment), then the
    # routed call (encode + one-hot product; for the softmax, the row-streaming
    # kernel again)
    for idx in (offset_index_array(p.N), None):
        y = host(mdn.matmul_act(*args, col_bias=dev(bias), act=act, idx_out=idx))
        got = y[rows].astype(np.float64)
        if act != "softmax":
            assert np.array_equal(got, ref)
        else:
            z = orc.sigma(yr, bias, 1)
            tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + 512 + 5) * 2.0 ** -24 * ref + 2.0 ** -120
            assert np.all(np.abs(got - ref) <= tol)
