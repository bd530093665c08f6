"""Different kernels, same bits.

The planner sends the same call to different kernels depending on pointer
alignment, on which outputs are asked for and on the entry point; each pair
below reaches two different kernels (or two instantiations of one) with the
same inputs, and their results must be bit-identical (integer sums exact
everywhere, fp32-table sums in the same fixed order, the same epilogue).
Each case's docstring names the two routes, as a kernel trace of the case
shows them."""
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


def shifted(x, dtype, nbytes):
    """Device copy of x placed `nbytes` past an allocation's start."""
    el = torch.empty((), dtype=dtype).element_size()
    assert nbytes % el == 0
    flat = torch.empty(x.size + nbytes // el, dtype=dtype, device=DEV)
    v = flat[nbytes // el:].view(x.shape)
    v.copy_(torch.from_numpy(np.ascontiguousarray(x)).to(DEV))
    return v


def layer(N, D, C, M, seed, max_shift=1):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=seed + 1, max_shift=max_shift)
    return A, split, thr, lut, scale, offset


def test_gather_fused_vs_general_kernel():
    """conv3x3-shaped layer: a 16-byte-aligned table takes the gather-fused
    kernel, the same table one byte off alignment the general kernel."""
    A, split, thr, lut, scale, offset = layer(5003, 576, 32, 64, seed=11)
    args = (dev(A), dev(split), dev(thr))
    y0, a0, i0 = mdn.matmul(*args, dev(lut), dev(scale), dev(offset), want_acc=True, want_idx=True)
    y1, a1, i1 = mdn.matmul(*args, shifted(lut, torch.int8, 1), dev(scale), dev(offset), want_acc=True,
                            want_idx=True)
    assert np.array_equal(host(i0), host(i1))
    assert np.array_equal(host(a0), host(a1))
    assert np.array_equal(host(y0), host(y1))


def test_row_streaming_vs_encode_then_accumulate():
    """dense_hidden-shaped layer (98304 + 9 rows, 128 columns): the fused call
    runs the row-streaming kernel; encode followed by the accumulate-only
    entry point runs the encoder and the column-tiled accumulate."""
    A, split, thr, lut, scale, offset = layer(98304 + 9, 64, 64, 128, seed=12)
    Ad, sd, td, ld, scd, od = dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset)
    y0, _, i0 = mdn.matmul(Ad, sd, td, ld, scd, od, want_idx=True)
    idx = mdn.encode(Ad, sd, td)
    _, y1 = mdn.lut_accumulate(idx, ld, scd, od)
    assert np.array_equal(host(i0), host(idx))
    assert np.array_equal(host(y0), host(y1))


def test_one_row_per_lane_vs_row_uniform_int8():
    """Accumulate-only, int8 table of 256 codebooks (past the one-hot
    product's 128) and 512 columns, one shared block exponent (so the 16-bit
    field sums fit): outputs alone take the one-row-per-lane kernel, outputs
    plus int32 sums the row-uniform kernel."""
    N, C, M = 20485, 256, 512
    idx = dev(W.random_indices(N, C, seed=13))
    lut, scale, offset = W.random_codes(C, M, seed=14, max_shift=0)
    _, y0 = mdn.lut_accumulate(idx, dev(lut), dev(scale), dev(offset))
    a1, y1 = mdn.lut_accumulate(idx, dev(lut), dev(scale), dev(offset), want_acc=True)
    assert np.array_equal(host(y0), host(y1))


def test_one_row_per_lane_vs_tiled_fp32():
    """fp32 table of 32 codebooks and 1000 columns: 16-byte-aligned takes the
    one-row-per-lane kernel, four bytes off alignment a column-tiled kernel;
    both sum codebooks in ascending order from +0."""
    N, C, M = 20485, 32, 1000
    idx = dev(W.random_indices(N, C, seed=15))
    tab = W.random_fp32_table(C, M, seed=16)
    y0 = mdn.lut_accumulate_f32(idx, dev(tab))
    y1 = mdn.lut_accumulate_f32(idx, shifted(tab, torch.float32, 4))
    assert np.array_equal(host(y0), host(y1))


def test_gather_fused_encode_vs_indices():
    """conv3x3-shaped layer: the fused call (gather-fused kernel, encoding)
    against the accumulate-only call on the indices it returned (the same
    kernel loading index bytes in place of the encode)."""
    A, split, thr, lut, scale, offset = layer(5003, 576, 32, 64, seed=19)
    ld, scd, od = dev(lut), dev(scale), dev(offset)
    y0, a0, idx = mdn.matmul(dev(A), dev(split), dev(thr), ld, scd, od, want_acc=True, want_idx=True)
    a1, y1 = mdn.lut_accumulate(idx, ld, scd, od, want_acc=True)
    assert np.array_equal(host(a0), host(a1))
    assert np.array_equal(host(y0), host(y1))


def test_one_hot_product_vs_row_uniform():
    """Accumulate-only, int8 table of 64 codebooks and 512 columns, outputs
    and int32 sums: 8-byte aligned index rows take the one-hot product on the
    matrix cores, index rows 4 bytes off that alignment the row-uniform
    kernel."""
    N, C, M = 20485, 64, 512
    idx = W.random_indices(N, C, seed=20)
    lut, scale, offset = W.random_codes(C, M, seed=21, max_shift=9)
    ld, scd, od = dev(lut), dev(scale), dev(offset)
    a0, y0 = mdn.lut_accumulate(dev(idx), ld, scd, od, want_acc=True)
    a1, y1 = mdn.lut_accumulate(shifted(idx, torch.uint8, 4), ld, scd, od, want_acc=True)
    assert np.array_equal(host(a0), host(a1))
    assert np.array_equal(host(y0), host(y1))
