"""Parity of the rounded 8-bit summation accumulate (reading R20) and of the
shared-exponent table build with the oracle.  Integer work: acc bit-exact,
and y bit-exact since both sides apply the same single-rounding dequant to the
same acc.  Also checks the documented error bound against the exact sum."""
import math

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


def run_avg(orc, idx, lut, scale, offset):
    acc, y = mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, validate=True)
    racc, ry = orc.lut_accumulate_avg(idx, lut, scale, offset)
    acc, y = host(acc), host(y)
    assert np.array_equal(acc, racc), f"{int((acc != racc).sum())} accumulators differ"
    assert np.array_equal(y, ry)
    return acc


CASES = [(1, 16), (2, 10), (3, 64), (5, 17), (8, 256), (9, 300), (16, 128), (33, 1024), (64, 512),
         (100, 64), (128, 4096), (120, 33),
         (40, 3), (128, 3), (128, 16)]   # narrow outputs: the column tile stays wide enough for a batch


@pytest.mark.parametrize("C,M", CASES)
def test_avg_random_codes(orc, C, M):
    """Tree depths 0..9, padded and unpadded codebook counts, one and several
    column tiles, M with and without 16-column units."""
    N = 777
    idx = W.random_indices(N, C, seed=C * 3 + M)
    lut, scale, offset = W.random_codes(C, M, seed=C + 7 * M, max_shift=0)
    acc = run_avg(orc, idx, lut, scale, offset)
    exact, _ = orc.lut_accumulate(idx, lut, scale, offset)
    P = 1 << max(0, math.ceil(math.log2(C)))
    err = acc.astype(np.int64) - exact.astype(np.int64)
    assert err.min() >= 0 and err.max() <= P * int(math.log2(P)) // 2


def test_avg_rejects_many_codebooks(orc):
    """C > 128: the column slice and an index batch do not fit in LDS."""
    idx = W.random_indices(10, 256, seed=1)
    lut, scale, offset = W.random_codes(256, 16, seed=2, max_shift=0)
    with pytest.raises(mdn.MaddnessError):
        mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset))


@pytest.mark.parametrize("N", [1, 63, 64, 65, 129, 1000])
def test_avg_ragged_rows(orc, N):
    idx = W.random_indices(N, 32, seed=N)
    lut, scale, offset = W.random_codes(32, 64, seed=N + 1, max_shift=0)
    run_avg(orc, idx, lut, scale, offset)


def test_avg_extreme_codes(orc):
    """Codes at +-127 (bytes 255 and 1): no wrap in the byte averages."""
    C, M, N = 64, 256, 300
    idx = W.random_indices(N, C, seed=5)
    lut, scale, offset = W.random_codes(C, M, seed=6, max_shift=0, extreme=True)
    run_avg(orc, idx, lut, scale, offset)


@pytest.mark.parametrize("name", ["conv3x3_im2col", "dense_hidden", "wide_layer"])
def test_avg_workloads_with_shared_tables(orc, name):
    """The shared-exponent table built on the GPU equals the oracle's, and the
    averaging accumulate over the workload's own indices matches."""
    N = {"conv3x3_im2col": 2000, "dense_hidden": 1500, "wide_layer": 400}[name]
    p = W.make(name, N=N)
    lut, scale, offset = mdn.build_lut_shared(dev(p.P), dev(p.B))
    rl, rs, ro = orc.build_shared_lut(p.P, p.B)
    assert np.array_equal(host(lut), rl) and np.array_equal(host(scale), rs) and np.array_equal(host(offset), ro)
    idx = orc.encode(p.A, p.split, p.thr)
    run_avg(orc, idx, rl, rs, ro)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["conv3x3_im2col", "dense_hidden", "wide_layer"])
def test_avg_full_size_sampled(orc, name):
    """Full-size workload in the launch configuration the benchmark's context
    times (GPU encoder, GPU shared-exponent table, averaging accumulate over
    every row); the oracle encodes and sums every row of the conv layer and
    a sample of about 6000 rows of the larger ones itself."""
    from test_gpu_parity import parity_rows
    p = W.make(name)
    rows = parity_rows(name, p.N)
    idx = mdn.encode(dev(p.A), dev(p.split), dev(p.thr))
    lut, scale, offset = mdn.build_lut_shared(dev(p.P), dev(p.B))
    rl, rs, ro = orc.build_shared_lut(p.P, p.B)
    assert np.array_equal(host(lut), rl) and np.array_equal(host(scale), rs)
    acc, y = mdn.lut_accumulate_avg(idx, lut, scale, offset, want_acc=True)
    racc, ry = orc.lut_accumulate_avg(orc.encode(p.A[rows], p.split, p.thr), rl, rs, ro)
    r = torch.from_numpy(rows).to(DEV)
    assert np.array_equal(host(acc[r]), racc)
    assert np.array_equal(host(y[r]), ry)
    del acc, y, idx
    torch.cuda.empty_cache()
