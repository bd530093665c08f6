"""Parity of the row-uniform accumulate with the oracle.

The dispatcher takes that kernel for int8 tables at least 512 columns wide
(C % 4 == 0, aligned buffers) once the 256-row work items fill a quarter of
the CUs, so every case here has N >= 16384 / (column tiles of 512): smaller
calls take the column-tiled kernel that the other parity tests cover.  Both
of its summation modes are exercised: 16-bit fields of (q + 128) << sh when
255 * sum_c 2^sh <= 65535 (including that bound exactly, with every code at
+127 or -128), and int32 sums with shifts otherwise.  Bar as in the other
parity tests: int32 sums and fp32 outputs bit-exact; softmax within the
bound of the sigma tests."""
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


def rows_for(M):
    """Rows that reach the row-uniform kernel: 64 work items of 256 rows x
    512 columns, plus a ragged tail."""
    tiles = -(-M // 512)
    return -(-64 // tiles) * 256 + 77


def check_accumulate(orc, idx, lut, scale, offset):
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, validate=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


# (C, M, max_shift): sum_c 2^sh <= 257 takes the 16-bit fields, else int32 sums
ROW_CASES = [(64, 512, 0), (64, 512, 2), (64, 512, 5), (32, 1008, 3), (4, 512, 0), (12, 768, 1),
             (128, 4096, 0), (256, 512, 0), (260, 512, 0), (512, 512, 0), (8, 2048, 7)]


@pytest.mark.parametrize("C,M,max_shift", ROW_CASES)
def test_row_accumulate_random(orc, C, M, max_shift):
    N = rows_for(M)
    idx = W.random_indices(N, C, seed=C * 31 + M)
    lut, scale, offset = W.random_codes(C, M, seed=C + 7 * M + max_shift, max_shift=max_shift)
    check_accumulate(orc, idx, lut, scale, offset)


@pytest.mark.parametrize("code", [127, -128, -127])
@pytest.mark.parametrize("shifts", [(7, 6, 6, 0), (7, 6, 6, 1)])
def test_row_accumulate_field_bound(orc, code, shifts):
    """sum 2^sh = 257: every 16-bit field reaches 255 * 257 = 65535 (codes
    +127) or 0 (codes -128); 258 is the first sum that takes int32 sums."""
    C, M = 4, 512
    N = rows_for(M)
    idx = W.random_indices(N, C, seed=sum(shifts) + code + 200)
    lut = np.full((C, 16, M), code, dtype=np.int8)
    lut[:, 3, ::7] = -code if code != -128 else 127   # a few other codes
    scale = np.ldexp(np.float32(1.0), np.array(shifts, dtype=np.int32) - 9).astype(np.float32)
    offset = np.random.default_rng(3).standard_normal(C).astype(np.float32)
    check_accumulate(orc, idx, lut, scale, offset)


def test_row_accumulate_single_outputs(orc):
    C, M = 64, 512
    N = rows_for(M)
    idx = W.random_indices(N, C, seed=11)
    lut, scale, offset = W.random_codes(C, M, seed=12, max_shift=1)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, want_y=False)
    assert y is None and np.array_equal(host(acc), racc)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=False, want_y=True)
    assert acc is None and np.array_equal(host(y), ry)


@pytest.mark.parametrize("name,N", [("dense_hidden", 16411), ("wide_layer", 2100)])
def test_row_matmul_workloads(orc, name, N):
    """Encode, then the row-uniform accumulate (tables larger than LDS)."""
    p = W.make(name, N=N)
    lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    y, acc, idx = mdn.matmul(dev(p.A), dev(p.split), dev(p.thr), lut, scale, offset, want_acc=True,
                             want_idx=True)
    ridx, racc, ry = orc.matmul(p.A, p.split, p.thr, rl, rs, ro)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


@pytest.mark.parametrize("M,max_shift", [(512, 2), (1024, 2), (512, 6)])
@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_row_layer_output(orc, M, max_shift, act):
    """matmul_act with a table larger than LDS: encode, then sigma in the
    row-uniform kernel's epilogue (one column tile: M = 512), or bias there
    and the row softmax as a second pass (M = 1024); max_shift 6 takes the
    int32 sums."""
    C, D = 64, 96
    N = rows_for(M)
    rng = np.random.default_rng(M + len(act))
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=M + 1, max_shift=max_shift)
    bias = rng.standard_normal(M).astype(np.float32)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    y = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                            col_bias=dev(bias), act=act))
    _, _, yref = orc.matmul(A, split, thr, lut, scale, offset)
    ref = orc.sigma(yref, bias, code)
    if act != "softmax":
        assert np.array_equal(y.astype(np.float64), ref)
        return
    z = orc.sigma(yref, bias, 1)
    tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(y.astype(np.float64) - ref) <= tol)


@pytest.mark.parametrize("M,act,bias_off", [(8192, "relu", 0), (1024, "bias", 1)])
def test_row_layer_output_bias_placement(orc, M, act, bias_off):
    """Column biases staged in LDS once per workgroup (M = 1024, with the bias
    row 4 bytes off 16-byte alignment), or read from memory in every work
    item's epilogue when the row does not fit next to the table tiles (M =
    8192: 32 KB)."""
    C, D = 8, 64
    N = rows_for(M)
    rng = np.random.default_rng(M + bias_off)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=M + 3, max_shift=2)
    bias_all = rng.standard_normal(M + bias_off).astype(np.float32)
    bias = bias_all[bias_off:]
    bias_dev = dev(bias_all)[bias_off:]
    assert (bias_dev.data_ptr() % 16 == 0) == (bias_off == 0)
    code = {"bias": 1, "relu": 2}[act]
    y = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                            col_bias=bias_dev, act=act))
    _, _, yref = orc.matmul(A, split, thr, lut, scale, offset)
    assert np.array_equal(y.astype(np.float64), orc.sigma(yref, bias, code))


# ---------------------------------- int8 tables, one output row per lane (y)
# Calls that want y only (no int32 sums) take that kernel when C % 16 == 0
# and C >= 32 within the row-uniform kernel's shapes; it does nothing when
# the 16-bit field sums do not fit, and the row-uniform kernel launched after
# it (which otherwise does nothing) then sums in int32.  Each workgroup keeps
# one 128-column tile and streams row blocks; from 4 row blocks per workgroup
# on, its wavefronts start at different codebook tiles.  Below 128 codebooks
# the outputs go through a quad transpose before the stores.  Cases: both
# store forms with and without the phases, C = 32 (two tiles per cycle), a
# ragged last row block and last column tile, the field bound exactly, sums
# that need int32, and the layer outputs.
def check_y(orc, idx, lut, scale, offset, rows=None):
    _, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=False, validate=True)
    N = idx.shape[0]
    if rows is None:
        rows = np.unique(np.r_[0:300, N - 300:N, np.random.default_rng(N).integers(0, N, size=600)])
    got = y[torch.from_numpy(rows).to(DEV)]
    _, ry = orc.lut_accumulate(idx[rows], lut, scale, offset)
    assert np.array_equal(host(got), ry)


# (C, M, N, max_shift): phases need N >= 4 row blocks of 1024 x the workgroups per column tile
LANE_I8_CASES = [(64, 512, 262144 + 333, 1), (64, 512, 20485, 2), (128, 4096, 32768 + 1500, 1), (256, 1024, 131072 + 7, 0),
                 (32, 1008, 131072 + 65, 3), (48, 2048, 40961, 1)]


@pytest.mark.parametrize("C,M,N,max_shift", LANE_I8_CASES)
def test_lane_accumulate_i8(orc, C, M, N, max_shift):
    idx = W.random_indices(N, C, seed=C + M + N)
    lut, scale, offset = W.random_codes(C, M, seed=3 * C + M, max_shift=max_shift)
    check_y(orc, idx, lut, scale, offset)


@pytest.mark.parametrize("code", [127, -128])
@pytest.mark.parametrize("shifts", [(7, 6, 1, 1, 1), (7, 6, 1, 1, 2)])
def test_lane_accumulate_i8_field_bound(orc, code, shifts):
    """sum 2^sh = 257 exactly (every field at 65535 or 0), and 258, the
    first sum that takes the row-uniform kernel's int32 sums."""
    C, M, N = 64, 512, 262144 + 5
    sh = np.array(list(shifts) + [0] * (C - len(shifts)), dtype=np.int32)
    idx = W.random_indices(N, C, seed=int(sh.sum()) + code + 300)
    lut = np.full((C, 16, M), code, dtype=np.int8)
    lut[:, 5, ::3] = -code if code != -128 else 127
    scale = np.ldexp(np.float32(1.0), sh - 9).astype(np.float32)
    offset = np.random.default_rng(5).standard_normal(C).astype(np.float32)
    check_y(orc, idx, lut, scale, offset)


@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_lane_layer_output_i8(orc, act):
    """Bias and ReLU in the epilogue (the workgroup's 128 column biases in
    LDS, M = 1008: a ragged last column tile), softmax as a second pass."""
    C, D, M, N = 64, 72, 1008, 65536 + 123
    rng = np.random.default_rng(len(act) + 21)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=M + 3, max_shift=1)
    bias = rng.standard_normal(M).astype(np.float32)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    y = mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset), col_bias=dev(bias), act=act)
    rows = np.unique(np.r_[0:200, N - 200:N, rng.integers(0, N, size=500)])
    got = host(y[torch.from_numpy(rows).to(DEV)]).astype(np.float64)
    _, _, yref = orc.matmul(A[rows], split, thr, lut, scale, offset)
    ref = orc.sigma(yref, bias, code)
    if act != "softmax":
        assert np.array_equal(got, ref)
        return
    z = orc.sigma(yref, bias, 1)
    tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(got - ref) <= tol)


# ------------------------------------------------------------- fp32 tables
def rows_for_f32(M):
    """Rows that reach the fp32 row-uniform kernel: 64 work items of 256 rows
    x 256 columns, plus a ragged tail."""
    tiles = -(-M // 256)
    return -(-64 // tiles) * 256 + 77


@pytest.mark.parametrize("C,M", [(256, 1024), (4, 256), (8, 260), (64, 1000), (12, 512), (100, 4096)])
def test_row_accumulate_f32(orc, C, M):
    """Ordered fp32 sums, codebooks ascending from +0.0f: bit-identical."""
    N = rows_for_f32(M)
    idx = W.random_indices(N, C, seed=C * 13 + M)
    tab = W.random_fp32_table(C, M, seed=C + 5 * M)
    y = host(mdn.lut_accumulate_f32(dev(idx), dev(tab), validate=True))
    assert np.array_equal(y, orc.lut_accumulate_f32(idx, tab))


def test_row_matmul_f32_workload(orc):
    p = W.make("encode_heavy_f32", N=rows_for_f32(1024))
    tab = mdn.build_lut_f32(dev(p.P), dev(p.B))
    rtab = orc.build_lut_f32(p.P, p.B)
    assert np.array_equal(host(tab), rtab)
    y, idx = mdn.matmul_f32(dev(p.A), dev(p.split), dev(p.thr), tab, want_idx=True)
    ridx, ry = orc.matmul_f32(p.A, p.split, p.thr, rtab)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(y), ry)


@pytest.mark.parametrize("M", [256, 512])
@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_row_layer_output_f32(orc, M, act):
    """sigma in the fp32 kernel's epilogue (one column tile: M = 256), or bias
    there and the row softmax as a second pass (M = 512)."""
    C, D = 32, 80
    N = rows_for_f32(M)
    rng = np.random.default_rng(3 * M + len(act))
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    tab = W.random_fp32_table(C, M, seed=M + 7)
    bias = rng.standard_normal(M).astype(np.float32)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    y = host(mdn.matmul_act_f32(dev(A), dev(split), dev(thr), dev(tab), col_bias=dev(bias), act=act))
    _, yref = orc.matmul_f32(A, split, thr, tab)
    ref = orc.sigma(yref, bias, code)
    if act != "softmax":
        assert np.array_equal(y.astype(np.float64), ref)
        return
    z = orc.sigma(yref, bias, 1)
    tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(y.astype(np.float64) - ref) <= tol)


# --------------------------------------- fp32 tables, one output row per lane
# The dispatcher takes that kernel for fp32 tables with C % 16 == 0 and at
# least 256 columns (work items of 1024 rows x 64 columns, 16 codebooks per
# staged tile), unless the row softmax fits the row-uniform kernel's epilogue
# (M = 256).  Cases: several work items per workgroup (more items than CUs),
# a grid that is not a multiple of 8, one codebook tile (C = 16), a ragged
# last column tile (M % 64 != 0) with the layer outputs, and a last row block
# of a few rows.
LANE_CASES = [(32, 1000, 20485), (16, 384, 10241), (256, 1024, 16389), (48, 4100, 2051)]


@pytest.mark.parametrize("C,M,N", LANE_CASES)
def test_lane_accumulate_f32(orc, C, M, N):
    idx = W.random_indices(N, C, seed=C + M + N)
    tab = W.random_fp32_table(C, M, seed=7 * C + M)
    y = host(mdn.lut_accumulate_f32(dev(idx), dev(tab), validate=True))
    rows = np.unique(np.r_[0:300, N - 300:N, np.random.default_rng(N).integers(0, N, size=700)])
    assert np.array_equal(y[rows], orc.lut_accumulate_f32(idx[rows], tab))


@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
def test_lane_layer_output_f32(orc, act):
    """Bias and ReLU in the epilogue (bias row zero-padded in LDS to whole
    column tiles: M = 1000), softmax as a second pass."""
    C, D, M, N = 32, 72, 1000, 20485
    rng = np.random.default_rng(len(act) + 11)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    tab = W.random_fp32_table(C, M, seed=M + 9)
    bias = rng.standard_normal(M).astype(np.float32)
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    y = host(mdn.matmul_act_f32(dev(A), dev(split), dev(thr), dev(tab), col_bias=dev(bias), act=act))
    rows = np.unique(np.r_[0:200, N - 200:N, rng.integers(0, N, size=500)])
    _, yref = orc.matmul_f32(A[rows], split, thr, tab)
    ref = orc.sigma(yref, bias, code)
    got = y[rows].astype(np.float64)
    if act != "softmax":
        assert np.array_equal(got, ref)
        return
    z = orc.sigma(yref, bias, 1)
    tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(got - ref) <= tol)


# ------------------------------------------- rounded 8-bit summation (R20)
# The averaging accumulate at the row counts of the cases above (its kernel
# keeps one column slice of the table per workgroup and streams row batches):
# many batches per workgroup, ragged last batch.
def rows_for_avg(M):
    tiles = -(-M // 512)
    return -(-64 // tiles) * 128 + 77


# (C, M): P < 8; one subtree of 8; padding codebooks in the last subtree
# (C 12); whole padding subtrees (C 36: P 64); C > 64; column tails
AVG_ROW_CASES = [(4, 512), (8, 512), (12, 768), (36, 1024), (64, 512), (100, 512), (128, 4096), (60, 1008)]


@pytest.mark.parametrize("C,M", AVG_ROW_CASES)
def test_row_accumulate_avg(orc, C, M):
    N = rows_for_avg(M)
    idx = W.random_indices(N, C, seed=C * 17 + M)
    lut, scale, offset = W.random_codes(C, M, seed=C + 3 * M, max_shift=0)
    acc, y = mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True)
    racc, ry = orc.lut_accumulate_avg(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


def test_row_accumulate_avg_extreme_and_single_outputs(orc):
    """Codes at +-127 and -128, then acc only and y only."""
    C, M = 64, 512
    N = rows_for_avg(M)
    idx = W.random_indices(N, C, seed=5)
    lut, scale, offset = W.random_codes(C, M, seed=6, max_shift=0, extreme=True)
    lut[::3, 5, ::11] = -128
    racc, ry = orc.lut_accumulate_avg(idx, lut, scale, offset)
    acc, y = mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, want_y=False)
    assert y is None and np.array_equal(host(acc), racc)
    acc, y = mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=False, want_y=True)
    assert acc is None and np.array_equal(host(y), ry)
