"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bar: indices, int32 accumulators and int8 tables bit-exact; fp32 outputs
within 1e-6 relative error, and in fact bit-identical since both sides
compute the same single-rounding formula (int8 tables) or the same ordered
fp32 sum (fp32 tables).  Every input comes from the seeded generator in
paper_2207_05808_amd.workloads; no expected value comes from the GPU.
"""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FLT_MIN = np.float32(np.finfo(np.float32).tiny)


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_y(y, ref):
    """fp32 outputs: relative error <= 1e-6 elementwise, and identical."""
    assert y.shape == ref.shape and y.dtype == np.float32
    d = np.abs(y.astype(np.float64) - ref.astype(np.float64))
    rel = d / np.maximum(np.abs(ref.astype(np.float64)), FLT_MIN)
    assert float(rel.max(initial=0.0)) <= 1e-6, f"max rel err {rel.max()}"
    assert np.array_equal(y, ref), f"{int((y != ref).sum())} outputs differ in the last bits"


def max_shift_for(C):
    """Largest shift s (at most 12) with 128 C 2^s <= 2^31: any codes of C
    codebooks shifted by up to s keep the int32 sum exact."""
    s = 0
    while 128.0 * C * 2.0 ** (s + 1) <= 2.0 ** 31 and s < 12:
        s += 1
    return s


# ---------------------------------------------------------------- encode
@pytest.mark.parametrize("name", list(W.SPECS))
def test_encode_workloads(orc, name):
    N = 1024 if name == "classifier_tiny" else 3001
    p = W.make(name, N=N)
    idx = host(mdn.encode(dev(p.A), dev(p.split), dev(p.thr), validate=True))
    ref = orc.encode(p.A, p.split, p.thr)
    assert np.array_equal(idx, ref)


@pytest.mark.parametrize("N", [1, 2, 3, 63, 64, 65, 255, 257, 1000])
def test_encode_ragged_rows(orc, N):
    p = W.make("conv3x3_im2col", N=N)
    idx = host(mdn.encode(dev(p.A), dev(p.split), dev(p.thr)))
    assert np.array_equal(idx, orc.encode(p.A, p.split, p.thr))


@pytest.mark.parametrize("D,C,pad", [(577, 7, 0), (576, 32, 3), (64, 4, 5), (33, 1, 0), (16, 16, 0),
                                     (1024, 128, 0), (12, 200, 4), (2050, 3, 2)])
def test_encode_shapes_and_strides(orc, D, C, pad):
    rng = np.random.default_rng(D * 1000 + C)
    N = 777
    full = rng.standard_normal((N, D + pad), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    At = dev(full)[:, :D]   # row stride D + pad
    idx = host(mdn.encode(At, dev(split), dev(thr)))
    assert np.array_equal(idx, orc.encode(full[:, :D], split, thr))


def test_encode_special_values(orc):
    rng = np.random.default_rng(5)
    N, D, C = 500, 64, 8
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    thr[0, 0] = 0.0
    thr[1, :] = -0.0
    A = rng.standard_normal((N, D), dtype=np.float32)
    # exact ties with thresholds, signed zeros, infinities and NaNs
    for n in range(0, N, 3):
        c = n % C
        A[n, split[c, 0]] = thr[c, 0]
    A[1::7, :] = 0.0
    A[2::7, :] = -0.0
    A[3::11, ::3] = np.inf
    A[4::11, ::5] = -np.inf
    A[5::13, ::2] = np.nan
    idx = host(mdn.encode(dev(A), dev(split), dev(thr)))
    assert np.array_equal(idx, orc.encode(A, split, thr))


# ------------------------------------------------------- lookup-accumulate
ACC_CASES = [(1, 1), (3, 10), (4, 17), (32, 64), (5, 1000), (33, 77), (64, 512), (128, 300),
             (16, 4096), (256, 8), (512, 20)]


@pytest.mark.parametrize("C,M", ACC_CASES)
def test_lut_accumulate_random(orc, C, M):
    N = 1537
    idx = W.random_indices(N, C, seed=C * 7 + M)
    lut, scale, offset = W.random_codes(C, M, seed=C + 13 * M, max_shift=max_shift_for(C))
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True,
                                validate=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)
    assert_y(host(y), ry)


@pytest.mark.parametrize("C,shift", [(4, 0), (4, 6), (4, 7), (32, 12), (64, 9), (128, 0)])
def test_lut_accumulate_extreme_codes(orc, C, shift):
    """All codes +-127 with the largest shifts: the accumulator near its bound."""
    N, M = 600, 64
    idx = W.random_indices(N, C, seed=99 + C)
    lut, scale, offset = W.random_codes(C, M, seed=7 + C, max_shift=min(shift, max_shift_for(C)),
                                        extreme=True)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)
    assert_y(host(y), ry)


def test_lut_accumulate_single_outputs(orc):
    C, M, N = 32, 64, 999
    idx = W.random_indices(N, C, seed=1)
    lut, scale, offset = W.random_codes(C, M, seed=2, max_shift=3)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, want_y=False)
    assert y is None and np.array_equal(host(acc), racc)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=False, want_y=True)
    assert acc is None
    assert_y(host(y), ry)


@pytest.mark.parametrize("C,shifts", [(4, (7, 6, 6, 0)), (12, (7, 6, 5, 3, 3, 2, 2, 1, 1, 1, 1, 0))])
@pytest.mark.parametrize("code", [-128, 127])
def test_lut_accumulate_16bit_bound(orc, C, shifts, code):
    """sum_c 2^sh = 257: 127 * 257 fits a 16-bit lane but -128 * 257 does
    not, so these tables must take the 32-bit sums (C = 4: the gather-fused
    kernel with index loads; C = 12: the column-tiled kernel)."""
    N, M = 3000, 64
    rng = np.random.default_rng(C + code + 256)
    idx = rng.integers(0, 16, size=(N, C)).astype(np.uint8)
    lut = np.full((C, 16, M), code, dtype=np.int8)
    lut[:, :, 1] = rng.integers(-128, 128, size=(C, 16)).astype(np.int8)
    scale = np.ldexp(np.float32(1.0), np.array(shifts, dtype=np.int32) - 10).astype(np.float32)
    offset = rng.standard_normal(C).astype(np.float32)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, validate=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


EDGE_SHIFTS = {
    # C = 2: the gather-fused kernel with index loads, 32-bit sums
    2: [23, 0],
    # C = 25: the column-tiled kernel; sum 2^sh = 2^24, so -128 codes sum to -2^31
    25: list(range(23, -1, -1)) + [0],
    # C = 28: the row-uniform kernel's 32-bit sums; sum 2^sh = 2^24 again
    28: list(range(23, 3, -1)) + [2, 1, 1, 1, 1, 1, 0, 0],
}


@pytest.mark.parametrize("C", sorted(EDGE_SHIFTS))
@pytest.mark.parametrize("code", [-128, 127, None])
def test_lut_accumulate_int32_edge(orc, C, code):
    """Tables at the accumulator's precondition, 128 sum_c 2^sh <= 2^31: all
    codes -128 (the sum reaches -2^31 for C = 25 and 28), all 127, or random
    int8 codes; acc and y bit-identical to the oracle in each kernel."""
    sh = np.array(EDGE_SHIFTS[C], np.int64)
    assert 128 * int((2 ** sh).sum()) <= 2 ** 31
    N, M = (16384 + 77, 512) if C == 28 else (3000, 64)
    rng = np.random.default_rng(C * 3 + (0 if code is None else code + 200))
    idx = W.random_indices(N, C, seed=C + 5)
    if code is None:
        lut = rng.integers(-128, 128, size=(C, 16, M)).astype(np.int8)
    else:
        lut = np.full((C, 16, M), code, np.int8)
    scale = np.ldexp(np.float32(1.0), (sh - 30).astype(np.int32)).astype(np.float32)
    offset = rng.standard_normal(C).astype(np.float32)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True, validate=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    if code == -128 and C != 2:
        assert np.all(racc == np.int32(-2 ** 31))
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


def test_validator_rejects_past_int32_edge():
    """Shifts (24, 0) pass 127 sum 2^sh < 2^31 but a -128 code would leave
    int32: the binding's validator rejects them."""
    idx = dev(np.zeros((4, 2), np.uint8))
    lut = dev(np.zeros((2, 16, 8), np.int8))
    scale = dev(np.array([2.0 ** 4, 2.0 ** -20], np.float32))
    with pytest.raises(ValueError):
        mdn.lut_accumulate(idx, lut, scale, dev(np.zeros(2, np.float32)), validate=True)


@pytest.mark.parametrize("C,M", [(1, 1), (3, 10), (32, 64), (64, 512), (256, 1024), (7, 33), (200, 5)])
def test_lut_accumulate_f32_random(orc, C, M):
    N = 1111
    idx = W.random_indices(N, C, seed=C + M)
    lut = W.random_fp32_table(C, M, seed=C * M)
    y = mdn.lut_accumulate_f32(dev(idx), dev(lut), validate=True)
    assert_y(host(y), orc.lut_accumulate_f32(idx, lut))


# ----------------------------------------------------------- table build
@pytest.mark.parametrize("name", list(W.SPECS))
def test_build_lut_matches_oracle(orc, name):
    p = W.make(name, N=1)
    if p.spec.quantized:
        lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
        rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
        assert np.array_equal(host(lut), rl)
        assert np.array_equal(host(scale), rs)
        assert np.array_equal(host(offset), ro)
    else:
        lut = mdn.build_lut_f32(dev(p.P), dev(p.B))
        assert np.array_equal(host(lut), orc.build_lut_f32(p.P, p.B))


# ------------------------------------------------------------ fused path
@pytest.mark.parametrize("name", list(W.SPECS))
def test_matmul_workloads_reduced(orc, name):
    """Fused path on the workload's own layer (table built on each side), reduced N."""
    N = 1024 if name == "classifier_tiny" else 3001
    p = W.make(name, N=N)
    A, split, thr = dev(p.A), dev(p.split), dev(p.thr)
    if p.spec.quantized:
        lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
        y, acc, idx = mdn.matmul(A, split, thr, lut, scale, offset, want_acc=True, want_idx=True,
                                 validate=True)
        rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
        ridx, racc, ry = orc.matmul(p.A, p.split, p.thr, rl, rs, ro)
        assert np.array_equal(host(idx), ridx)
        assert np.array_equal(host(acc), racc)
        assert_y(host(y), ry)
        # without the optional outputs the indices stay on chip
        y2, _, _ = mdn.matmul(A, split, thr, lut, scale, offset)
        assert_y(host(y2), ry)
    else:
        lut = mdn.build_lut_f32(dev(p.P), dev(p.B))
        y, idx = mdn.matmul_f32(A, split, thr, lut, want_idx=True)
        ridx, ry = orc.matmul_f32(p.A, p.split, p.thr, orc.build_lut_f32(p.P, p.B))
        assert np.array_equal(host(idx), ridx)
        assert_y(host(y), ry)
        y2, _ = mdn.matmul_f32(A, split, thr, lut)
        assert_y(host(y2), ry)


@pytest.mark.parametrize("N,D,C,M", [(1, 64, 4, 10), (65, 576, 32, 64), (1000, 100, 10, 10),
                                     (513, 512, 64, 512), (300, 1024, 128, 4096), (77, 36, 3, 129),
                                     (2049, 256, 256, 20)])
def test_matmul_random_codes(orc, N, D, C, M):
    rng = np.random.default_rng(N + D + C + M)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=N * 3 + M, max_shift=max_shift_for(C))
    y, acc, idx = mdn.matmul(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                             want_acc=True, want_idx=True)
    ridx, racc, ry = orc.matmul(A, split, thr, lut, scale, offset)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(acc), racc)
    assert_y(host(y), ry)
    lut32 = W.random_fp32_table(C, M, seed=M)
    y32, idx32 = mdn.matmul_f32(dev(A), dev(split), dev(thr), dev(lut32), want_idx=True)
    assert np.array_equal(host(idx32), ridx)
    assert_y(host(y32), orc.lut_accumulate_f32(ridx, lut32))


def test_outputs_stay_in_bounds_and_repeat(orc):
    """Sentinel guard after every output; two runs are bit-identical; side stream."""
    p = W.make("conv3x3_im2col", N=1003)
    N, C, M = p.N, p.C, p.M
    lut, scale, offset = W.random_codes(C, M, seed=3, max_shift=2)
    guard = 4096
    ybuf = torch.full((N * M + guard,), 12345.0, device=DEV)
    abuf = torch.full((N * M + guard,), -7, dtype=torch.int32, device=DEV)
    ibuf = torch.full((N * C + guard,), 0xAB, dtype=torch.uint8, device=DEV)
    y, acc, idx = ybuf[:N * M].view(N, M), abuf[:N * M].view(N, M), ibuf[:N * C].view(N, C)
    s = torch.cuda.Stream()
    args = (dev(p.A), dev(p.split), dev(p.thr), dev(lut), dev(scale), dev(offset))
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        mdn.matmul(*args, y_out=y, acc_out=acc, idx_out=idx)
    s.synchronize()
    first = (host(y).copy(), host(acc).copy(), host(idx).copy())
    assert np.all(host(ybuf[N * M:]) == 12345.0)
    assert np.all(host(abuf[N * M:]) == -7)
    assert np.all(host(ibuf[N * C:]) == 0xAB)
    ridx, racc, ry = orc.matmul(p.A, p.split, p.thr, lut, scale, offset)
    assert np.array_equal(first[2], ridx) and np.array_equal(first[1], racc)
    assert_y(first[0], ry)
    mdn.matmul(*args, y_out=y, acc_out=acc, idx_out=idx)
    assert np.array_equal(host(y), first[0]) and np.array_equal(host(acc), first[1])


def test_empty_inputs():
    A = torch.empty((0, 64), device=DEV)
    split = torch.zeros((4, 4), dtype=torch.int32, device=DEV)
    thr = torch.zeros((4, 15), device=DEV)
    idx = mdn.encode(A, split, thr)
    assert idx.shape == (0, 4)
    lut = torch.zeros((4, 16, 10), dtype=torch.int8, device=DEV)
    scale = torch.ones(4, device=DEV)
    offset = torch.zeros(4, device=DEV)
    y, _, _ = mdn.matmul(A, split, thr, lut, scale, offset)
    assert y.shape == (0, 10)


# ------------------------------------------------------ full-size, sampled
# workloads whose every row the oracle recomputes in well under a second
ALL_ROWS = ("classifier_tiny", "conv3x3_im2col")


def sample_rows(N, RW=64, seed=0, edge=1000, random=4000, cuts=200):
    """First and last `edge` rows, `random` rows drawn uniformly, and the two
    rows around `cuts` evenly spaced boundaries (chunk, work-item and tile
    edges fall among them)."""
    rng = np.random.default_rng(seed)
    rows = set(range(min(N, edge))) | set(range(max(0, N - edge), N))
    rows |= set(int(r) for r in rng.integers(0, N, size=random))
    for b in range(RW, N, max(RW, N // cuts)):
        rows |= {b - 1, b}
    return np.array(sorted(r for r in rows if 0 <= r < N))


def parity_rows(name, N):
    return np.arange(N) if name in ALL_ROWS else sample_rows(N)


@pytest.mark.slow
@pytest.mark.parametrize("name", list(W.SPECS))
def test_matmul_full_size_sampled(orc, name):
    """Full-size workload in the launch configuration the benchmark times.
    The oracle recomputes every row of the classifier and conv layers, and
    about 6000 rows of the three large layers (first and last 1000, 4000
    random, both sides of 200 evenly spaced boundaries)."""
    p = W.make(name)
    rows = parity_rows(name, p.N)
    A = dev(p.A)
    split, thr = dev(p.split), dev(p.thr)
    racc = acc = None
    if p.spec.quantized:
        lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
        y, acc, idx = mdn.matmul(A, split, thr, lut, scale, offset, want_acc=True, want_idx=True)
        rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
        assert np.array_equal(host(lut), rl)
        ridx, racc, ry = orc.matmul(p.A[rows], p.split, p.thr, rl, rs, ro)
    else:
        lut = mdn.build_lut_f32(dev(p.P), dev(p.B))
        y, idx = mdn.matmul_f32(A, split, thr, lut, want_idx=True)
        ridx, ry = orc.matmul_f32(p.A[rows], p.split, p.thr, orc.build_lut_f32(p.P, p.B))
    r = torch.from_numpy(rows).to(DEV)
    assert np.array_equal(host(idx[r]), ridx)
    if acc is not None:
        assert np.array_equal(host(acc[r]), racc)
    assert_y(host(y[r]), ry)
    # every index of every row is a valid leaf (a property at any size)
    assert int(idx.max()) < 16
    del y, acc, idx, A
    torch.cuda.empty_cache()


def test_prepared_call_matches(orc):
    p = W.make("conv3x3_im2col", N=2222)
    lut, scale, offset = W.random_codes(p.C, p.M, seed=11, max_shift=3)
    args = (dev(p.A), dev(p.split), dev(p.thr), dev(lut), dev(scale), dev(offset))
    call = mdn.prepare_matmul(*args)
    y, _, _ = call()
    first = host(y).copy()
    call()
    _, _, ry = orc.matmul(p.A, p.split, p.thr, lut, scale, offset)
    assert_y(first, ry)
    assert np.array_equal(host(y), first)
