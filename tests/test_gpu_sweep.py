"""Seeded sweep over random shapes for the main entry points, each against the
oracle: N, D, C, M, row strides and table exponents drawn per case (a fixed
list of seeds, so every run checks the same cases).  Bar as in the other
parity tests: indices, accumulators and int8 outputs bit-exact, fp32-table
outputs bit-identical (same fixed summation order), averaging bit-exact,
softmax within the bound of the sigma tests."""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SEEDS = list(range(40))


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def draw(seed):
    rng = np.random.default_rng(1000 + seed)
    C = int(rng.choice([1, 2, 3, 4, 5, 8, 12, 16, 24, 32, 40, 64, 96, 128, 200]))
    D = int(rng.integers(1, 300))
    M = int(rng.choice([1, 3, 4, 7, 16, 33, 64, 100, 128, 250, 512, 700]))
    N = int(rng.integers(0, 1500))
    pad = int(rng.choice([0, 0, 1, 5]))          # row stride D + pad
    A = rng.standard_normal((N, D + pad), dtype=np.float32)[:, :D]
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    max_shift = int(rng.choice([0, 0, 2, 5]))
    lut, scale, offset = W.random_codes(C, M, seed=2000 + seed, max_shift=max_shift)
    return rng, A, split, thr, lut, scale, offset


def dev_rows(A):
    """Device copy keeping A's row stride (a view of a wider buffer)."""
    full = np.ascontiguousarray(A.base if A.base is not None else A)
    t = torch.from_numpy(full).to(DEV)
    return t[:, :A.shape[1]]


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_matmul(orc, seed):
    _, A, split, thr, lut, scale, offset = draw(seed)
    y, acc, idx = mdn.matmul(dev_rows(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                             want_acc=True, want_idx=True)
    ridx, racc, ry = orc.matmul(A, split, thr, lut, scale, offset)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_matmul_f32(orc, seed):
    _, A, split, thr, lut, _, _ = draw(seed)
    C, M = lut.shape[0], lut.shape[2]
    tab = W.random_fp32_table(C, M, seed=3000 + seed)
    y, idx = mdn.matmul_f32(dev_rows(A), dev(split), dev(thr), dev(tab), want_idx=True)
    ridx, ry = orc.matmul_f32(A, split, thr, tab)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(y), ry)


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_accumulate_and_avg(orc, seed):
    rng, A, split, thr, lut, scale, offset = draw(seed)
    N, C, M = A.shape[0], lut.shape[0], lut.shape[2]
    idx = W.random_indices(N, C, seed=4000 + seed)
    acc, y = mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), want_acc=True)
    racc, ry = orc.lut_accumulate(idx, lut, scale, offset)
    assert np.array_equal(host(acc), racc) and np.array_equal(host(y), ry)
    if C <= 128:
        slut, sscale, soffset = W.random_codes(C, M, seed=5000 + seed, max_shift=0)
        acc, y = mdn.lut_accumulate_avg(dev(idx), dev(slut), dev(sscale), dev(soffset), want_acc=True)
        racc, ry = orc.lut_accumulate_avg(idx, slut, sscale, soffset)
        assert np.array_equal(host(acc), racc) and np.array_equal(host(y), ry)


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_matmul_act(orc, seed):
    rng, A, split, thr, lut, scale, offset = draw(seed)
    M = lut.shape[2]
    bias = rng.standard_normal(M).astype(np.float32)
    act = ["bias", "relu", "softmax"][seed % 3]
    code = {"bias": 1, "relu": 2, "softmax": 3}[act]
    y = host(mdn.matmul_act(dev_rows(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                            col_bias=dev(bias), act=act))
    _, _, yref = orc.matmul(A, split, thr, lut, scale, offset)
    ref = orc.sigma(yref, bias, code)
    if act != "softmax":
        assert np.array_equal(y.astype(np.float64), ref)
        return
    z = orc.sigma(yref, bias, 1)
    d = z - (z.max(axis=1, keepdims=True) if z.size else 0.0)
    tol = 1.01 * (np.abs(d) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    assert np.all(np.abs(y.astype(np.float64) - ref) <= tol)


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_encode_and_f32_act(orc, seed):
    rng, A, split, thr, lut, _, _ = draw(seed)
    idx = host(mdn.encode(dev_rows(A), dev(split), dev(thr)))
    assert np.array_equal(idx, orc.encode(A, split, thr))
    C, M = lut.shape[0], lut.shape[2]
    tab = W.random_fp32_table(C, M, seed=6000 + seed)
    bias = rng.standard_normal(M).astype(np.float32)
    act = ["bias", "relu"][seed % 2]
    y = host(mdn.matmul_act_f32(dev_rows(A), dev(split), dev(thr), dev(tab), col_bias=dev(bias), act=act))
    _, yref = orc.matmul_f32(A, split, thr, tab)
    assert np.array_equal(y.astype(np.float64), orc.sigma(yref, bias, {"bias": 1, "relu": 2}[act]))


@pytest.mark.parametrize("seed", SEEDS[:16])
def test_sweep_fit(orc, seed):
    """Gram counts, G^T Y and the closed-form fit on random shapes (C up to
    40, so the oracle's dense solve stays fast)."""
    rng = np.random.default_rng(7000 + seed)
    N = int(rng.integers(0, 3000))
    C = int(rng.choice([1, 2, 3, 5, 8, 13, 20, 32, 40]))
    M = int(rng.choice([1, 2, 7, 63, 64, 65, 130]))
    idx = W.random_indices(N, C, seed=8000 + seed)
    Y = (rng.standard_normal((N, M)) * 2).astype(np.float32)
    T0 = rng.standard_normal((C, 16, M)).astype(np.float32)
    lam = float(rng.choice([0.01, 0.5, 3.0]))
    assert np.array_equal(host(mdn.encoder_gram(dev(idx))).astype(np.int64), orc.encoder_gram(idx))
    assert np.array_equal(host(mdn.encoder_scatter(dev(idx), dev(Y))), orc.encoder_scatter(idx, Y))
    assert np.array_equal(host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), lam)), orc.fit_lut_ridge(idx, Y, T0, lam))


def shifted(x, dtype):
    """Device copy of x starting one element past a fresh allocation (so not
    16-byte aligned)."""
    flat = torch.empty(x.size + 1, dtype=dtype, device=DEV)
    v = flat[1:].view(x.shape)
    v.copy_(torch.from_numpy(np.ascontiguousarray(x)).to(DEV))
    return v


@pytest.mark.parametrize("seed", SEEDS[:16])
def test_sweep_misaligned(orc, seed):
    """A, tables, indices and outputs off 16-byte alignment: the entry points
    take their element-wise paths and give the same results."""
    _, A, split, thr, lut, scale, offset = draw(seed)
    A = np.ascontiguousarray(A)
    N, C, M = A.shape[0], lut.shape[0], lut.shape[2]
    Ad, lutd = shifted(A, torch.float32), shifted(lut, torch.int8)
    y_out = torch.empty(N * M + 1, dtype=torch.float32, device=DEV)[1:].view(N, M)
    y, _, _ = mdn.matmul(Ad, dev(split), dev(thr), lutd, dev(scale), dev(offset), y_out=y_out)
    _, _, ry = orc.matmul(A, split, thr, lut, scale, offset)
    assert np.array_equal(host(y), ry)
    idx = W.random_indices(N, C, seed=9000 + seed)
    idxd = shifted(idx, torch.uint8)
    _, y = mdn.lut_accumulate(idxd, lutd, dev(scale), dev(offset), y_out=y_out)
    assert np.array_equal(host(y), orc.lut_accumulate(idx, lut, scale, offset)[1])
    tab = W.random_fp32_table(C, M, seed=9500 + seed)
    y = mdn.lut_accumulate_f32(idxd, shifted(tab, torch.float32), y_out=y_out)
    assert np.array_equal(host(y), orc.lut_accumulate_f32(idx, tab))


@pytest.mark.parametrize("M", [1, 3, 10, 12, 33])
@pytest.mark.parametrize("off", [0, 1, 2, 3])
def test_general_kernel_table_at_any_byte_offset(orc, M, off):
    """Small layers whose table rows are not whole 16-byte units run the
    general single-launch kernel, which reads the int8 table one dword per
    four columns at any byte alignment (the table's last dword shifted down
    from its last four bytes).  Tables placed 0-3 bytes past an allocation,
    ragged N over several chunks: indices, accumulators and outputs
    bit-exact."""
    rng = np.random.default_rng(7100 + 10 * M + off)
    C, D, N = 4, 64, 4100 + M
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=7200 + M, max_shift=3)
    flat = torch.empty(lut.size + off, dtype=torch.int8, device=DEV)
    lutd = flat[off:].view(lut.shape)
    lutd.copy_(dev(lut))
    y, acc, idx = mdn.matmul(dev(A), dev(split), dev(thr), lutd, dev(scale), dev(offset),
                             want_acc=True, want_idx=True)
    ridx, racc, ry = orc.matmul(A, split, thr, lut, scale, offset)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(acc), racc)
    assert np.array_equal(host(y), ry)
