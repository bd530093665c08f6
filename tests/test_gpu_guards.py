"""Output bounds and run-to-run determinism of every kernel family.

Each output array is a view into a larger buffer with 4096 sentinel elements
before and after it; after the call the sentinels must be untouched, a
second call into outputs refilled with other values must give bit-identical
results, and sampled rows must match the oracle (indices, int32 sums and
outputs bit-exact, the same bar as the parity tests).  One case per kernel
family, at a shape that the planner routes to it."""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
G = 4096   # sentinel elements on each side


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


class Guarded:
    """An output view with sentinels around it."""

    def __init__(self, shape, dtype, fill):
        n = int(np.prod(shape))
        self.n, self.fill = n, fill
        self.buf = torch.full((G + n + G,), fill, dtype=dtype, device=DEV)
        self.view = self.buf[G:G + n].view(*shape)

    def refill(self, value):
        self.view.fill_(value)

    def check_sentinels(self):
        b = host(self.buf)
        assert np.all(b[:G] == self.fill), "write before the output"
        assert np.all(b[G + self.n:] == self.fill), "write past the output"


def rows_of(N, n=1024, seed=0):
    if N <= 4 * n:
        return np.arange(N)
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(n // 4), np.arange(N - n // 4, N), rng.integers(0, N, n // 2)]))


def layer(N, D, C, M, seed, max_shift=1):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=seed + 1, max_shift=max_shift)
    return A, split, thr, lut, scale, offset


def run_twice(call, outs):
    call()
    first = [host(o.view).copy() for o in outs]
    for o in outs:
        o.check_sentinels()
    for o, v in zip(outs, (77, 55, 33)):
        o.refill(v)
    call()
    for o, f in zip(outs, first):
        assert np.array_equal(host(o.view), f), "second run differs"
        o.check_sentinels()
    return first


FUSED = [  # (kernel family, N, D, C, M, outputs)
    ("general", 4100, 64, 4, 10, "yai"),
    ("gather-fused", 5003, 576, 32, 64, "yai"),
    ("row-streaming", 98304 + 17, 64, 64, 128, "yi"),   # (table too large for the gather-fused kernel)
]


@pytest.mark.parametrize("name,N,D,C,M,outs", FUSED, ids=[c[0] for c in FUSED])
def test_fused_guards(orc, name, N, D, C, M, outs):
    A, split, thr, lut, scale, offset = layer(N, D, C, M, seed=N + C)
    y = Guarded((N, M), torch.float32, 12345.0)
    acc = Guarded((N, M), torch.int32, -7) if "a" in outs else None
    idx = Guarded((N, C), torch.uint8, 0xAB) if "i" in outs else None
    args = [dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset)]
    present = [o for o in (y, acc, idx) if o is not None]
    first = run_twice(lambda: mdn.matmul(*args, y_out=y.view, acc_out=acc.view if acc else None,
                                         idx_out=idx.view if idx else None), present)
    r = rows_of(N)
    ridx, racc, ry = orc.matmul(A[r], split, thr, lut, scale, offset)
    assert np.array_equal(first[0][r], ry)
    if acc:
        assert np.array_equal(first[1][r], racc)
    if idx:
        assert np.array_equal(first[-1][r], ridx)


ACCUM = [  # (kernel family, N, C, M, table, with int32 sums, spread of the block exponents)
    ("one-hot-product", 20485, 64, 512, "i8", True, 1),
    ("one-row-per-lane-int8", 20485, 256, 512, "i8", False, 0),   # (past the one-hot product's 128 codebooks)
    ("row-uniform", 20485, 256, 512, "i8", True, 1),
    ("column-tiled", 5001, 96, 200, "i8", True, 1),
    ("gather-fused-indices", 5003, 32, 64, "i8", True, 1),
    ("one-row-per-lane-fp32", 20485, 32, 1000, "f32", False, 0),
    ("averaging", 5001, 64, 512, "avg", False, 0),
]


@pytest.mark.parametrize("name,N,C,M,table,with_acc,max_shift", ACCUM, ids=[c[0] for c in ACCUM])
def test_accumulate_guards(orc, name, N, C, M, table, with_acc, max_shift):
    idx = W.random_indices(N, C, seed=N + M)
    y = Guarded((N, M), torch.float32, 12345.0)
    acc = Guarded((N, M), torch.int32, -7) if with_acc else None
    present = [o for o in (y, acc) if o is not None]
    r = rows_of(N)
    if table == "f32":
        tab = W.random_fp32_table(C, M, seed=N)
        first = run_twice(lambda: mdn.lut_accumulate_f32(dev(idx), dev(tab), y_out=y.view), present)
        assert np.array_equal(first[0][r], orc.lut_accumulate_f32(idx[r], tab))
        return
    lut, scale, offset = W.random_codes(C, M, seed=N + 1, max_shift=max_shift)
    if table == "avg":   # (max_shift 0: one block exponent shared by every codebook)
        first = run_twice(lambda: mdn.lut_accumulate_avg(dev(idx), dev(lut), dev(scale), dev(offset),
                                                         y_out=y.view), present)
        assert np.array_equal(first[0][r], orc.lut_accumulate_avg(idx[r], lut, scale, offset)[1])
        return
    first = run_twice(lambda: mdn.lut_accumulate(dev(idx), dev(lut), dev(scale), dev(offset), y_out=y.view,
                                                 acc_out=acc.view if acc else None), present)
    racc, ry = orc.lut_accumulate(idx[r], lut, scale, offset)
    assert np.array_equal(first[0][r], ry)
    if acc:
        assert np.array_equal(first[1][r], racc)


def test_encode_guards(orc):
    N, D, C = 5001, 1024, 128
    A, split, thr, _, _, _ = layer(N, D, C, 16, seed=91)
    idx = Guarded((N, C), torch.uint8, 0xAB)
    first = run_twice(lambda: mdn.encode(dev(A), dev(split), dev(thr), idx_out=idx.view), [idx])
    assert np.array_equal(first[0], orc.encode(A, split, thr))
