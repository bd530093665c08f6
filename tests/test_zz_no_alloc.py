"""maddness_matmul_noalloc (for callers that cannot allocate) against
maddness_matmul with a caller index array, through the C ABI: outputs
bit-identical on consecutive calls (the second smaller, so the scratch array
holds the first call's indices when it starts), on a call large enough to run
in two row chunks, and on shapes that never touch the scratch array."""
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


def layer(N, D, C, M, seed):
    """Random trees over D columns, int8 codes with per-codebook shifts <= 2."""
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=seed + 1, max_shift=2)
    return A, split, thr, lut, scale, offset


def both(A, split, thr, lut, scale, offset):
    """(noalloc y, acc) and (matmul y, acc, idx) on the same device inputs."""
    N, C, M = A.shape[0], split.shape[0], lut.shape[2]
    args = [dev(x) for x in (A, split, thr, lut, scale, offset)]
    y0 = torch.full((N, M), float("nan"), device=DEV)
    a0 = torch.full((N, M), -7, dtype=torch.int32, device=DEV)
    mdn.matmul_noalloc(*args, y_out=y0, acc_out=a0)
    y1, a1, i1 = mdn.matmul(*args, want_acc=True, want_idx=True)
    return host(y0), host(a0), host(y1), host(a1), host(i1)


def test_noalloc_two_calls_second_smaller(orc):
    """Call 1: C = 512, M = 512, 100000 rows: two chunks of 65536 rows
    through the 32 MiB scratch array.  Call 2: the dense hidden layer at
    3000 rows (C = 64, M = 512), one chunk, after call 1's indices."""
    A, split, thr, lut, scale, offset = layer(100000, 64, 512, 512, seed=11)
    y0, a0, y1, a1, idx = both(A, split, thr, lut, scale, offset)
    assert np.array_equal(a0, a1) and np.array_equal(y0, y1)
    rows = np.r_[0:700, 65536 - 300:65536 + 300, 100000 - 700:100000]
    racc, ry = orc.lut_accumulate(orc.encode(A[rows], split, thr), lut, scale, offset)
    assert np.array_equal(a0[rows], racc) and np.array_equal(y0[rows], ry)

    p = W.make("dense_hidden", N=3000)
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    y0, a0, y1, a1, _ = both(p.A, p.split, p.thr, rl, rs, ro)
    assert np.array_equal(a0, a1) and np.array_equal(y0, y1)
    _, racc, ry = orc.matmul(p.A, p.split, p.thr, rl, rs, ro)
    assert np.array_equal(a0, racc) and np.array_equal(y0, ry)


def test_noalloc_repeat_and_other_paths(orc):
    """The same two-phase call twice in a row on one stream (the scratch
    array reused), a shape whose table fits the single-launch kernel (no
    scratch), and a caller index array (written as by maddness_matmul)."""
    A, split, thr, lut, scale, offset = layer(20000, 128, 64, 512, seed=5)
    first = both(A, split, thr, lut, scale, offset)
    second = both(A, split, thr, lut, scale, offset)
    for a, b in zip(first, second):
        assert np.array_equal(a, b)
    assert np.array_equal(first[0], first[2]) and np.array_equal(first[1], first[3])

    p = W.make("conv3x3_im2col", N=2000)
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    y0, a0, y1, a1, _ = both(p.A, p.split, p.thr, rl, rs, ro)
    assert np.array_equal(a0, a1) and np.array_equal(y0, y1)

    p = W.make("dense_hidden", N=1000)
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    args = [dev(x) for x in (p.A, p.split, p.thr, rl, rs, ro)]
    idx = torch.zeros((1000, 64), dtype=torch.uint8, device=DEV)
    y = torch.empty((1000, 512), device=DEV)
    mdn.matmul_noalloc(*args, y_out=y, idx_out=idx)
    ridx, _, ry = orc.matmul(p.A, p.split, p.thr, rl, rs, ro)
    assert np.array_equal(host(idx), ridx) and np.array_equal(host(y), ry)
