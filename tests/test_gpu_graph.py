"""The entry points inside a captured HIP graph (torch.cuda.CUDAGraph): each
call enqueues kernels only, so a serving loop can capture it once and replay
it.  Every case is captured after one eager call, then replayed several
times with eager work, new input contents and synchronisations between the
replays; every replay is checked against the oracle for the inputs it saw.
The library never allocates: the two-phase matmul writes its indices to a
caller index array, which the Python binding takes from torch's allocator
(the graph's private pool under capture) when the caller passes none."""
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


def replay_and_check(g, A_dev, inputs, outputs, expected):
    """Replay g once per input set: load it into A_dev, clear the outputs
    eagerly, replay, compare with expected(i)."""
    for rnd in range(2):
        for i, A in enumerate(inputs):
            A_dev.copy_(torch.from_numpy(A).to(DEV))
            for o in outputs:
                o.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            expected(i, rnd)


@pytest.mark.parametrize("name,N", [("conv3x3_im2col", 3000), ("dense_hidden", 2000)])
def test_matmul_replays(orc, name, N):
    """Fused kernel (conv3x3_im2col's table fits in LDS) and the two-phase
    path (dense_hidden: encode, then the column-tiled accumulate)."""
    p = W.make(name, N=N)
    rng = np.random.default_rng(N)
    inputs = [p.A, (p.A * np.float32(-0.5) + rng.standard_normal(p.A.shape).astype(np.float32))]
    lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    A = dev(inputs[0])
    split, thr = dev(p.split), dev(p.thr)
    y = torch.empty((N, p.spec.M), device=DEV)
    idx = torch.empty((N, p.spec.C), dtype=torch.uint8, device=DEV)
    mdn.matmul(A, split, thr, lut, scale, offset, y_out=y, idx_out=idx)   # eager first call
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mdn.matmul(A, split, thr, lut, scale, offset, y_out=y, idx_out=idx)
    refs = [orc.matmul(x, p.split, p.thr, rl, rs, ro) for x in inputs]

    def expected(i, rnd):
        assert np.array_equal(host(idx), refs[i][0]), (i, rnd)
        assert np.array_equal(host(y), refs[i][2]), (i, rnd)

    replay_and_check(g, A, inputs, [y, idx], expected)


def test_matmul_act_softmax_replays(orc):
    """Rows spanning several column tiles: the accumulate writes z, then the
    row-softmax pass runs; both are in the graph."""
    p = W.make("dense_hidden", N=1500)
    rng = np.random.default_rng(5)
    inputs = [p.A, rng.standard_normal(p.A.shape).astype(np.float32)]
    lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
    rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
    bias = rng.standard_normal(p.spec.M).astype(np.float32)
    A, split, thr, b = dev(inputs[0]), dev(p.split), dev(p.thr), dev(bias)
    y = torch.empty((p.N, p.spec.M), device=DEV)
    idx = torch.empty((p.N, p.spec.C), dtype=torch.uint8, device=DEV)
    mdn.matmul_act(A, split, thr, lut, scale, offset, col_bias=b, act="softmax", y_out=y, idx_out=idx)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mdn.matmul_act(A, split, thr, lut, scale, offset, col_bias=b, act="softmax", y_out=y, idx_out=idx)
    M = p.spec.M
    refs = []
    for x in inputs:
        ridx, _, yref = orc.matmul(x, p.split, p.thr, rl, rs, ro)
        ref = orc.sigma(yref, bias, 3)
        z = orc.sigma(yref, bias, 1)
        tol = 1.01 * (np.abs(z - z.max(axis=1, keepdims=True)) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
        refs.append((ridx, ref, tol))

    def expected(i, rnd):
        ridx, ref, tol = refs[i]
        assert np.array_equal(host(idx), ridx), (i, rnd)
        assert np.all(np.abs(host(y).astype(np.float64) - ref) <= tol), (i, rnd)

    replay_and_check(g, A, inputs, [y, idx], expected)


def test_accumulate_avg_replays(orc):
    N, C, M = 3000, 64, 512
    lut, scale, offset = W.random_codes(C, M, seed=3, max_shift=0)
    inputs = [W.random_indices(N, C, seed=s) for s in (1, 2)]
    idx = dev(inputs[0])
    y = torch.empty((N, M), device=DEV)
    args = (dev(lut), dev(scale), dev(offset))
    mdn.lut_accumulate_avg(idx, *args, y_out=y)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mdn.lut_accumulate_avg(idx, *args, y_out=y)
    refs = [orc.lut_accumulate_avg(x, lut, scale, offset)[1] for x in inputs]

    def expected(i, rnd):
        assert np.array_equal(host(y), refs[i]), (i, rnd)

    replay_and_check(g, idx, inputs, [y], expected)


@pytest.mark.parametrize("name,N", [("dense_hidden", 16411), ("encode_heavy_f32", 4173)])
def test_two_phase_row_kernels_replay(orc, name, N):
    """Row counts large enough for the large-table accumulates (int8 table:
    dense_hidden, the one-hot product on the matrix cores; fp32 table:
    encode_heavy_f32, the row-uniform kernel), captured with a caller index
    buffer and replayed with new inputs."""
    p = W.make(name, N=N)
    rng = np.random.default_rng(N + 3)
    inputs = [p.A, rng.standard_normal(p.A.shape).astype(np.float32)]
    A = dev(inputs[0])
    split, thr = dev(p.split), dev(p.thr)
    y = torch.empty((N, p.spec.M), device=DEV)
    idx = torch.empty((N, p.spec.C), dtype=torch.uint8, device=DEV)
    if p.spec.quantized:
        lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
        rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
        call = lambda: mdn.matmul(A, split, thr, lut, scale, offset, y_out=y, idx_out=idx)
        refs = [orc.matmul(x, p.split, p.thr, rl, rs, ro) for x in inputs]
        refs = [(r[0], r[2]) for r in refs]
    else:
        tab = mdn.build_lut_f32(dev(p.P), dev(p.B))
        rtab = orc.build_lut_f32(p.P, p.B)
        call = lambda: mdn.matmul_f32(A, split, thr, tab, y_out=y, idx_out=idx)
        refs = [orc.matmul_f32(x, p.split, p.thr, rtab) for x in inputs]
    call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()

    def expected(i, rnd):
        assert np.array_equal(host(idx), refs[i][0]), (i, rnd)
        assert np.array_equal(host(y), refs[i][1]), (i, rnd)

    replay_and_check(g, A, inputs, [y, idx], expected)


@pytest.mark.parametrize("name,N", [("dense_hidden", 2000), ("dense_hidden", 16411), ("wide_layer", 3000),
                                    ("encode_heavy_f32", 4173)])
def test_two_phase_without_caller_index_array_replays(orc, name, N):
    """The two-phase path captured with no index array from the caller: the
    binding asks maddness_matmul_index_bytes, takes the array from torch's
    allocator inside the capture, and the replays match the oracle."""
    p = W.make(name, N=N)
    rng = np.random.default_rng(N + 7)
    inputs = [p.A, rng.standard_normal(p.A.shape).astype(np.float32)]
    A = dev(inputs[0])
    split, thr = dev(p.split), dev(p.thr)
    y = torch.empty((N, p.spec.M), device=DEV)
    f32 = not p.spec.quantized
    assert mdn.matmul_index_bytes(A, p.spec.C, p.spec.M, f32=f32) == N * p.spec.C
    if not f32:
        lut, scale, offset = mdn.build_lut(dev(p.P), dev(p.B))
        rl, rs, ro = orc.build_quantized_lut(p.P, p.B)
        call = lambda: mdn.matmul(A, split, thr, lut, scale, offset, y_out=y)
        refs = [orc.matmul(x, p.split, p.thr, rl, rs, ro)[2] for x in inputs]
    else:
        tab = mdn.build_lut_f32(dev(p.P), dev(p.B))
        rtab = orc.build_lut_f32(p.P, p.B)
        call = lambda: mdn.matmul_f32(A, split, thr, tab, y_out=y)
        refs = [orc.matmul_f32(x, p.split, p.thr, rtab)[1] for x in inputs]
    call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()

    def expected(i, rnd):
        assert np.array_equal(host(y), refs[i]), (i, rnd)

    replay_and_check(g, A, inputs, [y], expected)
