"""Parity of the layer output sigma (§2.2: bias, then ReLU or a row softmax)
fused into the HIP path, against the oracle's sigma applied to the oracle's
product.

Bar: bias and ReLU outputs bit-exact (the same single fp32 rounding on both
sides, reading R19).  Softmax: the kernels evaluate it in fp32 (expf, their
own summation order); the oracle in double from the same fp32 inputs z.  With
u = 2^-24, d = z - max_row z and M terms, the fp32 evaluation carries a
relative error of at most |d| u (rounding of d, amplified by exp) + 4u (expf)
+ (M - 1) u (sum of positive terms, any order) + u (division), so the test
allows 1.01 (|d| + M + 5) u relative, plus 2^-120 absolute for results that
underflow in fp32.
"""
import numpy as np
import pytest
import torch

import paper_2207_05808_amd as mdn
from paper_2207_05808_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ACTS = ["none", "bias", "relu", "softmax"]
CODE = {"none": 0, "bias": 1, "relu": 2, "softmax": 3}


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def check_sigma(orc, y_gpu, y_ref, bias, act):
    """y_gpu: the kernel's sigma output; y_ref: the oracle's product (fp32)."""
    ref = orc.sigma(y_ref, bias, CODE[act])
    assert y_gpu.shape == ref.shape and y_gpu.dtype == np.float32
    if act != "softmax":
        assert np.array_equal(y_gpu.astype(np.float64), ref), \
            f"{int((y_gpu.astype(np.float64) != ref).sum())} outputs differ"
        if act == "relu":
            assert not np.any(np.signbit(y_gpu))
        return
    z = orc.sigma(y_ref, bias, 1)
    d = z - z.max(axis=1, keepdims=True)
    M = y_ref.shape[1]
    tol = 1.01 * (np.abs(d) + M + 5) * 2.0 ** -24 * ref + 2.0 ** -120
    err = np.abs(y_gpu.astype(np.float64) - ref)
    worst = float((err / tol).max())
    assert worst <= 1.0, f"softmax error {worst:.3f} x the bound"
    assert np.allclose(y_gpu.astype(np.float64).sum(axis=1), 1.0, rtol=0, atol=(M + 8) * 2.0 ** -23)


def col_bias_for(M, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(M) * scale).astype(np.float32)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("name", list(W.SPECS))
def test_matmul_act_workloads(orc, name, act):
    """Every workload (reduced N): fused kernel for the tables that fit in LDS,
    encode + column-tiled accumulate (+ a softmax pass when a row spans
    several column tiles) for the others."""
    N = {"classifier_tiny": 1024, "conv3x3_im2col": 2001, "dense_hidden": 1500, "wide_layer": 700,
         "encode_heavy_f32": 1000}[name]
    p = W.make(name, N=N)
    bias = col_bias_for(p.spec.M, seed=len(name) * 31 + CODE[act])
    if p.spec.quantized:
        lut, scale, offset = orc.build_quantized_lut(p.P, p.B)
        y = mdn.matmul_act(dev(p.A), dev(p.split), dev(p.thr), dev(lut), dev(scale), dev(offset),
                           col_bias=dev(bias), act=act, validate=True)
        _, _, yref = orc.matmul(p.A, p.split, p.thr, lut, scale, offset)
    else:
        lut = orc.build_lut_f32(p.P, p.B)
        y = mdn.matmul_act_f32(dev(p.A), dev(p.split), dev(p.thr), dev(lut), col_bias=dev(bias), act=act)
        _, yref = orc.matmul_f32(p.A, p.split, p.thr, lut)
    check_sigma(orc, host(y), yref, bias, act)


def random_layer(N, D, C, M, seed, max_shift=3):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut, scale, offset = W.random_codes(C, M, seed=seed + 1, max_shift=max_shift)
    return A, split, thr, lut, scale, offset


@pytest.mark.parametrize("act", ["relu", "softmax"])
@pytest.mark.parametrize("N,D,C,M", [(999, 96, 128, 100),    # column-tiled, one tile: softmax in the kernel
                                     (513, 64, 96, 10),      # C not dividing 64, M = 10
                                     (300, 40, 4, 77),       # fused kernel, M not a multiple of 8
                                     (257, 128, 64, 600)])   # several column tiles
def test_matmul_act_shapes(orc, N, D, C, M, act):
    A, split, thr, lut, scale, offset = random_layer(N, D, C, M, seed=N + D + C + M)
    bias = col_bias_for(M, seed=M)
    y = mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset), col_bias=dev(bias),
                       act=act)
    _, _, yref = orc.matmul(A, split, thr, lut, scale, offset)
    check_sigma(orc, host(y), yref, bias, act)


@pytest.mark.parametrize("act", ["bias", "relu", "softmax"])
@pytest.mark.parametrize("C,M", [(96, 40), (32, 24), (256, 200)])
def test_matmul_act_f32_shapes(orc, C, M, act):
    rng = np.random.default_rng(C * 100 + M)
    N, D = 701, 80
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, 4)).astype(np.int32)
    thr = rng.standard_normal((C, 15), dtype=np.float32)
    lut = W.random_fp32_table(C, M, seed=C + M)
    bias = col_bias_for(M, seed=M + 1)
    y = mdn.matmul_act_f32(dev(A), dev(split), dev(thr), dev(lut), col_bias=dev(bias), act=act)
    _, yref = orc.matmul_f32(A, split, thr, lut)
    check_sigma(orc, host(y), yref, bias, act)


@pytest.mark.parametrize("M", [10, 64, 512])
def test_softmax_large_logits_and_no_bias(orc, M):
    """Logits in the hundreds (a bias of +-300): the row maximum is subtracted
    before exp, so nothing overflows; and the same layer without a bias."""
    C = 32 if M != 512 else 64
    A, split, thr, lut, scale, offset = random_layer(640, 72, C, M, seed=M + 5)
    _, _, yref = orc.matmul(A, split, thr, lut, scale, offset)
    big = col_bias_for(M, seed=3, scale=300.0)
    y = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset),
                            col_bias=dev(big), act="softmax"))
    assert np.all(np.isfinite(y))
    check_sigma(orc, y, yref, big, "softmax")
    y0 = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset), act="softmax"))
    check_sigma(orc, y0, yref, None, "softmax")
    r0 = host(mdn.matmul_act(dev(A), dev(split), dev(thr), dev(lut), dev(scale), dev(offset), act="relu"))
    check_sigma(orc, r0, yref, None, "relu")


def test_act_none_matches_matmul(orc):
    p = W.make("conv3x3_im2col", N=1000)
    lut, scale, offset = orc.build_quantized_lut(p.P, p.B)
    args = (dev(p.A), dev(p.split), dev(p.thr), dev(lut), dev(scale), dev(offset))
    y0 = host(mdn.matmul_act(*args, act="none"))
    y1, _, _ = mdn.matmul(*args)
    assert np.array_equal(y0, host(y1))
