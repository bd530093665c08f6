"""Parity of the model-aware table fit (Eq. 3, affine output, reading R21)
and its pieces with the oracle, through the C ABI.

Bar: bit-exact everywhere.  The Gram counts are integers; the scatter sums
each entry's rows in ascending order in double on both sides; the solve
takes the same correctly rounded operations (fma, division, square root) in
the same order per entry on both sides (blocked on the GPU, unblocked in the
oracle), so the fitted tables agree to the bit.  The quantizer applied to a
given table is the build's quantizer: codes, scales and offsets bit-exact.
"""
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


def problem(N, C, M, seed, missing=()):
    rng = np.random.default_rng(seed)
    idx = W.random_indices(N, C, seed=seed)
    for c, k in missing:
        col = idx[:, c]
        col[col == k] = (k + 1) % 16
    Y = (rng.standard_normal((N, M)) * 3).astype(np.float32)
    T0 = rng.standard_normal((C, 16, M)).astype(np.float32)
    return idx, Y, T0


@pytest.mark.parametrize("N,C", [(0, 4), (1, 1), (300, 5), (1000, 8), (777, 17), (2049, 33), (513, 64)])
def test_gram_counts(orc, N, C):
    idx = W.random_indices(N, C, seed=N + C)
    H = host(mdn.encoder_gram(dev(idx)))
    assert np.array_equal(H.astype(np.int64), orc.encoder_gram(idx))


@pytest.mark.parametrize("N,C,M", [(0, 3, 10), (1, 1, 1), (257, 4, 63), (1000, 9, 64), (999, 16, 130),
                                   (3001, 32, 65)])
def test_scatter_sums(orc, N, C, M):
    idx, Y, _ = problem(N, C, M, seed=N + 7 * C + M)
    R = host(mdn.encoder_scatter(dev(idx), dev(Y)))
    assert np.array_equal(R, orc.encoder_scatter(idx, Y))


@pytest.mark.parametrize("N,C,M,lam", [(50, 1, 1, 0.5),        # one panel, 16 unknowns
                                       (400, 3, 7, 2.0),       # ragged last panel (48 = 32 + 16)
                                       (1000, 8, 64, 1e-3),    # weak regularisation
                                       (777, 17, 100, 10.0),   # 272 unknowns, ragged column tile
                                       (2000, 33, 130, 1.0),   # 528 unknowns
                                       (5000, 64, 40, 0.25)])  # 1024 unknowns
def test_fit_matches_oracle(orc, N, C, M, lam):
    idx, Y, T0 = problem(N, C, M, seed=N + C + M, missing=[(0, 3)])
    T = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), lam))
    ref = orc.fit_lut_ridge(idx, Y, T0, lam)
    assert np.array_equal(T, ref), f"max |diff| {np.abs(T - ref).max():.3g}"


def test_fit_empty_training_set(orc):
    """No rows: the penalty alone, so the fit returns T0 (up to the solve's rounding)."""
    _, _, T0 = problem(1, 6, 9, seed=3)
    idx = np.zeros((0, 6), np.uint8)
    Y = np.zeros((0, 9), np.float32)
    T = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), 0.3))
    assert np.array_equal(T, orc.fit_lut_ridge(idx, Y, T0, 0.3))
    assert np.allclose(T, T0, rtol=1e-14, atol=0)


def test_fit_reuses_workspace_and_rejects(orc):
    idx, Y, T0 = problem(300, 4, 12, seed=5)
    ws = torch.empty((1 << 20,), dtype=torch.uint8, device=DEV)
    a = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), 1.5, workspace=ws))
    b = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), 1.5, workspace=ws))
    assert np.array_equal(a, b) and np.array_equal(a, orc.fit_lut_ridge(idx, Y, T0, 1.5))
    for lam in (0.0, -1.0, float("nan")):
        with pytest.raises(mdn.MaddnessError):
            mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), lam)
    with pytest.raises(ValueError):
        mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), 1.0, workspace=ws[:1000])


@pytest.mark.parametrize("shared", [False, True])
def test_quantize_given_table(orc, shared):
    rng = np.random.default_rng(11 + shared)
    T = rng.standard_normal((12, 16, 37)) * np.exp(rng.uniform(-3, 3, size=(12, 1, 1)))
    lut, scale, offset = (host(t) for t in mdn.quantize_lut(dev(T), shared=shared))
    ref = orc.quantize_table_shared(T) if shared else orc.quantize_table(T)
    assert np.array_equal(lut, ref[0]) and np.array_equal(scale, ref[1]) and np.array_equal(offset, ref[2])


@pytest.mark.parametrize("name", ["conv3x3_im2col", "dense_hidden"])
def test_fit_on_workload_training_rows(orc, name):
    """A workload's own layer: training rows of A encoded by its trees,
    targets Y = AB, the prototype table as T0.  The fitted table equals the
    oracle's, and it lowers the objective of Eq. 3 below T0's."""
    p = W.make(name, N=4096)
    idx = orc.encode(p.A, p.split, p.thr)
    Y = (p.A.astype(np.float64) @ p.B.astype(np.float64)).astype(np.float32)
    T0 = orc.build_lut_f32(p.P, p.B)
    lam = 1.0
    T = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), lam))
    assert np.array_equal(T, orc.fit_lut_ridge(idx, Y, T0, lam))

    def objective(Tx):
        G = sum(np.asarray(Tx, np.float64)[c][idx[:, c]] for c in range(idx.shape[1]))
        r = Y.astype(np.float64) - G
        return float((r * r).sum() + lam * ((np.asarray(Tx, np.float64) - T0) ** 2).sum())

    assert objective(T) < objective(T0)
