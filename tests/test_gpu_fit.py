"""Parity of the model-aware table fit (Eq. 3: affine output, reading R21;
ReLU and softmax outputs by gradient descent, reading R22) and its pieces with
the oracle, through the C ABI.

Bar: bit-exact everywhere except the softmax fit (bound derived below).  The Gram counts are integers; the scatter sums
each entry's rows in ascending order in double on both sides; the solve
takes the same correctly rounded operations (fma, division, square root) in
the same order per entry on both sides (blocked on the GPU, unblocked in the
oracle), so the fitted tables agree to the bit.  The quantizer applied to a
given table is the table builder's quantizer: codes, scales and offsets bit-exact.
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


# ------------------------------------------------ nonlinear output (R22)
# (N, C, M, lambda, step as a fraction of 1 / L, steps, bias)
GD_CASES = [(200, 2, 5, 0.2, 1.0, 10, False),
            (700, 8, 64, 0.0, 0.5, 6, True),
            (1500, 17, 100, 1.0, 1.0, 5, True),
            (999, 32, 10, 0.5, 1.5, 8, False)]


def lipschitz(orc, idx, lam):
    """L = lambda_max(G^T G) / 2 + 2 lambda bounds the curvature of the
    softmax objective (the Hessian of log-sum-exp has norm <= 1/2); a step
    eta <= 2 / L makes the exact gradient step non-expansive."""
    H = orc.encoder_gram(idx).astype(np.float64)
    return 0.5 * float(np.linalg.eigvalsh(H)[-1]) + 2.0 * lam


@pytest.mark.parametrize("N,C,M,lam,frac,iters,with_bias", GD_CASES)
def test_fit_gd_relu_matches_oracle(orc, N, C, M, lam, frac, iters, with_bias):
    """ReLU + squared error: every operation is correctly rounded and in the
    same order on both sides, so the tables agree to the bit."""
    idx, Y, T0 = problem(N, C, M, seed=N + C + M + iters)
    bias = np.random.default_rng(N).standard_normal(M).astype(np.float32) if with_bias else None
    eta = frac / (2.0 * lipschitz(orc, idx, lam))
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "relu", lam, eta, iters,
                            col_bias=dev(bias) if with_bias else None))
    ref = orc.fit_lut_gd(idx, Y, T0, 2, lam, eta, iters, bias)
    assert np.array_equal(T, ref), f"max |diff| {np.abs(T - ref).max():.3g}"


def softmax_tolerance(idx, C, M, eta, iters, tmax):
    """Bound on max |T_gpu - T_oracle| after K softmax steps with eta <= 2 / L.
    Against the exact step, each side's computed step errs only by rounding:
    a probability (exp within 1 ulp, an M-term sum, a division) by at most
    (2M + 4) u, so a residual entry (two of them) by (4M + 8) u; a gradient
    entry, a sum over its bucket's Nb rows, by Nb (4M + 8) u plus its own
    rounding, at most Nb^2 u; the update by 4 u |T|.  The exact step is
    non-expansive, so the two sides drift apart by at most the sum of both
    sides' errors per step: in the 2-norm over the 16 C M entries,
    K (eta (Nb (4M + 8) + Nb^2) + 4 tmax) u sqrt(16 C M) x 2."""
    u = 2.0 ** -53
    Nb = max(int(np.bincount(idx[:, c], minlength=16).max()) for c in range(C))
    return 2 * iters * (eta * (Nb * (4 * M + 8) + Nb * Nb) + 4 * tmax) * u * np.sqrt(16 * C * M)


@pytest.mark.parametrize("N,C,M,lam,frac,iters,with_bias", GD_CASES)
def test_fit_gd_softmax_matches_oracle(orc, N, C, M, lam, frac, iters, with_bias):
    idx, Y, T0 = problem(N, C, M, seed=N + 2 * C + M)
    bias = np.random.default_rng(N + 1).standard_normal(M).astype(np.float32) if with_bias else None
    eta = frac / lipschitz(orc, idx, lam)
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "softmax", lam, eta, iters,
                            col_bias=dev(bias) if with_bias else None))
    ref = orc.fit_lut_gd(idx, Y, T0, 3, lam, eta, iters, bias)
    tol = softmax_tolerance(idx, C, M, eta, iters, float(np.abs(ref).max()))
    err = float(np.abs(T - ref).max())
    assert err <= tol, f"max |diff| {err:.3g} > bound {tol:.3g}"


def softmax_sqerr_tolerance(idx, C, M, eta, iters, tmax, lip):
    """Bound on max |T_gpu - T_oracle| after K steps of the squared error
    between row softmaxes.  Per side, against the exact step from the same
    T: with each probability within e = (2M + 4) u relative (as above), the
    difference d = p - p* errs by (e + u)(p + p*), the weighted sum
    s = sum d p by 4 e + (2M + 4) u, and the residual r = 2 p (d - s) by
    2 (10 e + (2M + 14) u) <= (44 M + 108) u; |r| <= 6, so a gradient entry
    over its Nb rows errs by Nb (44 M + 108) u + 6 Nb^2 u and the update by
    4 u |T|.  This objective is not convex, so the exact step is not
    non-expansive: with its gradient L-Lipschitz (L = lip) the step map is
    (1 + eta L)-Lipschitz, and the two sides drift apart by at most
    K (1 + eta L)^(K - 1) times both sides' per-step errors (2-norm over the
    16 C M entries)."""
    u = 2.0 ** -53
    Nb = max(int(np.bincount(idx[:, c], minlength=16).max()) for c in range(C))
    step = (eta * (Nb * (44 * M + 108) + 6 * Nb * Nb) + 4 * tmax) * u * np.sqrt(16 * C * M)
    return 2 * iters * (1 + eta * lip) ** max(iters - 1, 0) * step


def lipschitz_sqerr(orc, idx, lam):
    """The Hessian of ||softmax(z) - p*||^2 in z has norm <= 10.5 (2 J^T J
    with ||J|| <= 1/2, plus sum_i d_i Hess(p_i) with ||Hess(p_i)|| <= 2.5 p_i
    and sum_i |d_i| p_i <= 2), so L = 10.5 lambda_max(G^T G) + 2 lambda."""
    H = orc.encoder_gram(idx).astype(np.float64)
    return 10.5 * float(np.linalg.eigvalsh(H)[-1]) + 2.0 * lam


@pytest.mark.parametrize("N,C,M,lam,frac,iters,with_bias", GD_CASES)
def test_fit_gd_softmax_sqerr_matches_oracle(orc, N, C, M, lam, frac, iters, with_bias):
    """Eq. 3 as written for a softmax output: the squared error between the
    row softmaxes of the table's outputs and the targets."""
    idx, Y, T0 = problem(N, C, M, seed=N + 3 * C + M)
    bias = np.random.default_rng(N + 2).standard_normal(M).astype(np.float32) if with_bias else None
    lip = lipschitz_sqerr(orc, idx, lam)
    eta = min(frac, 1.0) / lip
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "softmax_sqerr", lam, eta, iters,
                            col_bias=dev(bias) if with_bias else None))
    ref = orc.fit_lut_gd(idx, Y, T0, 4, lam, eta, iters, bias)
    tol = softmax_sqerr_tolerance(idx, C, M, eta, iters, float(np.abs(ref).max()), lip)
    err = float(np.abs(T - ref).max())
    assert err <= tol, f"max |diff| {err:.3g} > bound {tol:.3g}"
    assert np.abs(T - T0).max() > 100 * tol   # the steps moved the table well past the bound


def test_fit_gd_softmax_sqerr_classifier(orc):
    """The classifier workload (C = 4, M = 10) under Eq. 3's squared error
    between softmaxes: the GPU fit matches the oracle within the bound and
    lowers that objective below the prototype table's."""
    p = W.make("classifier_tiny")
    idx = orc.encode(p.A[:512], p.split, p.thr)
    Y = (p.A[:512].astype(np.float64) @ p.B.astype(np.float64)).astype(np.float32)
    T0 = orc.build_lut_f32(p.P, p.B)
    lam, iters = 0.1, 40
    lip = lipschitz_sqerr(orc, idx, lam)
    eta = 1.0 / lip
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "softmax_sqerr", lam, eta, iters))
    ref = orc.fit_lut_gd(idx, Y, T0, 4, lam, eta, iters)
    assert np.abs(T - ref).max() <= softmax_sqerr_tolerance(idx, 4, 10, eta, iters, float(np.abs(ref).max()), lip)
    from scipy.special import softmax

    def sqerr(Tx):
        z = sum(np.asarray(Tx, np.float64)[c][idx[:, c]] for c in range(4))
        d = softmax(z, axis=1) - softmax(Y.astype(np.float64), axis=1)
        return float((d * d).sum())

    assert sqerr(T) < sqerr(T0)


def test_fit_gd_zero_steps_and_rejects(orc):
    idx, Y, T0 = problem(100, 3, 7, seed=9)
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "softmax", 0.1, 0.01, 0))
    assert np.array_equal(T, T0.astype(np.float64))
    for act, lam, eta, iters in (("relu", -1.0, 0.01, 2), ("relu", 0.1, 0.0, 2),
                                 ("softmax", 0.1, 0.01, -1), ("softmax_sqerr", -0.5, 0.01, 2), (1, 0.1, 0.01, 2),
                                 (5, 0.1, 0.01, 2)):
        with pytest.raises(mdn.MaddnessError):
            mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), act, lam, eta, iters)


def test_fit_gd_softmax_classifier(orc):
    """The paper's softmax-classifier setting on the classifier workload
    (C = 4, M = 10): the KL-divergence fit on 512 training rows (step 1 / L)
    matches the oracle within the bound and lowers the training objective
    below the prototype table's."""
    p = W.make("classifier_tiny")
    idx = orc.encode(p.A[:512], p.split, p.thr)
    Y = (p.A[:512].astype(np.float64) @ p.B.astype(np.float64)).astype(np.float32)
    T0 = orc.build_lut_f32(p.P, p.B)
    lam, iters = 0.1, 40
    eta = 1.0 / lipschitz(orc, idx, lam)
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "softmax", lam, eta, iters))
    ref = orc.fit_lut_gd(idx, Y, T0, 3, lam, eta, iters)
    assert np.abs(T - ref).max() <= softmax_tolerance(idx, 4, 10, eta, iters, float(np.abs(ref).max()))
    from scipy.special import rel_entr, softmax

    def kl(Tx):
        z = sum(np.asarray(Tx, np.float64)[c][idx[:, c]] for c in range(4))
        return float(rel_entr(softmax(Y.astype(np.float64), axis=1), softmax(z, axis=1)).sum())

    assert kl(T) < kl(T0)


@pytest.mark.slow
def test_fits_at_benchmark_size(orc):
    """The benchmark's fit configuration on dense_hidden: 16384 training rows,
    C = 64, M = 512 (1024 unknowns per column), lambda = 1; the closed-form
    fit and three ReLU gradient steps equal the oracle's bit for bit."""
    p = W.make("dense_hidden", N=16384)
    idx = orc.encode(p.A, p.split, p.thr)
    Y = (p.A.astype(np.float64) @ p.B.astype(np.float64)).astype(np.float32)
    T0 = orc.build_lut_f32(p.P, p.B)
    T = host(mdn.fit_lut_ridge(dev(idx), dev(Y), dev(T0), 1.0))
    assert np.array_equal(T, orc.fit_lut_ridge(idx, Y, T0, 1.0))
    nb = max(int(np.bincount(idx[:, c], minlength=16).max()) for c in range(64))
    eta = 1.0 / (2.0 * 64 * nb + 2.0)
    T = host(mdn.fit_lut_gd(dev(idx), dev(Y), dev(T0), "relu", 1.0, eta, 3))
    assert np.array_equal(T, orc.fit_lut_gd(idx, Y, T0, 2, 1.0, eta, 3))
