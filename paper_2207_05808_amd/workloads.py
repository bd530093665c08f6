"""Seeded synthetic inputs for the encode + lookup-accumulate path.

This module only draws random numbers (numpy, host memory).  It contains none
of the method's arithmetic: no encoding, no table products, no quantization.
Both the HIP path and the CPU oracle take their inputs from here.

The five named workloads stand in for the layers studied in the paper (a
classifier layer over 512-wide activations, §3.1; MLP layers, §3.2) and for
the layer shapes of a small CNN; no dataset or trained weight is used.  Each
draws, from independent child streams of one seed:
  A      activations [N][D] fp32,
  split  split columns [C][4] int32 (global column indices),
  thr    thresholds [C][15] fp32 in heap order,
  P      prototypes [C][16][D] fp32, zero outside codebook c's subspace,
  B      weights [D][M] fp32.
Subspaces are C contiguous blocks of D / C columns (optionally after a random
permutation of the columns, which then also applies to split and P).
Because every array has its own stream, a workload drawn with fewer rows N
has exactly the same trees, prototypes and weights as the full-size one, and
its rows are a prefix of the full-size rows.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

K, LEVELS, NODES = 16, 4, 15


@dataclasses.dataclass(frozen=True)
class Spec:
    name: str
    N: int
    D: int
    C: int
    M: int
    a_dist: str          # "normal" | "halfnormal_im2col" | "normal_zero10"
    thr_dist: str        # "normal" | "halfnormal" | "sorted_per_dim"
    p_dist: str          # "normal" | "halfnormal" | "bin_midpoints"
    b_std: float
    quantized: bool      # int8 block-FP table (True) or fp32 table (False)
    seed: int
    note: str


SPECS = {
    s.name: s
    for s in [
        Spec("classifier_tiny", 1024, 64, 4, 10, "normal", "normal", "normal", 1.0, True, 220705808,
             "classifier layer, 64-d activations, 10 classes, 4 codebooks of 16 dims"),
        Spec("conv3x3_im2col", 131072, 576, 32, 64, "halfnormal_im2col", "halfnormal", "halfnormal",
             float(np.sqrt(0.05)), True, 220705809,
             "3x3 conv over 64 channels as im2col (128 images x 32x32 positions), post-ReLU "
             "activations |N(0,1)| with zero padding, 32 codebooks of 18 dims, 64 filters"),
        Spec("dense_hidden", 1048576, 512, 64, 512, "normal", "normal", "normal",
             float(1.0 / np.sqrt(512)), True, 220705810,
             "dense hidden layer 512->512, 64 codebooks of 8 dims"),
        Spec("wide_layer", 262144, 1024, 128, 4096, "normal_zero10", "normal", "normal",
             float(1.0 / np.sqrt(1024)), True, 220705811,
             "wide layer 1024->4096 with 10% exact-zero activations, 128 codebooks of 8 dims; "
             "its int8 table (8 MB) exceeds LDS"),
        Spec("encode_heavy_f32", 524288, 256, 256, 1024, "normal", "sorted_per_dim", "bin_midpoints",
             float(1.0 / np.sqrt(256)), False, 220705812,
             "one dim per codebook (all 4 levels split on it, sorted thresholds), fp32 table"),
    ]
}

# the workload the headline throughput is quoted on
HEADLINE = "conv3x3_im2col"


@dataclasses.dataclass
class Problem:
    spec: Spec
    N: int
    A: np.ndarray        # [N][D] float32
    split: np.ndarray    # [C][4] int32
    thr: np.ndarray      # [C][15] float32
    P: np.ndarray        # [C][16][D] float32
    B: np.ndarray        # [D][M] float32
    perm: np.ndarray     # [D] column permutation applied to the subspaces

    @property
    def D(self):
        return self.spec.D

    @property
    def C(self):
        return self.spec.C

    @property
    def M(self):
        return self.spec.M


def heap_from_sorted(s: np.ndarray) -> np.ndarray:
    """Place 15 sorted thresholds in heap order so that the tree is a binary
    search tree: node (t, i) gets s[(2i + 1) * 2^(3 - t) - 1]."""
    out = np.empty(s.shape[:-1] + (NODES,), dtype=s.dtype)
    for t in range(LEVELS):
        for i in range(1 << t):
            out[..., (1 << t) - 1 + i] = s[..., (2 * i + 1) * (1 << (3 - t)) - 1]
    return out


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.default_rng(c) for c in ss.spawn(6)]


def _im2col_rows(rng, N: int, D: int) -> np.ndarray:
    """Rows of the im2col matrix of a [images][64][32][32] tensor of |N(0,1)|
    values, 3x3 window, stride 1, zero padding 1; column order (ky, kx, ch)."""
    ch, H, W = 64, 32, 32
    assert D == 9 * ch
    per_img = H * W
    n_img = (N + per_img - 1) // per_img
    out = np.empty((n_img * per_img, D), dtype=np.float32)
    for b in range(n_img):
        x = np.abs(rng.standard_normal((H, W, ch), dtype=np.float32))
        xp = np.zeros((H + 2, W + 2, ch), dtype=np.float32)
        xp[1:-1, 1:-1] = x
        blk = out[b * per_img:(b + 1) * per_img].reshape(H, W, 3, 3, ch)
        for ky in range(3):
            for kx in range(3):
                blk[:, :, ky, kx, :] = xp[ky:ky + H, kx:kx + W, :]
    return out[:N]


def draw_A(spec: Spec, N: int, rng) -> np.ndarray:
    if spec.a_dist == "normal":
        return rng.standard_normal((N, spec.D), dtype=np.float32)
    if spec.a_dist == "halfnormal_im2col":
        return _im2col_rows(rng, N, spec.D)
    if spec.a_dist == "normal_zero10":
        A = rng.standard_normal((N, spec.D), dtype=np.float32)
        A[rng.random((N, spec.D), dtype=np.float32) < 0.1] = 0.0
        return A
    raise ValueError(spec.a_dist)


def make(name: str, N: Optional[int] = None, permute: bool = False, seed: Optional[int] = None
         ) -> Problem:
    """Draw workload `name` with N rows (default: its full size)."""
    spec = SPECS[name]
    N = spec.N if N is None else int(N)
    rA, rT, rP, rB, rPerm, _ = _streams(spec.seed if seed is None else seed)
    D, C, M = spec.D, spec.C, spec.M
    if D % C:
        raise ValueError("D must be a multiple of C")
    L = D // C
    perm = rPerm.permutation(D).astype(np.int32) if permute else np.arange(D, dtype=np.int32)
    sub = perm.reshape(C, L)  # columns of codebook c's subspace

    A = draw_A(spec, N, rA)

    if spec.thr_dist == "sorted_per_dim":
        if L != 1:
            raise ValueError("sorted_per_dim needs one dim per codebook")
        split = np.repeat(sub[:, :1], LEVELS, axis=1).astype(np.int32)
        s = np.sort(rT.standard_normal((C, NODES), dtype=np.float32), axis=1)
        thr = heap_from_sorted(s)
    else:
        pick = rT.integers(0, L, size=(C, LEVELS))
        split = np.take_along_axis(sub, pick, axis=1).astype(np.int32)
        thr = rT.standard_normal((C, NODES), dtype=np.float32)
        if spec.thr_dist == "halfnormal":
            thr = np.abs(thr)

    P = np.zeros((C, K, D), dtype=np.float32)
    if spec.p_dist == "bin_midpoints":
        # codebook c's 16 prototypes sit at the midpoints of the 16 bins cut by
        # its sorted thresholds (outer bins: half a unit beyond the extremes)
        srt = np.sort(thr, axis=1)
        lo = np.concatenate([srt[:, :1] - 1.0, srt], axis=1)
        hi = np.concatenate([srt, srt[:, -1:] + 1.0], axis=1)
        mid = ((lo + hi) * 0.5).astype(np.float32)
        for c in range(C):
            P[c, :, sub[c, 0]] = mid[c]
    else:
        vals = rP.standard_normal((C, K, L), dtype=np.float32)
        if spec.p_dist == "halfnormal":
            vals = np.abs(vals)
        for c in range(C):
            P[c][:, sub[c]] = vals[c]

    B = (rB.standard_normal((D, M), dtype=np.float32) * np.float32(spec.b_std)).astype(np.float32)
    return Problem(spec, N, A, split, thr, P, B, perm)


def random_codes(C: int, M: int, seed: int, max_shift: int, extreme: bool = False):
    """An int8 block-FP table drawn directly (not from P B): codes uniform in
    [-127, 127] (all +-127 when `extreme`), scales 2^e with e - min(e) drawn in
    [0, max_shift], offsets N(0, 1).  The caller picks max_shift so that the
    int32 sum cannot overflow."""
    rng = np.random.default_rng(seed)
    if extreme:
        lut = np.where(rng.random((C, K, M)) < 0.5, -127, 127).astype(np.int8)
    else:
        lut = rng.integers(-127, 128, size=(C, K, M)).astype(np.int8)
    e0 = int(rng.integers(-20, 5))
    sh = rng.integers(0, max_shift + 1, size=C)
    if C > 0:
        sh[rng.integers(0, C)] = 0
    scale = np.ldexp(np.float32(1.0), (e0 + sh).astype(np.int32)).astype(np.float32)
    offset = rng.standard_normal(C).astype(np.float32)
    return lut, scale, offset


def random_fp32_table(C: int, M: int, seed: int, std: float = 1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((C, K, M), dtype=np.float32) * np.float32(std)).astype(np.float32)


def random_indices(N: int, C: int, seed: int):
    rng = np.random.default_rng(seed)
    return rng.integers(0, K, size=(N, C)).astype(np.uint8)
