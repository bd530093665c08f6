"""Plain CPU oracle for the encode + lookup-accumulate path (numpy in, numpy out).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product package.  The arithmetic
lives in ``maddness_oracle.c`` (plain C, double precision where the method
leaves precision open); this module only marshals arrays through ctypes.

Functions and the passages they follow (the paper: McCarter & Dronen,
"Look-ups are not (yet) all you need for deep learning inference"):

* :func:`encode` -- §1 (encoding function, log2(K)-bit indices) and §2.1
  (one comparison per tree level, four levels, K = 16 leaves).
* :func:`lut_accumulate` -- §1 (sum of the table rows picked per codebook;
  8-bit block floating point tables).
* :func:`lut_accumulate_f32` -- same sum over an unquantized fp32 table.
* :func:`build_table` -- §2.2 (T = P B).
* :func:`quantize_table` -- §1 (8-bit block floating point), reading R6.
* :func:`sigma` -- §2.2 (layer output: bias, then ReLU or row softmax), R19.
* :func:`lut_accumulate_avg`, :func:`quantize_table_shared` -- §1 (rounded
  8-bit summation over codebooks, one shared block exponent), reading R20.
* :func:`encoder_gram`, :func:`encoder_scatter`, :func:`fit_lut_ridge` --
  §2.2, Eq. 3 (model-aware table fit) with sigma affine, reading R21.
* :func:`fit_lut_gd` -- Eq. 3 with sigma = ReLU (squared error) or softmax
  (KL divergence, the alternative §3.1 uses for classifiers, or the squared
  error of Eq. 3 itself), gradient descent, reading R22.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "maddness_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-fPIC", "-shared", "-Wall", "-Wextra"]

K = 16
LEVELS = 4
NODES = 15


def build(out: str = _LIB, extra_flags=()) -> str:
    """Compile the oracle with gcc into ``out`` (always recompiles)."""
    cmd = ["gcc", *CFLAGS, *extra_flags, _SRC, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class OracleError(RuntimeError):
    pass


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class Oracle:
    """ctypes view of one compiled oracle library (the default one, or a test build)."""

    def __init__(self, path: str = _LIB):
        if not os.path.exists(path):
            build(path)
        self.path = path
        lib = ctypes.CDLL(path)
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        vp = ctypes.c_void_p
        lib.oracle_encode.argtypes = [vp, i64, i32, i64, vp, vp, i32, vp]
        lib.oracle_lut_accumulate.argtypes = [vp, i64, i32, vp, vp, vp, i32, vp, vp]
        lib.oracle_lut_accumulate_f32.argtypes = [vp, i64, i32, vp, i32, vp]
        lib.oracle_build_table.argtypes = [vp, vp, i32, i32, i32, vp]
        lib.oracle_quantize_table.argtypes = [vp, i32, i32, vp, vp, vp]
        lib.oracle_round_table_f32.argtypes = [vp, i64, vp]
        lib.oracle_dequant_params.argtypes = [vp, vp, i32, vp, vp, vp]
        lib.oracle_exponent_cap.argtypes = [i32]
        lib.oracle_block_exponent.argtypes = [ctypes.c_float, vp]
        lib.oracle_sigma.argtypes = [vp, i64, i32, vp, i32, vp]
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        lib.oracle_quantize_table_shared.argtypes = [vp, i32, i32, vp, vp, vp]
        lib.oracle_lut_accumulate_avg.argtypes = [vp, i64, i32, vp, vp, vp, i32, vp, vp]
        lib.oracle_encoder_gram.argtypes = [vp, i64, i32, vp]
        lib.oracle_encoder_scatter.argtypes = [vp, i64, i32, vp, i32, vp]
        lib.oracle_fit_lut_ridge.argtypes = [vp, i64, i32, vp, i32, vp, ctypes.c_double, vp]
        lib.oracle_fit_lut_gd.argtypes = [vp, i64, i32, vp, i32, vp, i32, vp, ctypes.c_double, ctypes.c_double,
                                          i32, vp]
        self.lib = lib

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise OracleError(f"{what} failed with code {rc}")

    def max_threads(self) -> int:
        return int(self.lib.oracle_max_threads())

    def set_threads(self, n: int) -> None:
        """Host threads the row loops use from now on (timing only)."""
        self.lib.oracle_set_threads(int(n))

    def encode(self, A, split, thr):
        A = np.asarray(A, dtype=np.float32)
        assert A.ndim == 2
        if A.shape[0] > 0 and (A.strides[1] != 4 or A.strides[0] % 4 or A.strides[0] < 4 * A.shape[1]):
            A = np.ascontiguousarray(A)
        N, D = A.shape
        lda = A.strides[0] // 4 if N > 0 else D
        split = np.ascontiguousarray(split, dtype=np.int32)
        thr = np.ascontiguousarray(thr, dtype=np.float32)
        C = split.shape[0]
        assert split.shape == (C, LEVELS) and thr.shape == (C, NODES)
        idx = np.zeros((N, C), dtype=np.uint8)
        rc = self.lib.oracle_encode(A.ctypes.data, N, D, lda, split.ctypes.data,
                                    thr.ctypes.data, C, idx.ctypes.data)
        self._check(rc, "oracle_encode")
        return idx

    def lut_accumulate(self, idx, lut, scale, offset, want_acc=True, want_y=True):
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        lut = np.ascontiguousarray(lut, dtype=np.int8)
        scale = np.ascontiguousarray(scale, dtype=np.float32)
        offset = np.ascontiguousarray(offset, dtype=np.float32)
        N, C = idx.shape
        assert lut.shape[:2] == (C, K)
        M = lut.shape[2]
        acc = np.zeros((N, M), dtype=np.int32) if want_acc else None
        y = np.zeros((N, M), dtype=np.float32) if want_y else None
        rc = self.lib.oracle_lut_accumulate(
            idx.ctypes.data, N, C, lut.ctypes.data, scale.ctypes.data, offset.ctypes.data, M,
            acc.ctypes.data if acc is not None else None,
            y.ctypes.data if y is not None else None)
        self._check(rc, "oracle_lut_accumulate")
        return acc, y

    def lut_accumulate_f32(self, idx, lut):
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        lut = np.ascontiguousarray(lut, dtype=np.float32)
        N, C = idx.shape
        assert lut.shape[:2] == (C, K)
        M = lut.shape[2]
        y = np.zeros((N, M), dtype=np.float32)
        rc = self.lib.oracle_lut_accumulate_f32(idx.ctypes.data, N, C, lut.ctypes.data, M,
                                                y.ctypes.data)
        self._check(rc, "oracle_lut_accumulate_f32")
        return y

    def build_table(self, P, B):
        P = np.ascontiguousarray(P, dtype=np.float32)
        B = np.ascontiguousarray(B, dtype=np.float32)
        C, k, D = P.shape
        assert k == K and B.shape[0] == D
        M = B.shape[1]
        T = np.zeros((C, K, M), dtype=np.float64)
        rc = self.lib.oracle_build_table(P.ctypes.data, B.ctypes.data, C, D, M, T.ctypes.data)
        self._check(rc, "oracle_build_table")
        return T

    def quantize_table(self, T):
        T = np.ascontiguousarray(T, dtype=np.float64)
        C, k, M = T.shape
        assert k == K
        lut = np.zeros((C, K, M), dtype=np.int8)
        scale = np.zeros(C, dtype=np.float32)
        offset = np.zeros(C, dtype=np.float32)
        rc = self.lib.oracle_quantize_table(T.ctypes.data, C, M, lut.ctypes.data,
                                            scale.ctypes.data, offset.ctypes.data)
        self._check(rc, "oracle_quantize_table")
        return lut, scale, offset

    def quantize_table_shared(self, T):
        """The quantizer with one block exponent shared by all codebooks (R20)."""
        T = np.ascontiguousarray(T, dtype=np.float64)
        C, k, M = T.shape
        assert k == K
        lut = np.zeros((C, K, M), dtype=np.int8)
        scale = np.zeros(C, dtype=np.float32)
        offset = np.zeros(C, dtype=np.float32)
        rc = self.lib.oracle_quantize_table_shared(T.ctypes.data, C, M, lut.ctypes.data,
                                                   scale.ctypes.data, offset.ctypes.data)
        self._check(rc, "oracle_quantize_table_shared")
        return lut, scale, offset

    def lut_accumulate_avg(self, idx, lut, scale, offset):
        """Rounded 8-bit averaging accumulate (R20); returns (acc int32, y fp32)."""
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        lut = np.ascontiguousarray(lut, dtype=np.int8)
        scale = np.ascontiguousarray(scale, dtype=np.float32)
        offset = np.ascontiguousarray(offset, dtype=np.float32)
        N, C = idx.shape
        assert lut.shape[:2] == (C, K)
        M = lut.shape[2]
        acc = np.zeros((N, M), dtype=np.int32)
        y = np.zeros((N, M), dtype=np.float32)
        rc = self.lib.oracle_lut_accumulate_avg(idx.ctypes.data, N, C, lut.ctypes.data, scale.ctypes.data,
                                                offset.ctypes.data, M, acc.ctypes.data, y.ctypes.data)
        self._check(rc, "oracle_lut_accumulate_avg")
        return acc, y

    def round_table_f32(self, T):
        T = np.ascontiguousarray(T, dtype=np.float64)
        out = np.zeros(T.shape, dtype=np.float32)
        rc = self.lib.oracle_round_table_f32(T.ctypes.data, T.size, out.ctypes.data)
        self._check(rc, "oracle_round_table_f32")
        return out

    def dequant_params(self, scale, offset):
        scale = np.ascontiguousarray(scale, dtype=np.float32)
        offset = np.ascontiguousarray(offset, dtype=np.float32)
        C = scale.shape[0]
        sh = np.zeros(C, dtype=np.int32)
        emin = np.zeros(1, dtype=np.int32)
        bias = np.zeros(1, dtype=np.float32)
        rc = self.lib.oracle_dequant_params(scale.ctypes.data, offset.ctypes.data, C,
                                            sh.ctypes.data, emin.ctypes.data, bias.ctypes.data)
        self._check(rc, "oracle_dequant_params")
        return sh, int(emin[0]), np.float32(bias[0])

    def exponent_cap(self, C: int) -> int:
        return int(self.lib.oracle_exponent_cap(C))

    def block_exponent(self, s: float):
        e = np.zeros(1, dtype=np.int32)
        rc = self.lib.oracle_block_exponent(ctypes.c_float(s), e.ctypes.data)
        return None if rc != 0 else int(e[0])

    def sigma(self, y, bias=None, act=0):
        """Layer output sigma: 0 none, 1 bias, 2 bias + ReLU, 3 bias + row softmax
        (float64 [N, M])."""
        y = np.ascontiguousarray(y, dtype=np.float32)
        N, M = y.shape
        out = np.zeros((N, M), dtype=np.float64)
        bp = None
        if bias is not None:
            bias = np.ascontiguousarray(bias, dtype=np.float32)
            if bias.shape != (M,):
                raise OracleError("bias must be [M]")
            bp = bias.ctypes.data
        rc = self.lib.oracle_sigma(y.ctypes.data, N, M, bp, int(act), out.ctypes.data)
        self._check(rc, "oracle_sigma")
        return out

    def encoder_gram(self, idx):
        """H = G^T G of the one-hot encoder output, int64 [16C, 16C] (Eq. 3, R21)."""
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        N, C = idx.shape
        H = np.zeros((C * K, C * K), dtype=np.int64)
        self._check(self.lib.oracle_encoder_gram(idx.ctypes.data, N, C, H.ctypes.data), "oracle_encoder_gram")
        return H

    def encoder_scatter(self, idx, Y):
        """R = G^T Y, float64 [16C, M] (Eq. 3, R21)."""
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        Y = np.ascontiguousarray(Y, dtype=np.float32)
        N, C = idx.shape
        assert Y.shape[0] == N
        M = Y.shape[1]
        R = np.zeros((C * K, M), dtype=np.float64)
        rc = self.lib.oracle_encoder_scatter(idx.ctypes.data, N, C, Y.ctypes.data, M, R.ctypes.data)
        self._check(rc, "oracle_encoder_scatter")
        return R

    def fit_lut_ridge(self, idx, Y, T0, lam):
        """Eq. 3 with sigma affine (R21): the table T minimising
        ||Y - G T||^2 + lam ||T - T0||^2, float64 [C, 16, M]."""
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        Y = np.ascontiguousarray(Y, dtype=np.float32)
        T0 = np.ascontiguousarray(T0, dtype=np.float32)
        N, C = idx.shape
        M = Y.shape[1]
        assert Y.shape[0] == N and T0.shape == (C, K, M)
        T = np.zeros((C, K, M), dtype=np.float64)
        rc = self.lib.oracle_fit_lut_ridge(idx.ctypes.data, N, C, Y.ctypes.data, M, T0.ctypes.data,
                                           ctypes.c_double(lam), T.ctypes.data)
        self._check(rc, "oracle_fit_lut_ridge")
        return T

    def fit_lut_gd(self, idx, Y, T0, act, lam, eta, iters, bias=None):
        """Eq. 3 with a nonlinear sigma (R22): act 2 = ReLU + squared error,
        3 = softmax + KL divergence, 4 = softmax + squared error; gradient
        descent from T0.  float64 [C, 16, M]."""
        idx = np.ascontiguousarray(idx, dtype=np.uint8)
        Y = np.ascontiguousarray(Y, dtype=np.float32)
        T0 = np.ascontiguousarray(T0, dtype=np.float32)
        N, C = idx.shape
        M = Y.shape[1]
        assert Y.shape[0] == N and T0.shape == (C, K, M)
        bp = None
        if bias is not None:
            bias = np.ascontiguousarray(bias, dtype=np.float32)
            assert bias.shape == (M,)
            bp = bias.ctypes.data
        T = np.zeros((C, K, M), dtype=np.float64)
        rc = self.lib.oracle_fit_lut_gd(idx.ctypes.data, N, C, Y.ctypes.data, M, bp, int(act), T0.ctypes.data,
                                        ctypes.c_double(lam), ctypes.c_double(eta), int(iters), T.ctypes.data)
        self._check(rc, "oracle_fit_lut_gd")
        return T

    # convenience compositions (no arithmetic of their own)
    def matmul(self, A, split, thr, lut, scale, offset):
        idx = self.encode(A, split, thr)
        acc, y = self.lut_accumulate(idx, lut, scale, offset)
        return idx, acc, y

    def matmul_f32(self, A, split, thr, lut_f32):
        idx = self.encode(A, split, thr)
        return idx, self.lut_accumulate_f32(idx, lut_f32)

    def build_quantized_lut(self, P, B):
        return self.quantize_table(self.build_table(P, B))

    def build_shared_lut(self, P, B):
        return self.quantize_table_shared(self.build_table(P, B))

    def build_lut_f32(self, P, B):
        return self.round_table_f32(self.build_table(P, B))


_default = None


def get() -> Oracle:
    """The default build, or the library MADDNESS_ORACLE_LIB names (a
    sanitizer build of the same source, for the tests)."""
    global _default
    if _default is None:
        _default = Oracle(os.environ.get("MADDNESS_ORACLE_LIB", _LIB))
    return _default
