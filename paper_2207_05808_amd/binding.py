"""Torch-tensor front end of the C ABI (same names as include/maddness.h).

Each function checks dtypes, devices and shapes, allocates outputs that were
not supplied, and passes raw device pointers plus the current HIP stream to
the library.  No arithmetic of the method happens here.

With ``validate=True`` the device-array preconditions of the ABI (split
columns in range, indices below 16, scales exact powers of two, no int32
overflow) are checked on host copies first; this synchronises and is meant
for tests and debugging.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Tuple

import torch

from . import _lib

K, LEVELS, NODES = 16, 4, 15


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")


def _dense(t: torch.Tensor, name: str):
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _rows(A: torch.Tensor) -> Tuple[int, int, int]:
    _need(A, "A", torch.float32, 2)
    if A.shape[0] > 1 and A.stride(1) != 1:
        raise ValueError("A must have unit column stride")
    N, D = A.shape
    lda = A.stride(0) if N > 1 else D
    return N, D, lda


def _tree_args(split: torch.Tensor, thr: torch.Tensor) -> int:
    _need(split, "split_dims", torch.int32, 2)
    _need(thr, "thresholds", torch.float32, 2)
    _dense(split, "split_dims")
    _dense(thr, "thresholds")
    C = split.shape[0]
    if tuple(split.shape) != (C, LEVELS) or tuple(thr.shape) != (C, NODES):
        raise ValueError(f"split_dims must be [C,4] and thresholds [C,15], got "
                         f"{tuple(split.shape)} and {tuple(thr.shape)}")
    return C


def _validate_trees(split: torch.Tensor, D: int):
    s = split.cpu()
    if s.numel() and (int(s.min()) < 0 or int(s.max()) >= D):
        raise ValueError("split_dims outside [0, D)")


def _validate_scales(scale: torch.Tensor):
    s = scale.cpu().numpy()
    import numpy as np
    m, e = np.frexp(s)
    if not (np.all(m == 0.5) and np.all(e - 1 >= -126)):
        raise ValueError("scales must be exact normal powers of two")
    sh = (e - 1) - (e - 1).min()
    if np.any(sh > 30) or float(np.sum(128.0 * np.ldexp(1.0, sh))) > 2.0 ** 31:
        raise ValueError("scale exponents too far apart: a sum of int8 codes could leave int32")


def _validate_idx(idx: torch.Tensor):
    if idx.numel() and int(idx.max()) >= K:
        raise ValueError("indices must lie in [0, 16)")


def encode(A, split_dims, thresholds, idx_out=None, stream=None, validate=False):
    """Tree encoding: returns idx [N][C] uint8 (see maddness_encode)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    if validate:
        _validate_trees(split_dims, D)
    if idx_out is None:
        idx_out = torch.empty((N, C), dtype=torch.uint8, device=A.device)
    _need(idx_out, "idx_out", torch.uint8, 2)
    _dense(idx_out, "idx_out")
    st = _lib.lib().maddness_encode(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C,
                                    _ptr(idx_out), _stream(stream))
    _lib.check("maddness_encode", st)
    return idx_out


def _lut_i8(lut, scale, offset):
    _need(lut, "lut", torch.int8, 3)
    _need(scale, "scale", torch.float32, 1)
    _need(offset, "offset", torch.float32, 1)
    for t, n in ((lut, "lut"), (scale, "scale"), (offset, "offset")):
        _dense(t, n)
    C, k, M = lut.shape
    if k != K or scale.shape[0] != C or offset.shape[0] != C:
        raise ValueError("lut must be [C,16,M], scale and offset [C]")
    return C, M


def lut_accumulate(idx, lut, scale, offset, acc_out=None, y_out=None, want_acc=False, want_y=True,
                   stream=None, validate=False):
    """Gather-accumulate over an int8 block-FP table; returns (acc or None, y or None)."""
    _need(idx, "idx", torch.uint8, 2)
    _dense(idx, "idx")
    C, M = _lut_i8(lut, scale, offset)
    N = idx.shape[0]
    if idx.shape[1] != C:
        raise ValueError("idx must be [N, C]")
    if validate:
        _validate_idx(idx)
        _validate_scales(scale)
    if acc_out is None and want_acc:
        acc_out = torch.empty((N, M), dtype=torch.int32, device=idx.device)
    if y_out is None and want_y:
        y_out = torch.empty((N, M), dtype=torch.float32, device=idx.device)
    st = _lib.lib().maddness_lut_accumulate(_ptr(idx), N, C, _ptr(lut), _ptr(scale), _ptr(offset), M,
                                            _ptr(acc_out), _ptr(y_out), _stream(stream))
    _lib.check("maddness_lut_accumulate", st)
    return acc_out, y_out


def lut_accumulate_avg(idx, lut, scale, offset, acc_out=None, y_out=None, want_acc=False, want_y=True,
                       stream=None, validate=False):
    """Rounded 8-bit summation over codebooks (approximate; one shared scale);
    returns (acc or None, y or None)."""
    _need(idx, "idx", torch.uint8, 2)
    _dense(idx, "idx")
    C, M = _lut_i8(lut, scale, offset)
    N = idx.shape[0]
    if idx.shape[1] != C:
        raise ValueError("idx must be [N, C]")
    if validate:
        _validate_idx(idx)
        _validate_scales(scale)
        if not bool((scale == scale[0]).all()):
            raise ValueError("the averaging accumulate needs one scale shared by every codebook")
    if acc_out is None and want_acc:
        acc_out = torch.empty((N, M), dtype=torch.int32, device=idx.device)
    if y_out is None and want_y:
        y_out = torch.empty((N, M), dtype=torch.float32, device=idx.device)
    st = _lib.lib().maddness_lut_accumulate_avg(_ptr(idx), N, C, _ptr(lut), _ptr(scale), _ptr(offset), M,
                                                _ptr(acc_out), _ptr(y_out), _stream(stream))
    _lib.check("maddness_lut_accumulate_avg", st)
    return acc_out, y_out


def lut_accumulate_f32(idx, lut, y_out=None, stream=None, validate=False):
    """Gather-accumulate over an fp32 table [C][16][M]; returns y [N][M]."""
    _need(idx, "idx", torch.uint8, 2)
    _need(lut, "lut", torch.float32, 3)
    _dense(idx, "idx")
    _dense(lut, "lut")
    C, k, M = lut.shape
    N = idx.shape[0]
    if k != K or idx.shape[1] != C:
        raise ValueError("lut must be [C,16,M] and idx [N,C]")
    if validate:
        _validate_idx(idx)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=idx.device)
    st = _lib.lib().maddness_lut_accumulate_f32(_ptr(idx), N, C, _ptr(lut), M, _ptr(y_out),
                                                _stream(stream))
    _lib.check("maddness_lut_accumulate_f32", st)
    return y_out


def matmul(A, split_dims, thresholds, lut, scale, offset, y_out=None, acc_out=None, idx_out=None,
           want_acc=False, want_idx=False, stream=None, validate=False):
    """Fused encode + int8 lookup-accumulate; returns (y, acc or None, idx or None)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    C2, M = _lut_i8(lut, scale, offset)
    if C2 != C:
        raise ValueError("lut codebooks differ from the trees'")
    if validate:
        _validate_trees(split_dims, D)
        _validate_scales(scale)
    dev = A.device
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=dev)
    if acc_out is None and want_acc:
        acc_out = torch.empty((N, M), dtype=torch.int32, device=dev)
    if idx_out is None and want_idx:
        idx_out = torch.empty((N, C), dtype=torch.uint8, device=dev)
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, False, 0, stream)
    st = _lib.lib().maddness_matmul(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C,
                                    _ptr(lut), _ptr(scale), _ptr(offset), M, _ptr(y_out),
                                    _ptr(acc_out), _ptr(idx_arg), _stream(stream))
    _lib.check("maddness_matmul", st)
    return y_out, acc_out, idx_out


def matmul_noalloc(A, split_dims, thresholds, lut, scale, offset, y_out, acc_out=None, idx_out=None,
                   stream=None):
    """maddness_matmul_noalloc: the fused int8 path with every buffer given
    by the caller (y_out required) and, for large tables without idx_out,
    the library's static scratch array in place of an index array; neither
    this function nor the library allocates.  Returns y_out."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    C2, M = _lut_i8(lut, scale, offset)
    if C2 != C:
        raise ValueError("lut codebooks differ from the trees'")
    _need(y_out, "y_out", torch.float32, 2)
    _dense(y_out, "y_out")
    if tuple(y_out.shape) != (N, M):
        raise ValueError("y_out must be [N, M]")
    if acc_out is not None:
        _need(acc_out, "acc_out", torch.int32, 2)
        _dense(acc_out, "acc_out")
        if tuple(acc_out.shape) != (N, M):
            raise ValueError("acc_out must be [N, M]")
    idx_out = _idx_out(idx_out, N, C)
    st = _lib.lib().maddness_matmul_noalloc(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C,
                                            _ptr(lut), _ptr(scale), _ptr(offset), M, _ptr(y_out),
                                            _ptr(acc_out), _ptr(idx_out), _stream(stream))
    _lib.check("maddness_matmul_noalloc", st)
    return y_out


def matmul_f32(A, split_dims, thresholds, lut, y_out=None, idx_out=None, want_idx=False, stream=None,
               validate=False):
    """Fused encode + fp32 lookup-accumulate; returns (y, idx or None)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    _need(lut, "lut", torch.float32, 3)
    _dense(lut, "lut")
    if lut.shape[0] != C or lut.shape[1] != K:
        raise ValueError("lut must be [C,16,M]")
    M = lut.shape[2]
    if validate:
        _validate_trees(split_dims, D)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=A.device)
    if idx_out is None and want_idx:
        idx_out = torch.empty((N, C), dtype=torch.uint8, device=A.device)
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, True, 0, stream)
    st = _lib.lib().maddness_matmul_f32(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C,
                                        _ptr(lut), M, _ptr(y_out), _ptr(idx_arg), _stream(stream))
    _lib.check("maddness_matmul_f32", st)
    return y_out, idx_out


ACT = {"none": 0, "bias": 1, "relu": 2, "softmax": 3}
# objectives of fit_lut_gd (MADDNESS_FIT_*): the layer output and the loss
FIT = {"relu": 2, "softmax": 3, "softmax_kld": 3, "softmax_sqerr": 4}


def _act(act):
    if isinstance(act, str):
        if act not in ACT:
            raise ValueError(f"act must be one of {sorted(ACT)}")
        return ACT[act]
    return int(act)


def _col_bias(col_bias, M):
    if col_bias is None:
        return None
    _need(col_bias, "col_bias", torch.float32, 1)
    _dense(col_bias, "col_bias")
    if col_bias.shape[0] != M:
        raise ValueError("col_bias must be [M]")
    return col_bias


def _idx_out(idx_out, N, C):
    if idx_out is not None:
        _need(idx_out, "idx_out", torch.uint8, 2)
        _dense(idx_out, "idx_out")
        if tuple(idx_out.shape) != (N, C):
            raise ValueError("idx_out must be [N, C]")
    return idx_out


def matmul_index_bytes(A, C, M, f32=False, act=0) -> int:
    """Device bytes of idx_out the fused entry points use for this A and
    shape (maddness_matmul_index_bytes): 0 when the call runs as one launch,
    else N * C (the two-phase path; for the shapes that also have a slower
    one-launch route, the faster one through the index array)."""
    N, D, lda = _rows(A)
    n = int(_lib.lib().maddness_matmul_index_bytes(_ptr(A), N, D, lda, C, M, 1 if f32 else 0, _act(act)))
    if n < 0:
        _lib.check("maddness_matmul_index_bytes", _lib.EINVAL if n == -1 else _lib.EUNSUPPORTED)
    return n


def _index_array(idx_out, A, N, D, lda, C, M, f32, act, stream):
    """idx_out when the caller gave one; else, when the call uses an index
    array (the table does not fit the single-launch kernels, or two phases
    through it are faster), a new one from torch's allocator, kept alive for
    `stream`; else None.  The library itself never allocates."""
    if idx_out is not None:
        return idx_out
    n = int(_lib.lib().maddness_matmul_index_bytes(_ptr(A), N, D, lda, C, M, 1 if f32 else 0, int(act)))
    if n <= 0:
        return None   # one launch, or arguments the call itself rejects
    t = torch.empty((N, C), dtype=torch.uint8, device=A.device)
    if stream is not None:
        t.record_stream(stream)
    return t


def matmul_act(A, split_dims, thresholds, lut, scale, offset, col_bias=None, act="relu", y_out=None,
               idx_out=None, stream=None, validate=False):
    """Fused encode + lookup-accumulate + layer output sigma (bias, then
    "relu" / "softmax"; "bias" or "none" also accepted); returns y.  With
    idx_out the indices are written there; without it an index array is
    allocated here when the shape needs one (matmul_index_bytes)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    C2, M = _lut_i8(lut, scale, offset)
    if C2 != C:
        raise ValueError("lut codebooks differ from the trees'")
    col_bias = _col_bias(col_bias, M)
    if validate:
        _validate_trees(split_dims, D)
        _validate_scales(scale)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=A.device)
    _need(y_out, "y_out", torch.float32, 2)
    _dense(y_out, "y_out")
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, False, _act(act), stream)
    st = _lib.lib().maddness_matmul_act(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C, _ptr(lut),
                                        _ptr(scale), _ptr(offset), M, _ptr(col_bias), _act(act), _ptr(y_out),
                                        _ptr(idx_arg), _stream(stream))
    _lib.check("maddness_matmul_act", st)
    return y_out


def matmul_act_f32(A, split_dims, thresholds, lut, col_bias=None, act="relu", y_out=None, idx_out=None,
                   stream=None, validate=False):
    """matmul_act over an unquantized fp32 table; returns y."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    _need(lut, "lut", torch.float32, 3)
    _dense(lut, "lut")
    if lut.shape[0] != C or lut.shape[1] != K:
        raise ValueError("lut must be [C,16,M]")
    M = lut.shape[2]
    col_bias = _col_bias(col_bias, M)
    if validate:
        _validate_trees(split_dims, D)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=A.device)
    _need(y_out, "y_out", torch.float32, 2)
    _dense(y_out, "y_out")
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, True, _act(act), stream)
    st = _lib.lib().maddness_matmul_act_f32(_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C,
                                            _ptr(lut), M, _ptr(col_bias), _act(act), _ptr(y_out),
                                            _ptr(idx_arg), _stream(stream))
    _lib.check("maddness_matmul_act_f32", st)
    return y_out


def build_lut(P, B, stream=None):
    """Table T = P B, 8-bit block-FP quantized; returns (lut int8 [C,16,M], scale [C], offset [C])."""
    _need(P, "P", torch.float32, 3)
    _need(B, "B", torch.float32, 2)
    _dense(P, "P")
    _dense(B, "B")
    C, k, D = P.shape
    if k != K or B.shape[0] != D:
        raise ValueError("P must be [C,16,D] and B [D,M]")
    M = B.shape[1]
    lut = torch.empty((C, K, M), dtype=torch.int8, device=P.device)
    scale = torch.empty((C,), dtype=torch.float32, device=P.device)
    offset = torch.empty((C,), dtype=torch.float32, device=P.device)
    st = _lib.lib().maddness_build_lut(_ptr(P), _ptr(B), C, D, M, _ptr(lut), _ptr(scale),
                                       _ptr(offset), _stream(stream))
    _lib.check("maddness_build_lut", st)
    return lut, scale, offset


def build_lut_shared(P, B, stream=None):
    """build_lut with one block exponent shared by every codebook (for lut_accumulate_avg)."""
    _need(P, "P", torch.float32, 3)
    _need(B, "B", torch.float32, 2)
    _dense(P, "P")
    _dense(B, "B")
    C, k, D = P.shape
    if k != K or B.shape[0] != D:
        raise ValueError("P must be [C,16,D] and B [D,M]")
    M = B.shape[1]
    lut = torch.empty((C, K, M), dtype=torch.int8, device=P.device)
    scale = torch.empty((C,), dtype=torch.float32, device=P.device)
    offset = torch.empty((C,), dtype=torch.float32, device=P.device)
    st = _lib.lib().maddness_build_lut_shared(_ptr(P), _ptr(B), C, D, M, _ptr(lut), _ptr(scale),
                                              _ptr(offset), _stream(stream))
    _lib.check("maddness_build_lut_shared", st)
    return lut, scale, offset


def build_lut_f32(P, B, stream=None):
    """Table T = P B rounded to fp32; returns lut [C,16,M]."""
    _need(P, "P", torch.float32, 3)
    _need(B, "B", torch.float32, 2)
    _dense(P, "P")
    _dense(B, "B")
    C, k, D = P.shape
    if k != K or B.shape[0] != D:
        raise ValueError("P must be [C,16,D] and B [D,M]")
    M = B.shape[1]
    lut = torch.empty((C, K, M), dtype=torch.float32, device=P.device)
    st = _lib.lib().maddness_build_lut_f32(_ptr(P), _ptr(B), C, D, M, _ptr(lut), _stream(stream))
    _lib.check("maddness_build_lut_f32", st)
    return lut


def version() -> int:
    return int(_lib.lib().maddness_version())


class PreparedCall:
    """One C-ABI call with its arguments validated and marshalled once.

    Calling the object issues the same launch again on the stream captured
    when it was prepared (no checks, no allocation, no Python-side work
    beyond the ctypes call), for serving loops and benchmarks.  The tensors
    it was prepared with must stay alive and keep their storage.
    """

    def __init__(self, name, args, keep, outputs):
        self._fn = getattr(_lib.lib(), name)
        self._name = name
        self._args = args
        self._keep = keep          # tensors whose storage the pointers refer to
        self.outputs = outputs

    def __call__(self):
        st = self._fn(*self._args)
        if st:
            _lib.check(self._name, st)
        return self.outputs


def prepare_matmul_f32(A, split_dims, thresholds, lut, y_out=None, idx_out=None, stream=None, validate=False):
    """Prepared maddness_matmul_f32; ``call()`` returns (y, idx or None)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    _need(lut, "lut", torch.float32, 3)
    _dense(lut, "lut")
    C2, M = lut.shape[0], lut.shape[2]
    if lut.shape[1] != K:
        raise ValueError("lut must be [C,16,M]")
    if C2 != C:
        raise ValueError("lut codebooks differ from the trees'")
    if validate:
        _validate_trees(split_dims, D)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=A.device)
    _need(y_out, "y_out", torch.float32, 2)
    _dense(y_out, "y_out")
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, True, 0, stream)
    args = (_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C, _ptr(lut), M, _ptr(y_out),
            _ptr(idx_arg), _stream(stream))
    keep = (A, split_dims, thresholds, lut, y_out, idx_arg)
    return PreparedCall("maddness_matmul_f32", args, keep, (y_out, idx_out))


def prepare_matmul(A, split_dims, thresholds, lut, scale, offset, y_out=None, acc_out=None,
                   idx_out=None, stream=None, validate=False):
    """Prepared maddness_matmul; ``call()`` returns (y, acc or None, idx or None)."""
    N, D, lda = _rows(A)
    C = _tree_args(split_dims, thresholds)
    C2, M = _lut_i8(lut, scale, offset)
    if C2 != C:
        raise ValueError("lut codebooks differ from the trees'")
    if validate:
        _validate_trees(split_dims, D)
        _validate_scales(scale)
    if y_out is None:
        y_out = torch.empty((N, M), dtype=torch.float32, device=A.device)
    _need(y_out, "y_out", torch.float32, 2)
    _dense(y_out, "y_out")
    idx_out = _idx_out(idx_out, N, C)
    idx_arg = _index_array(idx_out, A, N, D, lda, C, M, False, 0, stream)
    args = (_ptr(A), N, D, lda, _ptr(split_dims), _ptr(thresholds), C, _ptr(lut), _ptr(scale),
            _ptr(offset), M, _ptr(y_out), _ptr(acc_out), _ptr(idx_arg), _stream(stream))
    keep = (A, split_dims, thresholds, lut, scale, offset, y_out, acc_out, idx_arg)
    return PreparedCall("maddness_matmul", args, keep, (y_out, acc_out, idx_out))


def quantize_lut(T, shared=False, stream=None):
    """8-bit block floating point quantization of a given float64 table
    [C,16,M] (e.g. a fitted one); returns (lut, scale, offset)."""
    _need(T, "T", torch.float64, 3)
    _dense(T, "T")
    C, k, M = T.shape
    if k != K:
        raise ValueError("T must be [C,16,M]")
    lut = torch.empty((C, K, M), dtype=torch.int8, device=T.device)
    scale = torch.empty((C,), dtype=torch.float32, device=T.device)
    offset = torch.empty((C,), dtype=torch.float32, device=T.device)
    st = _lib.lib().maddness_quantize_lut(_ptr(T), C, M, 1 if shared else 0, _ptr(lut), _ptr(scale), _ptr(offset),
                                          _stream(stream))
    _lib.check("maddness_quantize_lut", st)
    return lut, scale, offset


def _fit_inputs(idx, Y):
    _need(idx, "idx", torch.uint8, 2)
    _dense(idx, "idx")
    _need(Y, "Y", torch.float32, 2)
    _dense(Y, "Y")
    if Y.shape[0] != idx.shape[0]:
        raise ValueError("Y must have one row per index row")
    return idx.shape[0], idx.shape[1], Y.shape[1]


def encoder_gram(idx, stream=None):
    """H = G^T G of the one-hot encoder output: int32 [16C, 16C] counts."""
    _need(idx, "idx", torch.uint8, 2)
    _dense(idx, "idx")
    N, C = idx.shape
    H = torch.empty((C * K, C * K), dtype=torch.int32, device=idx.device)
    st = _lib.lib().maddness_encoder_gram(_ptr(idx), N, C, _ptr(H), _stream(stream))
    _lib.check("maddness_encoder_gram", st)
    return H


def _workspace(workspace, need, device, stream):
    """A 256-byte aligned pointer into ``workspace`` (allocated when None)."""
    if workspace is None:
        workspace = torch.empty((need + 256,), dtype=torch.uint8, device=device)
        if stream is not None:
            workspace.record_stream(stream)   # freed only after the work queued on `stream`
    base = workspace.data_ptr()
    off = (-base) % 256
    if workspace.numel() - off < need:
        raise ValueError(f"workspace must hold {need} bytes at a 256-byte aligned address")
    return workspace, ctypes.c_void_p(base + off)


def encoder_scatter(idx, Y, workspace=None, stream=None):
    """R = G^T Y: float64 [16C, M], each entry summed over its rows in order."""
    N, C, M = _fit_inputs(idx, Y)
    need = int(_lib.lib().maddness_encoder_scatter_workspace_bytes(N, C))
    if need < 0:
        _lib.check("maddness_encoder_scatter", _lib.EUNSUPPORTED)
    workspace, wp = _workspace(workspace, need, idx.device, stream)
    R = torch.empty((C * K, M), dtype=torch.float64, device=idx.device)
    st = _lib.lib().maddness_encoder_scatter(_ptr(idx), N, C, _ptr(Y), M, _ptr(R), wp, need, _stream(stream))
    _lib.check("maddness_encoder_scatter", st)
    return R


def fit_lut_ridge(idx, Y, T0, lam, workspace=None, stream=None):
    """Model-aware table fit (Eq. 3, affine output): the float64 table
    [C,16,M] minimising ||Y - G T||^2 + lam ||T - T0||^2.  ``workspace``: an
    optional preallocated uint8 device tensor of at least
    fit_lut_workspace_bytes(N, C) bytes (+ up to 255 for alignment)."""
    N, C, M = _fit_inputs(idx, Y)
    _need(T0, "T0", torch.float32, 3)
    _dense(T0, "T0")
    if tuple(T0.shape) != (C, K, M):
        raise ValueError("T0 must be [C,16,M]")
    need = int(_lib.lib().maddness_fit_lut_workspace_bytes(N, C))
    if need < 0:
        _lib.check("maddness_fit_lut_ridge", _lib.EUNSUPPORTED)
    workspace, wp = _workspace(workspace, need, idx.device, stream)
    T = torch.empty((C, K, M), dtype=torch.float64, device=idx.device)
    st = _lib.lib().maddness_fit_lut_ridge(_ptr(idx), N, C, _ptr(Y), M, _ptr(T0), float(lam), _ptr(T),
                                           wp, need, _stream(stream))
    _lib.check("maddness_fit_lut_ridge", st)
    return T


def fit_lut_workspace_bytes(N: int, C: int) -> int:
    """Device bytes fit_lut_ridge needs as workspace for N training rows and C codebooks."""
    n = int(_lib.lib().maddness_fit_lut_workspace_bytes(N, C))
    if n < 0:
        _lib.check("maddness_fit_lut_workspace_bytes", _lib.EUNSUPPORTED)
    return n


def fit_lut_gd(idx, Y, T0, act, lam, eta, iters, col_bias=None, workspace=None, stream=None):
    """Model-aware table fit (Eq. 3) with a nonlinear output by gradient
    descent from T0: act "relu" (squared error after bias + ReLU),
    "softmax" / "softmax_kld" (KL divergence between row softmaxes) or
    "softmax_sqerr" (squared error between row softmaxes); float64 [C,16,M]."""
    N, C, M = _fit_inputs(idx, Y)
    _need(T0, "T0", torch.float32, 3)
    _dense(T0, "T0")
    if tuple(T0.shape) != (C, K, M):
        raise ValueError("T0 must be [C,16,M]")
    if isinstance(act, str) and act not in FIT:
        raise ValueError(f"act must be one of {sorted(FIT)}")
    code = FIT[act] if isinstance(act, str) else int(act)
    if col_bias is not None:
        _need(col_bias, "col_bias", torch.float32, 1)
        _dense(col_bias, "col_bias")
        if col_bias.shape[0] != M:
            raise ValueError("col_bias must be [M]")
    need = int(_lib.lib().maddness_fit_lut_gd_workspace_bytes(N, C, M))
    if need < 0:
        _lib.check("maddness_fit_lut_gd", _lib.EUNSUPPORTED)
    workspace, wp = _workspace(workspace, need, idx.device, stream)
    T = torch.empty((C, K, M), dtype=torch.float64, device=idx.device)
    st = _lib.lib().maddness_fit_lut_gd(_ptr(idx), N, C, _ptr(Y), M, _ptr(col_bias), int(code), _ptr(T0), float(lam),
                                        float(eta), int(iters), _ptr(T), wp, need, _stream(stream))
    _lib.check("maddness_fit_lut_gd", st)
    return T


def fit_lut_gd_workspace_bytes(N: int, C: int, M: int) -> int:
    """Device bytes fit_lut_gd needs as workspace."""
    n = int(_lib.lib().maddness_fit_lut_gd_workspace_bytes(N, C, M))
    if n < 0:
        _lib.check("maddness_fit_lut_gd_workspace_bytes", _lib.EUNSUPPORTED)
    return n
