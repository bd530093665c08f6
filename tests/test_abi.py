"""The C ABI on the host: the library loads, exports every symbol that
include/maddness.h declares, and rejects bad arguments before any HIP call
(so these checks need no GPU and launch nothing)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "maddness.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(maddness_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    from paper_2207_05808_amd import _lib
    return _lib.lib()


def test_header_declares_the_path():
    names = declared_functions()
    for need in ("maddness_encode", "maddness_lut_accumulate", "maddness_matmul",
                 "maddness_lut_accumulate_f32", "maddness_matmul_f32", "maddness_build_lut"):
        assert need in names


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), f"{name} declared but not exported"


def test_status_strings(L):
    assert L.maddness_version() >= 100
    for s in range(5):
        assert L.maddness_status_string(s)
    assert L.maddness_status_string(99) == b"unknown status"


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first
NULL = None


def test_encode_rejects(L):
    E = L.maddness_encode
    assert E(FAKE, -1, 64, 64, FAKE, FAKE, 4, FAKE, NULL) == 1      # N < 0
    assert E(FAKE, 10, 0, 64, FAKE, FAKE, 4, FAKE, NULL) == 1       # D <= 0
    assert E(FAKE, 10, 64, 63, FAKE, FAKE, 4, FAKE, NULL) == 1      # lda < D
    assert E(FAKE, 10, 64, 64, FAKE, FAKE, 0, FAKE, NULL) == 1      # C <= 0
    assert E(NULL, 10, 64, 64, FAKE, FAKE, 4, FAKE, NULL) == 1      # NULL A
    assert E(FAKE, 10, 64, 64, NULL, FAKE, 4, FAKE, NULL) == 1      # NULL split
    assert E(FAKE, 10, 64, 64, FAKE, FAKE, 4, NULL, NULL) == 1      # NULL out
    assert E(ctypes.c_void_p(0x1002), 10, 64, 64, FAKE, FAKE, 4, FAKE, NULL) == 1  # misaligned A
    assert E(FAKE, 10, 64, 64, FAKE, FAKE, 513, FAKE, NULL) == 3    # too many codebooks
    assert E(NULL, 0, 64, 64, NULL, NULL, 4, NULL, NULL) == 0       # N == 0: nothing to do


def test_accumulate_rejects(L):
    A = L.maddness_lut_accumulate
    assert A(FAKE, 10, 4, FAKE, FAKE, FAKE, 10, NULL, NULL, NULL) == 1   # both outputs NULL
    assert A(FAKE, 10, 4, FAKE, FAKE, FAKE, 0, FAKE, FAKE, NULL) == 1    # M <= 0
    assert A(FAKE, 10, 4, NULL, FAKE, FAKE, 10, FAKE, FAKE, NULL) == 1   # NULL lut
    assert A(FAKE, 10, 4, FAKE, NULL, FAKE, 10, FAKE, FAKE, NULL) == 1   # NULL scale
    assert A(FAKE, 10, 4, FAKE, FAKE, ctypes.c_void_p(0x1001), 10, FAKE, FAKE, NULL) == 1
    assert A(FAKE, 10, 600, FAKE, FAKE, FAKE, 10, FAKE, FAKE, NULL) == 3
    assert A(NULL, 0, 4, NULL, NULL, NULL, 10, NULL, NULL, NULL) == 0
    F = L.maddness_lut_accumulate_f32
    assert F(FAKE, 10, 4, FAKE, 10, NULL, NULL) == 1
    assert F(FAKE, -5, 4, FAKE, 10, FAKE, NULL) == 1


def test_matmul_rejects(L):
    Mm = L.maddness_matmul
    args = [FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, FAKE, FAKE, 10, FAKE, NULL, NULL, NULL]
    bad = list(args); bad[11] = NULL          # y_out required
    assert Mm(*bad) == 1
    bad = list(args); bad[3] = 10             # lda < D
    assert Mm(*bad) == 1
    bad = list(args); bad[10] = -1            # M
    assert Mm(*bad) == 1
    F = L.maddness_matmul_f32
    assert F(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, 10, NULL, NULL, NULL) == 1


def test_matmul_index_bytes(L):
    """The fused entry points use a caller index array when their own
    single-launch kernels cannot take the table, or when encode + the one-hot
    product beats the row-streaming kernel: 0 for the im2col conv layer
    (C = 32, M = 64) and the tiny classifier; N * C for the dense hidden layer
    (C = 64, M = 512; without an index array it still runs, as one launch of
    the row-streaming kernel, from 98304 rows on), its shape below that, the
    wide layer and the fp32 search-tree layer; 0 again for 64 output columns
    (the row-streaming kernel alone)."""
    Q = L.maddness_matmul_index_bytes
    assert Q(FAKE, 131072, 576, 576, 32, 64, 0, 0) == 0
    assert Q(FAKE, 131072, 576, 576, 32, 64, 0, 3) == 0
    assert Q(FAKE, 1024, 64, 64, 4, 10, 0, 3) == 0
    assert Q(FAKE, 1 << 20, 512, 512, 64, 512, 0, 0) == (1 << 20) * 64
    assert Q(FAKE, 1 << 20, 512, 512, 64, 512, 0, 2) == (1 << 20) * 64
    assert Q(FAKE, 1 << 20, 512, 512, 64, 512, 0, 3) == 0   # a row softmax: the row-streaming kernel fuses it
    assert Q(FAKE, 98304, 512, 512, 64, 512, 0, 0) == 98304 * 64
    assert Q(FAKE, 1 << 20, 512, 512, 64, 64, 0, 0) == 0
    assert Q(FAKE, 98303, 512, 512, 64, 512, 0, 0) == 98303 * 64
    assert Q(FAKE, 1 << 20, 512, 512, 64, 520, 0, 0) == (1 << 20) * 64     # M % 16 != 0
    assert Q(FAKE, 1 << 20, 512, 512, 64, 512, 1, 0) == (1 << 20) * 64     # fp32 table
    assert Q(FAKE, 262144, 1024, 1024, 128, 4096, 0, 2) == 262144 * 128
    assert Q(FAKE, 524288, 256, 256, 256, 1024, 1, 0) == 524288 * 256
    assert Q(NULL, 0, 512, 512, 64, 512, 0, 0) == 0          # N == 0: nothing to do
    assert Q(FAKE, -1, 64, 64, 4, 10, 0, 0) == -1
    assert Q(FAKE, 10, 64, 63, 4, 10, 0, 0) == -1             # lda < D
    assert Q(FAKE, 10, 64, 64, 4, 10, 0, 4) == -1             # act outside 0..3
    assert Q(ctypes.c_void_p(0x1002), 10, 64, 64, 4, 10, 0, 0) == -1   # misaligned A
    assert Q(FAKE, 10, 64, 64, 600, 10, 0, 0) == -3           # too many codebooks


def test_fused_two_phase_needs_index_array(L):
    """Without idx_out a call whose table does not fit the single-launch
    kernels is rejected (EINVAL) before any HIP call: the library never
    allocates."""
    big = [FAKE, 4096, 512, 512, FAKE, FAKE, 64, FAKE, FAKE, FAKE, 512, FAKE, NULL, NULL, NULL]
    assert L.maddness_matmul(*big) == 1
    assert L.maddness_matmul_f32(FAKE, 4096, 256, 256, FAKE, FAKE, 256, FAKE, 1024, FAKE, NULL, NULL) == 1
    assert L.maddness_matmul_act(FAKE, 4096, 512, 512, FAKE, FAKE, 64, FAKE, FAKE, FAKE, 512, NULL, 2, FAKE,
                                 NULL, NULL) == 1
    assert L.maddness_matmul_act_f32(FAKE, 4096, 256, 256, FAKE, FAKE, 256, FAKE, 1024, NULL, 3, FAKE,
                                     NULL, NULL) == 1


def test_library_imports_no_allocator():
    """No device (or host-pinned) allocation routine is referenced by the
    library: every buffer beyond the inputs and outputs is the caller's."""
    import shutil
    import subprocess
    from paper_2207_05808_amd import _lib
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--undefined-only", _lib.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    syms = [l.split()[-1].split("@")[0] for l in out.splitlines() if l.strip()]
    alloc = [s for s in syms if re.match(r"hip(Ext)?(Malloc|Free|HostMalloc|HostAlloc|MallocManaged|"
                                         r"MallocAsync|FreeAsync|MallocFromPool|MemPool|HostRegister)", s)]
    assert not alloc, f"allocation routines referenced: {alloc}"


def test_matmul_act_rejects(L):
    Ma = L.maddness_matmul_act
    args = [FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, FAKE, FAKE, 10, NULL, 2, FAKE, NULL, NULL]
    for bad_act in (-1, 4):
        bad = list(args); bad[12] = bad_act
        assert Ma(*bad) == 1
    bad = list(args); bad[11] = ctypes.c_void_p(0x1002)   # misaligned bias
    assert Ma(*bad) == 1
    bad = list(args); bad[13] = NULL                      # y_out required
    assert Ma(*bad) == 1
    bad = list(args); bad[6] = 600                        # too many codebooks
    assert Ma(*bad) == 3
    zero = list(args); zero[1] = 0                        # N == 0
    assert Ma(*zero) == 0
    F = L.maddness_matmul_act_f32
    assert F(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, 10, NULL, 7, FAKE, NULL, NULL) == 1
    assert F(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, 10, NULL, 3, NULL, NULL, NULL) == 1


def test_accumulate_avg_rejects(L):
    A = L.maddness_lut_accumulate_avg
    assert A(FAKE, 10, 4, FAKE, FAKE, FAKE, 10, NULL, NULL, NULL) == 1   # both outputs NULL
    assert A(FAKE, 10, 4, FAKE, NULL, FAKE, 10, FAKE, FAKE, NULL) == 1   # NULL scale
    assert A(FAKE, 10, 600, FAKE, FAKE, FAKE, 10, FAKE, FAKE, NULL) == 3
    assert A(NULL, 0, 4, NULL, NULL, NULL, 10, NULL, NULL, NULL) == 0
    S = L.maddness_build_lut_shared
    assert S(FAKE, FAKE, 0, 64, 10, FAKE, FAKE, FAKE, NULL) == 1
    assert S(FAKE, FAKE, 600, 64, 10, FAKE, FAKE, FAKE, NULL) == 3


def test_build_lut_rejects(L):
    B = L.maddness_build_lut
    assert B(FAKE, FAKE, 0, 64, 10, FAKE, FAKE, FAKE, NULL) == 1
    assert B(FAKE, FAKE, 4, 64, 10, NULL, FAKE, FAKE, NULL) == 1
    assert B(FAKE, FAKE, 140000, 64, 10, FAKE, FAKE, FAKE, NULL) == 1  # 127 C >= 2^24
    assert L.maddness_build_lut_f32(FAKE, FAKE, 4, 0, 10, FAKE, NULL) == 1


def test_fit_entry_points_reject(L):
    Q = L.maddness_quantize_lut
    assert Q(FAKE, 0, 10, 0, FAKE, FAKE, FAKE, NULL) == 1
    assert Q(NULL, 4, 10, 0, FAKE, FAKE, FAKE, NULL) == 1
    assert Q(ctypes.c_void_p(0x1004), 4, 10, 0, FAKE, FAKE, FAKE, NULL) == 1   # T not 8-byte aligned
    assert Q(FAKE, 600, 10, 1, FAKE, FAKE, FAKE, NULL) == 3
    G = L.maddness_encoder_gram
    assert G(FAKE, -1, 4, FAKE, NULL) == 1
    assert G(FAKE, 10, 4, NULL, NULL) == 1
    assert G(FAKE, 10, 300, FAKE, NULL) == 3
    assert G(FAKE, 1 << 31, 4, FAKE, NULL) == 3
    S = L.maddness_encoder_scatter
    SW = L.maddness_encoder_scatter_workspace_bytes
    assert SW(10, 0) == -1 and SW(-1, 4) == -1 and SW(1 << 31, 4) == -1
    assert SW(10, 4) == 2304 + 4 * 17 * 4   # 4 lists of 10 + 128 rows (2208 bytes, rounded to 256), bucket starts
    sw = SW(10, 4)
    assert S(FAKE, 10, 4, FAKE, 0, FAKE, FAKE, sw, NULL) == 1
    assert S(FAKE, 10, 4, NULL, 8, FAKE, FAKE, sw, NULL) == 1
    assert S(FAKE, 10, 4, FAKE, 8, FAKE, FAKE, sw - 1, NULL) == 1   # workspace too small
    assert S(FAKE, 10, 4, FAKE, 8, FAKE, NULL, sw, NULL) == 1
    assert S(FAKE, 10, 300, FAKE, 8, FAKE, FAKE, 1 << 40, NULL) == 3
    W = L.maddness_fit_lut_workspace_bytes
    assert W(10, 0) == -1 and W(10, 257) == -1
    assert W(10, 4) == 64 * 64 * 4 + 64 * 64 * 8 + SW(10, 4)
    F = L.maddness_fit_lut_ridge
    ws = W(10, 4)
    assert F(FAKE, 10, 4, FAKE, 8, FAKE, 0.0, FAKE, FAKE, ws, NULL) == 1            # lambda = 0
    assert F(FAKE, 10, 4, FAKE, 8, FAKE, float("nan"), FAKE, FAKE, ws, NULL) == 1   # lambda NaN
    assert F(FAKE, 10, 4, FAKE, 8, FAKE, float("inf"), FAKE, FAKE, ws, NULL) == 1
    assert F(FAKE, 10, 4, FAKE, 8, FAKE, 1.0, FAKE, FAKE, ws - 1, NULL) == 1        # workspace too small
    assert F(FAKE, 10, 4, FAKE, 8, FAKE, 1.0, FAKE, ctypes.c_void_p(0x1010), ws, NULL) == 1   # not 256-aligned
    assert F(FAKE, 10, 4, FAKE, 8, NULL, 1.0, FAKE, FAKE, ws, NULL) == 1            # NULL T0
    assert F(FAKE, 10, 300, FAKE, 8, FAKE, 1.0, FAKE, FAKE, 1 << 40, NULL) == 3


def test_fit_gd_rejects(L):
    W = L.maddness_fit_lut_gd_workspace_bytes
    assert W(10, 0, 5) == -1 and W(10, 4, 0) == -1 and W(10, 300, 5) == -1
    ws = W(10, 4, 5)
    assert ws > 0
    G = L.maddness_fit_lut_gd
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 1, FAKE, 0.1, 0.01, 3, FAKE, FAKE, ws, NULL) == 1   # act 1
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 5, FAKE, 0.1, 0.01, 3, FAKE, FAKE, ws, NULL) == 1   # objective 5
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 4, FAKE, -0.1, 0.01, 3, FAKE, FAKE, ws, NULL) == 1  # objective 4, lambda < 0
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 3, FAKE, -0.1, 0.01, 3, FAKE, FAKE, ws, NULL) == 1  # lambda < 0
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 3, FAKE, 0.1, 0.0, 3, FAKE, FAKE, ws, NULL) == 1    # eta = 0
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 2, FAKE, 0.1, 0.01, -1, FAKE, FAKE, ws, NULL) == 1  # iters < 0
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 2, FAKE, 0.1, float("inf"), 3, FAKE, FAKE, ws, NULL) == 1
    assert G(FAKE, 10, 4, FAKE, 5, NULL, 2, FAKE, 0.1, 0.01, 3, FAKE, FAKE, ws - 1, NULL) == 1
    assert G(FAKE, 10, 300, FAKE, 5, NULL, 2, FAKE, 0.1, 0.01, 3, FAKE, FAKE, 1 << 40, NULL) == 3


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU is present: valid-looking calls would launch kernels")
def test_no_device_gives_ehip(L):
    """On a machine without a GPU, calls whose arguments pass validation fail
    in the HIP runtime and return EHIP (2) instead of crashing."""
    assert L.maddness_encode(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, NULL) == 2
    assert L.maddness_lut_accumulate(FAKE, 10, 4, FAKE, FAKE, FAKE, 10, NULL, FAKE, NULL) == 2
    assert L.maddness_lut_accumulate_f32(FAKE, 10, 4, FAKE, 12, FAKE, NULL) == 2
    assert L.maddness_matmul(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, FAKE, FAKE, 10, FAKE, NULL, NULL, NULL) == 2
    assert L.maddness_matmul_f32(FAKE, 10, 64, 64, FAKE, FAKE, 4, FAKE, 12, FAKE, NULL, NULL) == 2
    # the dense hidden layer without an index array is not rejected: it takes
    # the row-streaming kernel (one launch)
    assert L.maddness_matmul(FAKE, 1 << 20, 512, 512, FAKE, FAKE, 64, FAKE, FAKE, FAKE, 512, FAKE, NULL, NULL,
                             NULL) == 2
