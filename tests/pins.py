"""Checks that pin the CPU oracle to facts other than itself.

Each check takes an oracle object (the default build, or a build with a
planted mistake) and raises AssertionError when the oracle disagrees with
what the paper or the mathematics fixes.  The expected values come from
independent computations: brute-force enumeration, a textbook binary search,
a one-hot dense integer product, exact rational arithmetic (fractions), a
correctly rounded sum (math.fsum), or a hand-worked example in tests/golden.
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np

K, LEVELS, NODES = 16, 4, 15
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U32 = 2.0 ** -24
U64 = 2.0 ** -53


def gamma(n, u):
    return n * u / (1 - n * u)


# ------------------------------------------------------------------ encode
def brute_force_leaf(A, split, thr):
    """For every (row, codebook) test all 16 leaves against the path
    predicate: leaf k is reached iff, at every level t, the comparison of
    A[n, split[c,t]] with the threshold of the node on k's path (node number
    k >> (4 - t) within level t) gives bit 3 - t of k.  Returns the unique
    leaf, asserting that exactly one leaf satisfies the predicate."""
    N, C = A.shape[0], split.shape[0]
    ok = np.ones((N, C, K), dtype=bool)
    for k in range(K):
        for t in range(LEVELS):
            node = (1 << t) - 1 + (k >> (LEVELS - t))
            bit = (k >> (LEVELS - 1 - t)) & 1
            x = A[:, split[:, t]]                       # [N, C]
            v = thr[np.arange(C), node][None, :]        # [1, C]
            ok[:, :, k] &= ((x > v) == bool(bit))
    count = ok.sum(axis=2)
    assert np.all(count == 1), "leaf predicate not satisfied by exactly one leaf"
    return ok.argmax(axis=2).astype(np.uint8)


def bst_heap(sorted15):
    """Breadth-first listing of the balanced binary search tree over 15 sorted
    values (root = median, recursively): the heap layout of a search tree."""
    out, queue = [], [(0, 15)]
    while queue:
        lo, hi = queue.pop(0)
        mid = (lo + hi) // 2
        out.append(sorted15[mid])
        if hi - lo > 1:
            queue.append((lo, mid))
            queue.append((mid + 1, hi))
    assert len(out) == 15
    return np.array(out, dtype=np.float32)


def check_encode_brute_force(orc, seed=0):
    rng = np.random.default_rng(seed)
    for (N, D, C) in [(300, 64, 4), (200, 576, 32), (150, 7, 9), (64, 1, 3)]:
        A = rng.standard_normal((N, D), dtype=np.float32)
        split = rng.integers(0, D, size=(C, LEVELS)).astype(np.int32)
        thr = rng.standard_normal((C, NODES), dtype=np.float32)
        # a share of exact ties with the compared thresholds
        for n in range(0, N, 5):
            c = n % C
            A[n, split[c, 0]] = thr[c, 0]
        idx = orc.encode(A, split, thr)
        assert idx.shape == (N, C) and idx.dtype == np.uint8
        assert int(idx.max()) < K, "index outside [0, 16)"
        assert np.array_equal(idx, brute_force_leaf(A, split, thr)), "encode != brute force"
        # the same rows inside a wider array (row stride > D)
        wide = np.zeros((N, D + 3), dtype=np.float32)
        wide[:, :D] = A
        wide[:, D:] = np.nan
        assert np.array_equal(orc.encode(wide[:, :D], split, thr), idx), "row stride ignored"


def check_encode_search_tree(orc, seed=1):
    """One column per codebook, all levels on it, thresholds of a binary search
    tree: the leaf is the number of thresholds strictly below x, i.e.
    numpy.searchsorted(s, x, side='left'), ties going left."""
    rng = np.random.default_rng(seed)
    C, N = 6, 4000
    s = np.sort(rng.standard_normal((C, NODES), dtype=np.float32), axis=1)
    s[0] = np.arange(-7, 8, dtype=np.float32)            # integer grid: exact ties
    s[1, 7] = 0.0                                          # a zero threshold (against +-0 inputs)
    s = np.sort(s, axis=1)
    thr = np.stack([bst_heap(s[c]) for c in range(C)])
    split = np.repeat(np.arange(C, dtype=np.int32)[:, None], LEVELS, axis=1)
    A = rng.standard_normal((N, C), dtype=np.float32) * 2
    A[::3, 0] = rng.integers(-8, 9, size=A[::3, 0].shape).astype(np.float32)
    A[1::9, 1] = -0.0
    A[2::9, 1] = 0.0
    A[3::17, :] = np.inf
    A[4::17, :] = -np.inf
    idx = orc.encode(A, split, thr)
    for c in range(C):
        ref = np.searchsorted(s[c], A[:, c], side="left")
        assert np.array_equal(idx[:, c], ref), f"codebook {c}: encode != searchsorted"


def check_encode_nan(orc):
    """Comparisons with NaN are false: a NaN input takes the 0 branch at every level."""
    D, C = 8, 3
    split = np.array([[0, 1, 2, 3], [4, 4, 4, 4], [7, 6, 5, 0]], dtype=np.int32)
    thr = np.full((C, NODES), -1e30, dtype=np.float32)      # every finite value goes right
    A = np.zeros((4, D), dtype=np.float32)
    A[1, :] = np.nan
    A[2, 4] = np.nan
    idx = orc.encode(A, split, thr)
    assert idx[0].tolist() == [15, 15, 15]
    assert idx[1].tolist() == [0, 0, 0]
    assert idx[2].tolist() == [15, 0, 15]


def check_encode_permutation(orc, seed=2):
    """Permuting the columns of A together with the split columns leaves the
    indices unchanged (split columns are global indices)."""
    rng = np.random.default_rng(seed)
    N, D, C = 500, 40, 5
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = rng.integers(0, D, size=(C, LEVELS)).astype(np.int32)
    thr = rng.standard_normal((C, NODES), dtype=np.float32)
    perm = rng.permutation(D)
    inv = np.argsort(perm)
    A2 = A[:, perm]                         # column j of A2 is column perm[j] of A
    split2 = inv[split].astype(np.int32)    # so old column d is now at inv[d]
    assert np.array_equal(orc.encode(A, split, thr), orc.encode(A2, split2, thr))


def load_golden_tree_walk():
    """tests/golden/tree_walk_tiny.txt: a hand-worked encoding example."""
    path = os.path.join(GOLDEN, "tree_walk_tiny.txt")
    sections, cur = {}, None
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if line.startswith("[") and line.endswith("]"):
                cur = line[1:-1]
                sections[cur] = []
            else:
                sections[cur].append([float(v) for v in line.split()])
    split = np.array(sections["split"], dtype=np.int32)
    thr = np.array(sections["thresholds"], dtype=np.float32)
    A = np.array(sections["rows"], dtype=np.float32)
    idx = np.array(sections["expected_idx"], dtype=np.uint8)
    return A, split, thr, idx


def check_encode_golden(orc):
    A, split, thr, idx = load_golden_tree_walk()
    assert np.array_equal(orc.encode(A, split, thr), idx), "hand-worked tree walks differ"


# -------------------------------------------------------------- accumulate
def one_hot(idx):
    N, C = idx.shape
    G = np.zeros((N, C * K), dtype=np.int64)
    G[np.arange(N)[:, None], np.arange(C)[None, :] * K + idx.astype(np.int64)] = 1
    return G


def exponents(scale):
    m, e = np.frexp(scale.astype(np.float64))
    assert np.all(m == 0.5)
    return (e - 1).astype(np.int64)


def check_one_hot_identity(orc, seed=3):
    """The lookup sum equals the dense product of the one-hot encoder output G
    (N x 16C) with the stacked, shifted code table (16C x M), in int64."""
    rng = np.random.default_rng(seed)
    for (N, C, M, maxsh) in [(200, 4, 10, 3), (100, 32, 64, 5), (64, 7, 3, 10), (50, 1, 1, 0)]:
        idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
        lut = rng.integers(-127, 128, size=(C, K, M)).astype(np.int8)
        e = rng.integers(-3, -3 + maxsh + 1, size=C)
        scale = np.ldexp(np.float32(1), e.astype(np.int32)).astype(np.float32)
        offset = rng.standard_normal(C).astype(np.float32)
        acc, _ = orc.lut_accumulate(idx, lut, scale, offset)
        ex = exponents(scale)
        Q = (lut.astype(np.int64) * (2 ** (ex - ex.min()))[:, None, None]).reshape(C * K, M)
        assert np.array_equal(acc.astype(np.int64), one_hot(idx) @ Q), "acc != one-hot product"


def check_decoder_table(orc, seed=4):
    """With M = C and q[c][k][m] = k if m == c else 0 (equal scales), the sum
    reads back the indices: acc[n][m] == idx[n][m]."""
    rng = np.random.default_rng(seed)
    N, C = 300, 9
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    lut = np.zeros((C, K, C), dtype=np.int8)
    for c in range(C):
        lut[c, :, c] = np.arange(K)
    acc, _ = orc.lut_accumulate(idx, lut, np.ones(C, np.float32), np.zeros(C, np.float32))
    assert np.array_equal(acc, idx.astype(np.int32)), "decoder table does not read back indices"


def rne32(x: Fraction) -> float:
    """Round an exact rational to the nearest fp32 (ties to even), finite range."""
    if x == 0:
        return 0.0
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                        # subnormal spacing below 2^-126
    ulp = Fraction(2) ** (e - 23)
    q, r = divmod(a, ulp)
    q = int(q)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return sign * float(q * ulp)


def check_output_rounding(orc, seed=5):
    """y is the dequantized sum rounded once: with offsets whose double sum is
    exact (integers), y == RNE32(acc 2^e_min + RNE32(sum o)) computed in exact
    rationals, and |y - sum_c (2^e_c q_c + o_c)| obeys the closed-form bound."""
    rng = np.random.default_rng(seed)
    N, C, M = 60, 12, 9
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    lut = rng.integers(-127, 128, size=(C, K, M)).astype(np.int8)
    e = rng.integers(-9, -5, size=C)
    scale = np.ldexp(np.float32(1), e.astype(np.int32)).astype(np.float32)
    offset = rng.integers(-2 ** 20, 2 ** 20, size=C).astype(np.float32)
    acc, y = orc.lut_accumulate(idx, lut, scale, offset)
    S = sum(Fraction(float(o)) for o in offset)
    bias = rne32(S)
    emin = int(e.min())
    for n in range(N):
        for m in range(M):
            exact = sum(Fraction(float(scale[c])) * int(lut[c, idx[n, c], m]) for c in range(C))
            assert Fraction(int(acc[n, m])) * Fraction(2) ** emin == exact, "acc scaling wrong"
            want = rne32(exact + Fraction(bias))
            assert float(y[n, m]) == want, f"y[{n},{m}] not the single rounding of its value"
            deq = exact + S
            bound = U32 * abs(float(y[n, m])) + abs(float(Fraction(bias) - S))
            assert abs(float(Fraction(float(y[n, m])) - deq)) <= bound * (1 + 1e-12)
    # offsets of mixed magnitude: bias32 within the rounding bound of the exact sum
    offset2 = (rng.standard_normal(C) * 10.0 ** rng.integers(-6, 6, size=C)).astype(np.float32)
    _, _, b2 = orc.dequant_params(scale, offset2)
    S2 = sum(Fraction(float(o)) for o in offset2)
    tol = U32 * abs(float(S2)) + gamma(C, U64) * float(np.abs(offset2.astype(np.float64)).sum())
    assert abs(float(Fraction(float(b2)) - S2)) <= tol * (1 + 1e-12)


def check_scale_linearity(orc, seed=6):
    """Doubling every scale doubles acc * 2^e_min exactly (acc itself unchanged);
    shifting one codebook's exponent by +1 doubles its share of acc."""
    rng = np.random.default_rng(seed)
    N, C, M = 100, 5, 8
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    lut = rng.integers(-127, 128, size=(C, K, M)).astype(np.int8)
    scale = np.ldexp(np.float32(1), rng.integers(-4, 0, size=C).astype(np.int32)).astype(np.float32)
    off = np.zeros(C, np.float32)
    a1, y1 = orc.lut_accumulate(idx, lut, scale, off)
    a2, y2 = orc.lut_accumulate(idx, lut, scale * 2, off)
    assert np.array_equal(a1, a2) and np.array_equal(y2, y1 * 2)
    one = np.zeros((C, K, M), np.int8)
    one[2] = lut[2]
    b1, _ = orc.lut_accumulate(idx, one, scale, off)
    s3 = scale.copy()
    s3[2] *= 2
    b2, _ = orc.lut_accumulate(idx, one, s3, off)
    ex = exponents(scale)
    ex3 = exponents(s3)
    # codebook 2's contribution in units of each call's own 2^e_min
    assert np.array_equal(b2.astype(np.int64) * 2 ** int(ex3.min()),
                          2 * b1.astype(np.int64) * 2 ** int(ex.min()))


def check_f32_order(orc):
    """fp32 tables are summed in codebook order from +0: ((0 + 1e8) + 1) - 1e8
    is 0 in fp32, while other orders give 1."""
    lut = np.zeros((3, K, 1), np.float32)
    lut[0, :, 0] = 1e8
    lut[1, :, 0] = 1.0
    lut[2, :, 0] = -1e8
    y = orc.lut_accumulate_f32(np.zeros((1, 3), np.uint8), lut)
    assert y[0, 0] == 0.0
    lut2 = lut[[0, 2, 1]]
    assert orc.lut_accumulate_f32(np.zeros((1, 3), np.uint8), lut2)[0, 0] == 1.0


def exact_table(P, B):
    """T = P B entry by entry with math.fsum (correctly rounded double)."""
    C, _, D = P.shape
    M = B.shape[1]
    T = np.zeros((C, K, M))
    Pd, Bd = P.astype(np.float64), B.astype(np.float64)
    for c in range(C):
        for k in range(K):
            for m in range(M):
                T[c, k, m] = math.fsum(Pd[c, k] * Bd[:, m])
    return T


def check_table_build(orc, seed=7):
    """T = P B: exact for integer data; within gamma_D sum |P B| otherwise."""
    rng = np.random.default_rng(seed)
    C, D, M = 3, 12, 5
    Pi = rng.integers(-50, 50, size=(C, K, D)).astype(np.float32)
    Bi = rng.integers(-50, 50, size=(D, M)).astype(np.float32)
    T = orc.build_table(Pi, Bi)
    assert np.array_equal(T, np.einsum("ckd,dm->ckm", Pi.astype(np.int64), Bi.astype(np.int64)))
    P = rng.standard_normal((C, K, D), dtype=np.float32)
    B = rng.standard_normal((D, M), dtype=np.float32)
    T = orc.build_table(P, B)
    ref = exact_table(P, B)
    bnd = gamma(D, U64) * np.einsum("ckd,dm->ckm", np.abs(P.astype(np.float64)), np.abs(B.astype(np.float64)))
    assert np.all(np.abs(T - ref) <= bnd + 1e-300)


def check_quantizer(orc, seed=8):
    """Block floating point codes: power-of-two scales, |q| <= 127, every
    dequantized entry within half a step of T, the smallest exponent that fits
    (unless raised to the common floor), and the int32 sum exact in fp32."""
    rng = np.random.default_rng(seed)
    C, M = 6, 11
    T = rng.standard_normal((C, K, M)) * (10.0 ** np.arange(C))[:, None, None]
    T[3] = 0.25                                   # a constant codebook
    lut, scale, offset = orc.quantize_table(T)
    ex = exponents(scale)
    cap = orc.exponent_cap(C)
    assert 127 * C * 2 ** cap < 2 ** 24 <= 127 * C * 2 ** (cap + 1)
    assert int(ex.max() - ex.min()) <= cap
    assert np.all(np.abs(lut.astype(np.int64)) <= 127)
    deq = scale.astype(np.float64)[:, None, None] * lut + offset.astype(np.float64)[:, None, None]
    assert np.all(np.abs(deq - T) <= scale.astype(np.float64)[:, None, None] / 2 * (1 + 1e-12))
    assert np.all(lut[3] == 0) and offset[3] == np.float32(0.25)
    floor_e = int(ex.max()) - cap
    for c in range(C):
        if ex[c] > floor_e and c != 3:
            r = np.abs(T[c] - np.float64(offset[c])).max()
            assert r > 127 * 2.0 ** (ex[c] - 1), f"codebook {c}: exponent not minimal"
        lo, hi = T[c].min(), T[c].max()
        assert offset[c] == np.float32((lo + hi) / 2)


def rne32_or_inf(x: Fraction) -> float:
    """rne32 extended past the top binade: a value that rounds to 2^128 or
    beyond (at or above FLT_MAX + half an ulp, ties to even) is infinite."""
    r = rne32(x)
    return math.copysign(math.inf, r) if abs(r) >= 2.0 ** 128 else r


def check_round_table_f32(orc, seed=23):
    """Unquantized tables: every double entry is rounded to the nearest fp32,
    ties to even (R10's table), checked bit for bit against exact rational
    rounding on random doubles of every magnitude, exact halfway cases
    (even and odd neighbours), the top of the range (FLT_MAX, the halfway
    point above it, overflow to infinity), subnormals and signed zeros."""
    rng = np.random.default_rng(seed)
    vals = list(rng.standard_normal(400) * 10.0 ** rng.integers(-30, 30, size=400))
    vals += list(rng.standard_normal(100) * 2.0 ** -140)               # subnormal results
    for _ in range(200):                                                 # exact halfway cases
        f = float(np.float32(rng.standard_normal() * 10.0 ** int(rng.integers(-20, 20))))
        ulp = float(np.spacing(np.float32(abs(f))))
        vals.append(f + math.copysign(ulp / 2, f))
        vals.append(-(abs(f) + ulp / 2))
    fmax = float(np.finfo(np.float32).max)
    top = 2.0 ** 104                                                     # ulp of the top binade
    vals += [fmax, -fmax, fmax + top / 4, fmax + top / 2, -(fmax + top / 2), fmax * 1.5, 1e300,
             2.0 ** -149, 2.0 ** -150, 3 * 2.0 ** -151, 2.0 ** -151, 2.0 ** -126 - 2.0 ** -150,
             0.0, -0.0, 1.0, -1.0, 1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24]
    T = np.array(vals, np.float64)
    out = orc.round_table_f32(T)
    assert out.dtype == np.float32 and out.shape == T.shape
    for t, o in zip(T, out):
        want = np.float32(rne32_or_inf(Fraction(float(t))))
        if t == 0.0:
            want = np.float32(t)                                         # the sign of zero is kept
        assert o.tobytes() == want.tobytes(), f"round({t!r}) = {o!r}, want {want!r}"


def check_f32_reconstruction(orc, seed=9):
    """Unquantized mode against the fp64 reconstruction A_hat B, A_hat the
    sum of the selected prototypes.  With T the exact table entries, each
    fp32 entry is within 2^-24 |T| of T (round to nearest) and the ordered
    fp32 sum of C entries errs by at most gamma_C^(32) sum |T32| <=
    gamma_C^(32) (1 + 2^-24) sum |T|, so |y - A_hat B| <= (gamma_C^(32)
    (1 + 2^-24) + 2^-24) sum_c |T_c| plus the double roundings of T and of
    the reference: a rigorous bound that does not use the oracle's own table."""
    rng = np.random.default_rng(seed)
    N, C, L, M = 40, 6, 3, 7
    D = C * L
    P = np.zeros((C, K, D), np.float32)
    for c in range(C):
        P[c, :, c * L:(c + 1) * L] = rng.standard_normal((K, L), dtype=np.float32)
    B = rng.standard_normal((D, M), dtype=np.float32)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = (np.arange(C)[:, None] * L + rng.integers(0, L, size=(C, LEVELS))).astype(np.int32)
    thr = rng.standard_normal((C, NODES), dtype=np.float32)
    T32 = orc.build_lut_f32(P, B)
    idx, y = orc.matmul_f32(A, split, thr, T32)
    Tx = exact_table(P, B)
    for n in range(N):
        Ahat = sum(P[c, idx[n, c]].astype(np.float64) for c in range(C))
        for m in range(M):
            ref = math.fsum(Ahat * B[:, m].astype(np.float64))
            tx = np.array([Tx[c, idx[n, c], m] for c in range(C)])
            ax = float(np.abs(tx).sum())
            bound = (gamma(C, U32) * (1 + U32) + U32) * ax + 2 * U64 * ax + 4 * U64 * abs(ref)
            assert abs(float(y[n, m]) - ref) <= bound, f"({n},{m}) outside reconstruction bound"


def check_quantized_reconstruction(orc, seed=10):
    """Quantized end to end: |y - A_hat B| <= sum_c 2^e_c / 2 (code rounding)
    + |bias32 - sum o| + 2^-24 |y| + table and reconstruction rounding."""
    rng = np.random.default_rng(seed)
    N, C, L, M = 50, 8, 4, 6
    D = C * L
    P = np.zeros((C, K, D), np.float32)
    for c in range(C):
        P[c, :, c * L:(c + 1) * L] = rng.standard_normal((K, L), dtype=np.float32)
    B = rng.standard_normal((D, M), dtype=np.float32)
    A = rng.standard_normal((N, D), dtype=np.float32)
    split = (np.arange(C)[:, None] * L + rng.integers(0, L, size=(C, LEVELS))).astype(np.int32)
    thr = rng.standard_normal((C, NODES), dtype=np.float32)
    lut, scale, offset = orc.build_quantized_lut(P, B)
    idx, acc, y = orc.matmul(A, split, thr, lut, scale, offset)
    _, _, bias = orc.dequant_params(scale, offset)
    S = math.fsum(offset.astype(np.float64))
    half = float(np.sum(scale.astype(np.float64))) / 2
    for n in range(N):
        Ahat = sum(P[c, idx[n, c]].astype(np.float64) for c in range(C))
        for m in range(M):
            ref = math.fsum(Ahat * B[:, m].astype(np.float64))
            tab = sum(abs(float(x)) for x in (P[c, idx[n, c]].astype(np.float64) * B[:, m] for c in range(C)) for x in x)
            bound = (half + abs(float(bias) - S) + U32 * abs(float(y[n, m])) + gamma(D, U64) * tab
                     + 4 * U64 * abs(ref))
            assert abs(float(y[n, m]) - ref) <= bound * (1 + 1e-9), f"({n},{m}) outside bound"


def bound_shifts():
    """Shifts e_c - e_min whose sum of 2^sh is exactly 2^24: 23, 22, ..., 0, 0.
    With every code -128 the sum is -128 * 2^24 = -2^31, the int32 minimum."""
    return np.array(list(range(23, -1, -1)) + [0], np.int64)


def check_accumulator_bound(orc, seed=24):
    """R7: any int8 codes are admitted exactly when the most negative sum,
    -128 sum_c 2^sh_c, fits int32.  At sum 2^sh = 2^24 every code -128 sums
    to exactly -2^31 and every code 127 to 127 * 2^24 (both admitted, both
    exact); one more unit of 2^sh, or shifts (24, 0), is rejected although
    127 sum 2^sh is still below 2^31."""
    from oracle import OracleError
    rng = np.random.default_rng(seed)
    sh = bound_shifts()
    C, N, M = len(sh), 30, 5
    assert int((2 ** sh).sum()) == 2 ** 24
    e_min = -40
    scale = np.ldexp(np.float32(1), (sh + e_min).astype(np.int32)).astype(np.float32)
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    for code, want in ((-128, -2 ** 31), (127, 127 * 2 ** 24)):
        acc, y = orc.lut_accumulate(idx, np.full((C, K, M), code, np.int8), scale, np.zeros(C, np.float32))
        assert np.all(acc.astype(np.int64) == want), f"codes {code}: acc {acc[0, 0]} != {want}"
        assert np.all(y == np.float32(rne32(Fraction(want) * Fraction(2) ** e_min)))
    # mixed codes at the bound against the exact integer sum
    lut = rng.integers(-128, 128, size=(C, K, M)).astype(np.int8)
    acc, _ = orc.lut_accumulate(idx, lut, scale, np.zeros(C, np.float32))
    assert np.array_equal(acc.astype(np.int64), one_hot(idx) @ (lut.astype(np.int64) * (2 ** sh)[:, None, None]).reshape(C * K, M))
    over = [np.append(sh, 0), np.array([24, 0])]
    for bad in over:
        assert 127 * int((2 ** bad).sum()) < 2 ** 31 < 128 * int((2 ** bad).sum())
        sc = np.ldexp(np.float32(1), (bad + e_min).astype(np.int32)).astype(np.float32)
        try:
            orc.dequant_params(sc, np.zeros(len(bad), np.float32))
        except OracleError:
            continue
        raise AssertionError(f"shifts {bad.tolist()} admitted although -128 codes overflow int32")


def check_rejects_bad_inputs(orc):
    from oracle import OracleError
    idx = np.zeros((2, 2), np.uint8)
    lut = np.zeros((2, K, 3), np.int8)
    for bad in ([0.75, 1.0], [3.0, 1.0], [1.0, 2.0 ** 40], [2.0 ** -130, 1.0]):
        try:
            orc.lut_accumulate(idx, lut, np.array(bad, np.float32), np.zeros(2, np.float32))
        except OracleError:
            continue
        raise AssertionError(f"scale {bad} accepted")
    try:
        orc.encode(np.zeros((1, 4), np.float32), np.array([[0, 1, 2, 4]], np.int32),
                   np.zeros((1, NODES), np.float32))
    except OracleError:
        pass
    else:
        raise AssertionError("split column outside [0, D) accepted")


def check_sigma_bias_relu(orc, seed=11):
    """Layer output, elementwise part (§2.2, reading R19): the bias add is one
    fp32 rounding (numpy float32 addition) and ReLU keeps z > 0 and gives +0
    otherwise, -0 included."""
    rng = np.random.default_rng(seed)
    y = rng.standard_normal((37, 13)).astype(np.float32)
    y[0, :4] = [0.0, -0.0, 1e-30, -1e-30]
    b = rng.standard_normal(13).astype(np.float32)
    z32 = y + b[None, :]                       # float32 + float32: one rounding
    assert z32.dtype == np.float32
    assert np.array_equal(orc.sigma(y, None, 0), y.astype(np.float64))
    assert np.array_equal(orc.sigma(y, b, 1), z32.astype(np.float64))
    r = orc.sigma(y, b, 2)
    assert np.array_equal(r, np.maximum(z32, np.float32(0)).astype(np.float64))
    assert not np.any(np.signbit(r))
    r0 = orc.sigma(np.array([[-0.0, 0.0, -1.0, 2.5]], np.float32), None, 2)
    assert np.array_equal(r0, [[0.0, 0.0, 0.0, 2.5]]) and not np.any(np.signbit(r0))


def check_sigma_softmax(orc, seed=12):
    """Layer output, row-wise part (§2.2, R19): two columns reduce to the
    logistic function, rows match scipy's softmax and sum to one, a constant
    row shift (an exactly representable bias) changes nothing, equal entries
    give 1/M, large entries do not overflow, and the bias is per column."""
    from scipy.special import expit
    from scipy.special import softmax as sp_softmax
    rng = np.random.default_rng(seed)
    y2 = (rng.standard_normal((50, 2)) * 4).astype(np.float32)
    p = orc.sigma(y2, None, 3)
    assert np.allclose(p[:, 0], expit(y2[:, 0].astype(np.float64) - y2[:, 1].astype(np.float64)), rtol=1e-14, atol=0)
    y = (rng.standard_normal((64, 37)) * 3).astype(np.float32)
    p = orc.sigma(y, None, 3)
    assert np.all(p > 0)
    assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert np.allclose(p, sp_softmax(y.astype(np.float64), axis=1), rtol=1e-13, atol=0)
    yg = (np.round(rng.standard_normal((16, 9)) * 1024) / 1024).astype(np.float32)   # y + 256 exact
    assert np.allclose(orc.sigma(yg, np.full(9, 256.0, np.float32), 3), orc.sigma(yg, None, 3), rtol=1e-14, atol=0)
    assert np.allclose(orc.sigma(np.full((3, 7), 5.5, np.float32), None, 3), 1.0 / 7, rtol=1e-15, atol=0)
    e = math.exp(-1.0)
    for base in (1000.0, -1000.0):   # no overflow, no underflow to 0/0
        big = orc.sigma(np.array([[base, base - 1.0, base]], np.float32), None, 3)
        assert np.allclose(big[0], [1 / (2 + e), e / (2 + e), 1 / (2 + e)], rtol=1e-14, atol=0)
    b = np.array([0.0, np.float32(math.log(3.0))], np.float32)
    pb = orc.sigma(np.zeros((2, 2), np.float32), b, 3)
    w = math.exp(float(b[1]))
    assert np.allclose(pb, [[1 / (1 + w), w / (1 + w)]] * 2, rtol=1e-14, atol=0)


def _shared_codes(C, M, seed):
    rng = np.random.default_rng(seed)
    lut = rng.integers(-127, 128, size=(C, K, M)).astype(np.int8)
    scale = np.full(C, np.float32(2.0 ** -7), np.float32)
    offset = (rng.standard_normal(C) * 0.25).astype(np.float32)
    return lut, scale, offset


def check_avg_closed_forms(orc, seed=13):
    """Rounded 8-bit summation (§1, reading R20) in the cases the definition
    reduces to by hand: one codebook is exact; two codebooks are one rounded
    average, (u0 + u1 + 1) >> 1 with u = q + 128, times 2; three codebooks are
    padded with a 128 leaf; equal codes over a power-of-two count are exact;
    y uses the exact path's dequantization of acc."""
    rng = np.random.default_rng(seed)
    N, M = 50, 7
    for C in (1, 2, 3, 4, 8):
        lut, scale, offset = _shared_codes(C, M, seed + C)
        idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
        acc, y = orc.lut_accumulate_avg(idx, lut, scale, offset)
        q = np.stack([lut[c][idx[:, c]] for c in range(C)], axis=1).astype(np.int64)   # [N, C, M]
        u = q + 128
        if C == 1:
            ref = q[:, 0]
        elif C == 2:
            ref = 2 * (((u[:, 0] + u[:, 1] + 1) >> 1) - 128)
        elif C == 3:
            left = (u[:, 0] + u[:, 1] + 1) >> 1
            right = (u[:, 2] + 128 + 1) >> 1
            ref = 4 * (((left + right + 1) >> 1) - 128)
        else:
            ref = None
        if ref is not None:
            assert np.array_equal(acc, ref)
        sh, emin, bias32 = orc.dequant_params(scale, offset)
        assert np.array_equal(y, (acc.astype(np.float32) * np.float32(2.0 ** emin) + bias32).astype(np.float32)) or \
            np.array_equal(y, np.float32(2.0 ** emin) * acc.astype(np.float32) + bias32)
    for C in (4, 16, 64):
        lut = np.repeat(np.arange(-8, 8, dtype=np.int8)[None, :, None], C, axis=0).repeat(3, axis=2)
        scale = np.full(C, np.float32(0.5), np.float32)
        offset = np.zeros(C, np.float32)
        idx = np.full((5, C), 11, np.uint8)                  # every codebook picks code 3
        acc, _ = orc.lut_accumulate_avg(idx, lut, scale, offset)
        assert np.all(acc == 3 * C)


def check_avg_bounds(orc, seed=14):
    """Each rounded average adds at most 1/2 to its exact value and its error
    halves per level above, so 0 <= acc - sum_c q_c <= P L / 2 (P = 2^L >= C);
    raising one code never lowers acc; mixed scales are rejected."""
    rng = np.random.default_rng(seed)
    for C in (5, 32, 100):
        lut, scale, offset = _shared_codes(C, 9, seed + C)
        idx = rng.integers(0, K, size=(200, C)).astype(np.uint8)
        acc, _ = orc.lut_accumulate_avg(idx, lut, scale, offset)
        exact, _ = orc.lut_accumulate(idx, lut, scale, offset)
        P = 1 << int(math.ceil(math.log2(C)))
        L = int(math.log2(P))
        err = acc.astype(np.int64) - exact.astype(np.int64)
        assert err.min() >= 0 and err.max() <= P * L // 2
        lut2 = lut.copy()
        bump = lut2 < 127
        lut2[bump] += 1
        acc2, _ = orc.lut_accumulate_avg(idx, lut2, scale, offset)
        assert np.all(acc2 >= acc)
    lut, scale, offset = _shared_codes(4, 3, 1)
    scale[2] *= 2
    try:
        orc.lut_accumulate_avg(np.zeros((2, 4), np.uint8), lut, scale, offset)
    except Exception:
        pass
    else:
        raise AssertionError("mixed scales accepted")


def check_shared_quantizer(orc, seed=15):
    """The shared-exponent quantizer (R20): one scale for all codebooks, the
    largest of the per-codebook minimal exponents; codes within [-127, 127]
    and within half a step of T - offset; identical to the per-codebook
    quantizer when those exponents already agree (one codebook)."""
    rng = np.random.default_rng(seed)
    T = rng.standard_normal((6, K, 11)) * np.array([0.1, 1, 3, 0.02, 7, 0.5])[:, None, None]
    lut, scale, offset = orc.quantize_table_shared(T)
    assert np.all(scale == scale[0])
    lut_r, scale_r, _ = orc.quantize_table(T)
    assert scale[0] == scale_r.max()
    step = float(scale[0])
    resid = T - offset[:, None, None].astype(np.float64) - lut.astype(np.float64) * step
    assert np.abs(resid).max() <= step / 2 * (1 + 1e-12)
    T1 = T[4:5]
    assert all(np.array_equal(a, b) for a, b in zip(orc.quantize_table_shared(T1), orc.quantize_table(T1)))


# ------------------------------------------------------- table fit (Eq. 3)
def _fit_problem(N, C, M, seed, missing=()):
    """Seeded indices, targets and prototype table for the fit pins; the
    buckets listed in `missing` ((c, k) pairs) never occur."""
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    for c, k in missing:
        col = idx[:, c]
        col[col == k] = (k + 1) % K
    Y = rng.standard_normal((N, M)).astype(np.float32)
    T0 = rng.standard_normal((C, K, M)).astype(np.float32)
    return idx, Y, T0


def _gather(idx, T):
    """sum_c T[c, idx[:, c], :] in float64 (the product G T without forming G)."""
    T = np.asarray(T, dtype=np.float64)
    return sum(T[c][idx[:, c]] for c in range(idx.shape[1]))


def _ridge_objective(idx, Y, T, T0, lam):
    r = Y.astype(np.float64) - _gather(idx, T)
    d = np.asarray(T, np.float64) - np.asarray(T0, np.float64)
    return float((r * r).sum() + lam * (d * d).sum())


def check_encoder_gram(orc, seed=16):
    """H = G^T G: block (c, c') is the 16 x 16 contingency table of the
    indices of codebooks c and c' (numpy.histogram2d), so block (c, c) is
    diagonal with the bucket counts (numpy.bincount), H is symmetric and sums
    to N C^2."""
    rng = np.random.default_rng(seed)
    N, C = 300, 5
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    idx[:, 3] = np.minimum(idx[:, 3], 9)   # some buckets empty
    H = orc.encoder_gram(idx)
    assert H.shape == (C * K, C * K)
    for c in range(C):
        for c2 in range(C):
            ref, _, _ = np.histogram2d(idx[:, c], idx[:, c2], bins=K, range=[[0, K], [0, K]])
            assert np.array_equal(H[c * K:(c + 1) * K, c2 * K:(c2 + 1) * K], ref.astype(np.int64))
        assert np.array_equal(np.diag(H[c * K:(c + 1) * K, c * K:(c + 1) * K]), np.bincount(idx[:, c], minlength=K))
    assert np.array_equal(H, H.T) and H.sum() == N * C * C


def check_encoder_scatter(orc, seed=17):
    """R = G^T Y: row (c, k) is the sum of the target rows whose codebook-c
    index is k (correctly rounded reference sums, math.fsum); every codebook's
    block sums to the column totals of Y."""
    rng = np.random.default_rng(seed)
    N, C, M = 257, 4, 6
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    Y = (rng.standard_normal((N, M)) * 10).astype(np.float32)
    R = orc.encoder_scatter(idx, Y)
    bound = gamma(N, U64) * np.abs(Y.astype(np.float64)).sum(axis=0)
    for c in range(C):
        for k in range(K):
            rows = Y[idx[:, c] == k].astype(np.float64)
            ref = np.array([math.fsum(rows[:, m]) for m in range(M)])
            assert np.all(np.abs(R[c * K + k] - ref) <= bound)
        tot = np.array([math.fsum(Y[:, m].astype(np.float64)) for m in range(M)])
        assert np.all(np.abs(R[c * K:(c + 1) * K].sum(axis=0) - tot) <= 2 * bound)


def check_fit_closed_forms(orc, seed=18):
    """Eq. 3 with sigma affine (R21) where the minimiser is known in closed
    form: one codebook decouples into per-bucket ridge means (sum_k Y + lam
    T0_k) / (n_k + lam); a bucket that never occurs keeps its prototype row;
    targets that an integer table T* reproduces exactly, with T0 = T*, give
    T*; and for every lam, ||T - T0|| <= ||G^T (Y - G T0)|| / lam per column
    (the matrix H + lam I has smallest eigenvalue >= lam)."""
    rng = np.random.default_rng(seed)
    # one codebook
    idx, Y, T0 = _fit_problem(200, 1, 5, seed, missing=[(0, 13)])
    lam = 3.5
    T = orc.fit_lut_ridge(idx, Y, T0, lam)
    for k in range(K):
        rows = Y[idx[:, 0] == k].astype(np.float64)
        num = np.array([math.fsum(list(rows[:, m]) + [lam * float(T0[0, k, m])]) for m in range(5)])
        ref = num / (len(rows) + lam)
        assert np.allclose(T[0, k], ref, rtol=1e-12, atol=1e-14)
    assert np.allclose(T[0, 13], T0[0, 13], rtol=1e-14, atol=0)
    # several codebooks: an empty bucket keeps T0 exactly (up to the solve's rounding)
    idx, Y, T0 = _fit_problem(400, 6, 4, seed + 1, missing=[(2, 5), (4, 0)])
    T = orc.fit_lut_ridge(idx, Y, T0, 0.7)
    assert np.allclose(T[2, 5], T0[2, 5], rtol=1e-13, atol=0) and np.allclose(T[4, 0], T0[4, 0], rtol=1e-13, atol=0)
    # exact recovery
    C, M = 5, 3
    Ts = rng.integers(-8, 9, size=(C, K, M)).astype(np.float32)
    idx = rng.integers(0, K, size=(300, C)).astype(np.uint8)
    Yx = _gather(idx, Ts).astype(np.float32)
    assert np.array_equal(Yx.astype(np.float64), _gather(idx, Ts))   # integer sums: exact in fp32
    for lam in (1e-3, 1.0, 1e4):
        T = orc.fit_lut_ridge(idx, Yx, Ts, lam)
        assert np.abs(T - Ts).max() <= 1e-9
    # the eigenvalue bound, at weak and strong regularisation
    idx, Y, T0 = _fit_problem(500, 4, 3, seed + 2)
    G = np.zeros((500, 4 * K))
    G[np.arange(500)[:, None], K * np.arange(4)[None, :] + idx] = 1.0
    resid = G.T @ (Y.astype(np.float64) - _gather(idx, T0))
    for lam in (0.01, 1.0, 1e3, 1e9):
        T = orc.fit_lut_ridge(idx, Y, T0, lam)
        d = (T - T0.astype(np.float64)).reshape(4 * K, 3)
        assert np.all(np.linalg.norm(d, axis=0) <= np.linalg.norm(resid, axis=0) / lam * (1 + 1e-9))


def check_fit_optimality(orc, seed=19):
    """The fitted table minimises the objective of Eq. 3 (R21) evaluated
    directly (gather, squared residuals, penalty): at a minimiser of a
    quadratic, f(T + e E) - f(T) equals e^2 (||G E||^2 + lam ||E||^2) for
    every direction E (no first-order term), and a generic minimiser
    (scipy BFGS on a tiny case) agrees."""
    from scipy.optimize import minimize
    rng = np.random.default_rng(seed)
    idx, Y, T0 = _fit_problem(120, 3, 2, seed)
    lam = 0.4
    T = orc.fit_lut_ridge(idx, Y, T0, lam)
    f0 = _ridge_objective(idx, Y, T, T0, lam)
    for _ in range(6):
        E = rng.standard_normal(T.shape)
        for e in (1e-3, 1.0):
            GE = _gather(idx, E)
            quad = e * e * (float((GE * GE).sum()) + lam * float((E * E).sum()))
            df = _ridge_objective(idx, Y, T + e * E, T0, lam) - f0
            assert abs(df - quad) <= 1e-9 * (f0 + quad) + 1e-12
    # brute-force minimisation of the same objective on a tiny case
    idx, Y, T0 = _fit_problem(12, 2, 1, seed + 1)
    lam = 0.25
    T = orc.fit_lut_ridge(idx, Y, T0, lam)
    res = minimize(lambda v: _ridge_objective(idx, Y, v.reshape(2, K, 1), T0, lam), T0.astype(np.float64).ravel(),
                   method="BFGS", options={"gtol": 1e-10})
    assert np.abs(res.x.reshape(2, K, 1) - T).max() <= 1e-5


# ------------------------------------------- table fit, nonlinear sigma (R22)
def _gd_objective(idx, Y, T, T0, lam, act, bias):
    """Eq. 3 evaluated directly: act 2 = squared error after bias + ReLU, act 3
    = KL divergence between the row softmaxes (scipy), act 4 = squared error
    between the row softmaxes (scipy), plus lam ||T - T0||^2."""
    from scipy.special import rel_entr, softmax
    b = np.zeros(Y.shape[1]) if bias is None else bias.astype(np.float64)
    z = _gather(idx, T) + b
    t = Y.astype(np.float64) + b
    if act == 2:
        r = np.maximum(t, 0.0) - np.maximum(z, 0.0)
        f = float((r * r).sum())
    elif act == 3:
        f = float(rel_entr(softmax(t, axis=1), softmax(z, axis=1)).sum())
    else:
        r = softmax(z, axis=1) - softmax(t, axis=1)
        f = float((r * r).sum())
    d = np.asarray(T, np.float64) - np.asarray(T0, np.float64)
    return f + lam * float((d * d).sum())


def check_fit_gd_gradient(orc, seed=20):
    """One gradient step moves T by -eta times the gradient of Eq. 3's
    objective: (T_k - T_{k+1}) / eta matches central finite differences of the
    objective (evaluated directly), at T0 and after a first step (where the
    penalty contributes), for ReLU, softmax with the KL divergence and softmax
    with the squared error, with and without a bias."""
    rng = np.random.default_rng(seed)
    idx, Y, T0 = _fit_problem(30, 2, 4, seed)
    for act in (2, 3, 4):
        for bias in (None, rng.standard_normal(4).astype(np.float32)):
            lam, eta = 0.3, 1e-3
            T1 = orc.fit_lut_gd(idx, Y, T0, act, lam, eta, 1, bias)
            T2 = orc.fit_lut_gd(idx, Y, T0, act, lam, eta, 2, bias)
            for Ta, Tb in ((T0.astype(np.float64), T1), (T1, T2)):
                g = (Ta - Tb) / eta
                h = 1e-6
                for _ in range(12):
                    e = tuple(int(rng.integers(0, d)) for d in T0.shape)
                    Tp, Tm = Ta.copy(), Ta.copy()
                    Tp[e] += h
                    Tm[e] -= h
                    fd = (_gd_objective(idx, Y, Tp, T0, lam, act, bias) -
                          _gd_objective(idx, Y, Tm, T0, lam, act, bias)) / (2 * h)
                    assert abs(fd - g[e]) <= 1e-5 * (1 + abs(fd)), (act, e, fd, g[e])


def check_fit_gd_fixed_point(orc, seed=21):
    """Targets the prototype table already reproduces: for ReLU, Y = G T0
    exactly (integer table) leaves T0 unchanged bit for bit; for softmax, any
    per-row shift of G T0 gives the same row distributions (softmax is shift
    invariant), so the gradient vanishes and T stays at T0 to rounding."""
    rng = np.random.default_rng(seed)
    C, M, N = 3, 5, 60
    idx = rng.integers(0, K, size=(N, C)).astype(np.uint8)
    T0 = rng.integers(-6, 7, size=(C, K, M)).astype(np.float32)
    bias = rng.integers(-3, 4, size=M).astype(np.float32)
    Y = _gather(idx, T0).astype(np.float32)
    T = orc.fit_lut_gd(idx, Y, T0, 2, 0.5, 0.01, 25, bias)
    assert np.array_equal(T, T0.astype(np.float64))
    shift = rng.integers(-4, 5, size=(N, 1)).astype(np.float64)
    Ys = (_gather(idx, T0) + shift).astype(np.float32)
    for act in (3, 4):
        T = orc.fit_lut_gd(idx, Ys, T0, act, 0.5, 0.01, 25, bias)
        assert np.abs(T - T0).max() <= 1e-12


def check_fit_gd_descent_and_limit(orc, seed=22):
    """Small steps never raise the objective (softmax with KL: convex; ReLU
    and softmax with the squared error from a generic start), and many steps
    reach the minimiser a generic method (scipy BFGS on the directly
    evaluated objective) finds on a tiny case."""
    from scipy.optimize import minimize
    idx, Y, T0 = _fit_problem(40, 2, 3, seed)
    bias = np.array([0.2, -0.1, 0.4], np.float32)
    for act in (2, 3, 4):
        fs = [_gd_objective(idx, Y, orc.fit_lut_gd(idx, Y, T0, act, 0.2, 5e-3, k, bias), T0, 0.2, act, bias)
              for k in range(0, 6)]
        assert all(b <= a + 1e-12 for a, b in zip(fs, fs[1:])) and fs[-1] < fs[0]
    idx, Y, T0 = _fit_problem(16, 1, 2, seed + 1)
    lam = 0.5
    for act in (3, 4):
        T = orc.fit_lut_gd(idx, Y, T0, act, lam, 0.2, 4000)
        res = minimize(lambda v: _gd_objective(idx, Y, v.reshape(1, K, 2), T0, lam, act, None),
                       T0.astype(np.float64).ravel(), method="BFGS", options={"gtol": 1e-12})
        assert np.abs(res.x.reshape(1, K, 2) - T).max() <= 1e-5, act


ALL_CHECKS = [
    check_encode_brute_force, check_encode_search_tree, check_encode_nan, check_encode_permutation,
    check_encode_golden, check_one_hot_identity, check_decoder_table, check_output_rounding,
    check_scale_linearity, check_f32_order, check_table_build, check_quantizer,
    check_round_table_f32, check_f32_reconstruction, check_quantized_reconstruction, check_accumulator_bound,
    check_rejects_bad_inputs,
    check_sigma_bias_relu, check_sigma_softmax, check_avg_closed_forms, check_avg_bounds,
    check_shared_quantizer, check_encoder_gram, check_encoder_scatter, check_fit_closed_forms,
    check_fit_optimality, check_fit_gd_gradient, check_fit_gd_fixed_point, check_fit_gd_descent_and_limit,
]
