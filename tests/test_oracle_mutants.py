"""Plant plausible mistakes in copies of the oracle (on the CPU) and require
the pin suite to catch every one of them.  This checks that the pins are
sharp enough: a dropped term, a wrong sign, index or operand fails a pin."""
import os
import subprocess

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "maddness_oracle.c")

MUTANTS = [
    ("ties go right", "int bit = (x > v) ? 1 : 0;", "int bit = (x >= v) ? 1 : 0;"),
    ("root bit is the LSB", "i = 2 * i + bit;", "i = i + (bit << t);"),
    ("wrong node numbering", "thr[c * ORACLE_NODES + ((1 << t) - 1) + i]", "thr[c * ORACLE_NODES + t + i]"),
    ("split table transposed", "row[split[c * ORACLE_LEVELS + t]]", "row[split[t * C + c]]"),
    ("row stride ignored", "const float* row = A + n * lda;", "const float* row = A + n * D;"),
    ("shift dropped", "acc += q * ((int64_t)1 << sh[c]);", "acc += q;"),
    ("table operand transposed", "int64_t q = lut[((int64_t)c * ORACLE_K + k) * M + m];",
     "int64_t q = lut[((int64_t)k * C + c % ORACLE_K) * M + m];"),
    ("index table transposed", "int k = idx[n * C + c];\n                int64_t q",
     "int k = idx[(c * N + n) % (N * C)];\n                int64_t q"),
    ("bias dropped", "for (int32_t c = 0; c < C; ++c) s += (double)offset[c];",
     "for (int32_t c = 0; c < C; ++c) s += 0.0 * (double)offset[c];"),
    ("step off by one", "const float step = ldexpf(1.0f, emin);", "const float step = ldexpf(1.0f, emin + 1);"),
    ("fp32 sum reversed", "s = s + lut[((int64_t)c * ORACLE_K + k) * M + m];",
     "s = s + lut[((int64_t)(C - 1 - c) * ORACLE_K + idx[n * C + (C - 1 - c)]) * M + m];"),
    ("fp32 sum in double", "float s = 0.0f;\n            for (int32_t c = 0; c < C; ++c) {\n                int k",
     "double s = 0.0;\n            for (int32_t c = 0; c < C; ++c) {\n                int k"),
    ("weights transposed", "(double)B[(int64_t)d * M + m];", "(double)B[((int64_t)m * D + d) % ((int64_t)D * M)];"),
    ("codes floored", "double q = nearbyint((t[j] - o) / ldexp(1.0, e));", "double q = floor((t[j] - o) / ldexp(1.0, e));"),
    ("offset sign", "double q = nearbyint((t[j] - o) / ldexp(1.0, e));", "double q = nearbyint((t[j] + o) / ldexp(1.0, e));"),
    ("exponent one too large", "        offset[c] = o;\n        ec[c] = e;", "        offset[c] = o;\n        ec[c] = e + 1;"),
    ("exponent floor ignored", "if (e < emax - cap) e = emax - cap;", "(void)cap;"),
    ("offset not the midrange", "float o = (float)((lo + hi) / 2.0);", "float o = (float)lo;"),
    ("layer bias subtracted", "z = z + bias[m];", "z = z - bias[m];"),
    ("ReLU keeps -0", "z = (z > 0.0f) ? z : 0.0f;", "z = (z >= 0.0f) ? z : 0.0f;"),
    ("softmax without the max shift", "o[m] = exp(o[m] - mx);", "o[m] = exp(o[m]);"),
    ("softmax max not initialised from the row", "double mx = o[0];", "double mx = 0.0;"),
    ("softmax normalised by the first term", "for (int32_t m = 0; m < M; ++m) o[m] = o[m] / sum;",
     "for (int32_t m = M - 1; m >= 0; --m) o[m] = o[m] / o[0];"),
    ("average rounds down", "u[i] = (u[2 * i] + u[2 * i + 1] + 1) >> 1;", "u[i] = (u[2 * i] + u[2 * i + 1]) >> 1;"),
    ("padding leaves are zero", "                    u[c] = 128;\n", "                    u[c] = 0;\n"),
    ("estimate scaled by C", "const int32_t a = P * (u[0] - 128);", "const int32_t a = C * (u[0] - 128);"),
    ("code bias not removed", "const int32_t a = P * (u[0] - 128);", "const int32_t a = P * u[0];"),
    ("shared quantizer keeps per-codebook exponents", "return quantize_table_cap(T, C, M, 0, lut, scale, offset);",
     "return quantize_table_cap(T, C, M, oracle_exponent_cap(C), lut, scale, offset);"),
    ("gram pairs a codebook with itself", "const int64_t s = (int64_t)c2 * ORACLE_K + idx[n * C + c2];",
     "const int64_t s = (int64_t)c2 * ORACLE_K + idx[n * C + c];"),
    ("scatter adds column 0", "R[r * M + m] += (double)Y[n * M + m];", "R[r * M + m] += (double)Y[n * M];"),
    ("ridge term missing from the matrix", "(i == j ? lambda : 0.0)", "(i == j ? 1e-300 : 0.0)"),
    ("prototype term missing from the right-hand side", "z[i] = R[i * M + m] + lambda * (double)T0[i * M + m];",
     "z[i] = R[i * M + m];"),
    ("back substitution with the unfactored upper triangle", "v = fma(-L[k * n16 + i], z[k], v);",
     "v = fma(-L[i * n16 + k], z[k], v);"),
    ("ridge weight doubled in the matrix", "(i == j ? lambda : 0.0)", "(i == j ? 2.0 * lambda : 0.0)"),
    ("softmax residual of the wrong sign", "q[m] = q[m] - P[n * M + m];", "q[m] = P[n * M + m] - q[m];"),
    ("ReLU residual without the derivative",
     "q[m] = z[m] > 0.0 ? 2.0 * (z[m] - P[n * M + m]) : 0.0;",
     "q[m] = 2.0 * ((z[m] > 0.0 ? z[m] : 0.0) - P[n * M + m]);"),
    ("bias left out of the fitted outputs", "z[m] = sacc + (bias ? (double)bias[m] : 0.0);", "z[m] = sacc;"),
    ("penalty gradient without its factor 2", "const double g = R[j] + 2.0 * lambda * (T[j] - (double)T0[j]);",
     "const double g = R[j] + lambda * (T[j] - (double)T0[j]);"),
    ("step up the gradient", "T[j] = T[j] - eta * g;", "T[j] = T[j] + eta * g;"),
    ("softmax sum over half the row", "for (int32_t m = 0; m < M; ++m) { q[m] = exp(z[m] - mx); sum += q[m]; }",
     "for (int32_t m = 0; m < M; ++m) { q[m] = exp(z[m] - mx); if (m < M / 2 + 1) sum += q[m]; }"),
    ("fp32 table zeroed", "for (int64_t j = 0; j < n; ++j) out[j] = (float)T[j];",
     "for (int64_t j = 0; j < n; ++j) out[j] = 0.0f * (float)T[j];"),
    ("fp32 table scaled by 1.001", "for (int64_t j = 0; j < n; ++j) out[j] = (float)T[j];",
     "for (int64_t j = 0; j < n; ++j) out[j] = (float)(T[j] * 1.001);"),
    ("fp32 table rounded toward zero", "for (int64_t j = 0; j < n; ++j) out[j] = (float)T[j];",
     "for (int64_t j = 0; j < n; ++j) { float f = (float)T[j]; "
     "if (fabs((double)f) > fabs(T[j])) f = nextafterf(f, 0.0f); out[j] = f; }"),
    ("overflow bound for codes up to 127 only", "bound += 128.0 * ldexp(1.0, sh[c]);",
     "bound += 127.0 * ldexp(1.0, sh[c]);"),
    ("overflow bound excludes its edge", "if (bound > 2147483648.0) return -3;",
     "if (bound >= 2147483648.0) return -3;"),
    ("softmax squared-error residual without the Jacobian", "q[m] = 2.0 * (q[m] * (d - sdp));",
     "q[m] = 2.0 * d;"),
    ("softmax squared-error residual without the centring term", "q[m] = 2.0 * (q[m] * (d - sdp));",
     "q[m] = 2.0 * (q[m] * d);"),
    ("softmax squared-error centring term unweighted",
     "for (int32_t m = 0; m < M; ++m) sdp += (q[m] - P[n * M + m]) * q[m];",
     "for (int32_t m = 0; m < M; ++m) sdp += (q[m] - P[n * M + m]);"),
]


@pytest.mark.parametrize("what,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, what, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site not unique/found: {what}"
    mut = tmp_path / "mutant.c"
    mut.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", *oracle.CFLAGS, str(mut), "-o", str(so), "-lm"], check=True)
    orc = oracle.Oracle(str(so))
    caught = []
    for check in pins.ALL_CHECKS:
        try:
            check(orc)
        except (AssertionError, oracle.OracleError) as e:
            caught.append(check.__name__)
    assert caught, f"planted mistake '{what}' passed every pin"
