"""Planted mistakes in the oracle must each fail one of its pins (CPU only).

Each mutation below is one plausible single-line slip in ``oracle/`` (a wrong
bias, midpoint or constant, a tie rule, a dropped term or sign, a swapped
nibble or bit order, a missed NaN/Inf check, a transposed index).  The oracle
package is copied into a temporary directory with that one change, rebuilt
there, and the pin tests named with the mutation are run against the copy:
every mutation must make at least one of them fail, and the unmutated copy
must pass them all.  This is what makes the pins evidence: a pin set that a
planted mistake survives does not constrain the oracle there.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
C = "reqat_oracle.c"
PY = "__init__.py"
FMT = ["test_oracle_formats.py"]
TEN = ["test_oracle_tensor.py"]
BOTH = FMT + TEN

# (file, text, replacement, pins expected to catch it, what the slip is)
MUTATIONS = [
    (C, "ldexp(1.0 + 0.5 * m, e - 1)", "ldexp(1.0 + 0.5 * m, e)", FMT, "E2M1 exponent bias"),
    (C, "(e == 0) ? 0.5 * m :", "(e == 0) ? 1.0 * m :", FMT, "E2M1 subnormal value"),
    (C, "ldexp(1.0 + m / 8.0, e - 7)", "ldexp(1.0 + m / 8.0, e - 8)", BOTH, "E4M3 bias (FNUZ-like)"),
    (C, "if (e == 15 && m == 7) return NAN;", "if (e == 15 && m == 7) return 448.0;", FMT, "E4M3 NaN encoding"),
    (C, "return ldexp(1.0, (int)b - 127);", "return ldexp(1.0, (int)b - 128);", BOTH, "E8M0 bias"),
    (C, "(r == 0.5 && fmod(lo, 2.0) != 0.0)", "(r == 0.5)", FMT, "bfloat16 ties away from zero"),
    (C, "if (ex < -126) ex = -126;", "if (ex < -133) ex = -133;", FMT, "bfloat16 subnormal spacing"),
    (C, "e = (2.0 * f <= 1.5) ? (ex - 1) - 2 : (ex - 1) - 1;",
     "e = (2.0 * f < 1.5) ? (ex - 1) - 2 : (ex - 1) - 1;", BOTH, "MX scale boundary at 1.5"),
    (C, "e = (2.0 * f <= 1.5) ? (ex - 1) - 2 : (ex - 1) - 1;", "e = (ex - 1) - 2;", BOTH,
     "MX scale by the floor rule (clips)"),
    (C, "k = (2.0 * f <= 1.3125) ? (ex - 1) - 11 : (ex - 1) - 10;",
     "k = (2.0 * f <= 1.5) ? (ex - 1) - 11 : (ex - 1) - 10;", BOTH, "NV global scale constant"),
    (C, "    if (k < -126) k = -126;\n    return (float)ldexp(1.0, k);\n}\n\n/* Ascending",
     "    return (float)ldexp(1.0, k);\n}\n\n/* Ascending", BOTH, "NV global scale clamp dropped"),
    (C, "for (i = 0; i < 126 && e4m3_pos_val[i] < q; i++) {}",
     "for (i = 0; i < 126 && e4m3_pos_val[i] <= q; i++) {}", BOTH, "NV scale off by one at exact values"),
    (C, "    q = amax / (6.0 * g);", "    q = amax / 6.0;", BOTH, "NV scale ignores g"),
    (C, "if (i >= 126) return 0x7E;  /* above 448: saturate */", "if (i >= 126) return 0x7F;", BOTH,
     "NV scale saturates to the NaN byte"),
    (C, "static const double mid[7] = {0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0};",
     "static const double mid[7] = {0.25, 0.75, 1.25, 1.5, 2.5, 3.5, 5.0};", BOTH, "E2M1 midpoint"),
    (C, "if (ax == t) return (i % 2 == 0) ? i : i + 1;   /* tie: the even code */",
     "if (ax == t) return (i % 2 == 0) ? i + 1 : i;", BOTH, "E2M1 ties to the odd code"),
    (C, "return (uint8_t)((signbit(x) ? 8 : 0) | m);", "return (uint8_t)((x < 0.0 ? 8 : 0) | m);", BOTH,
     "sign of -0 dropped"),
    (C, "                if (isnan(v) || isinf(v)) bad = 1;", "                if (isnan(v)) bad = 1;", TEN,
     "Inf not treated as a bad block"),
    (C, "double v = fabs(orc_bf16_value(x[r * ldx + c]));\n            if (!isnan(v) && !isinf(v) && v > m) m = v;",
     "double v = fabs(orc_bf16_value(x[r * ldx + c]));\n            if (!isnan(v) && v > m) m = v;", TEN,
     "tensor amax counts Inf"),
    (C, "if (k % 2 == 0) *p = (uint8_t)((*p & 0xF0) | c);\n                else *p = (uint8_t)((*p & 0x0F) | (c << 4));\n            }\n        }\n    }\n    return 0;\n}\n\n/* Dequantized",
     "if (k % 2 == 1) *p = (uint8_t)((*p & 0xF0) | c);\n                else *p = (uint8_t)((*p & 0x0F) | (c << 4));\n            }\n        }\n    }\n    return 0;\n}\n\n/* Dequantized",
     TEN, "nibble order"),
    (C, "    S = (fmt == ORC_FMT_MXFP4) ? orc_e8m0_value(sb) : orc_e4m3_value(sb) * g;\n            for (j = 0; j < B; j++) {",
     "    S = (fmt == ORC_FMT_MXFP4) ? orc_e8m0_value(sb) : orc_e4m3_value(sb);\n            for (j = 0; j < B; j++) {",
     TEN, "element codes ignore g"),
    (C, "uint8_t c = (k % 2 == 0) ? (byte & 0xF) : (byte >> 4);\n    uint8_t sb = scales",
     "uint8_t c = (k % 2 == 0) ? (byte >> 4) : (byte & 0xF);\n    uint8_t sb = scales", TEN,
     "dequantize nibble order"),
    (C, "uint8_t sb = scales[r * (cols / B) + k / B];", "uint8_t sb = scales[r * (cols / B) + k / 16];", TEN,
     "dequantize block index"),
    (C, "                       deq(fmt, b_codes, b_scales, gb, K, n, k);\n            y[(m - m0)",
     "                       deq(fmt, b_codes, b_scales, ga, K, n, k);\n            y[(m - m0)", TEN,
     "GEMM uses the wrong global scale"),
    (C, "            acc += t;\n            aacc += fabs(t);\n        }\n        y[p] = acc;\n        absy[p] = aacc;\n    }\n}\n\n/* ---------- array",
     "            acc += fabs(t);\n            aacc += fabs(t);\n        }\n        y[p] = acc;\n        absy[p] = aacc;\n    }\n}\n\n/* ---------- array",
     TEN, "GEMM sums magnitudes"),
    (C, "int hneg = __builtin_popcount((unsigned)(i & j)) & 1;",
     "int hneg = __builtin_popcount((unsigned)(i | j)) & 1;", ["test_oracle_rht.py"], "Hadamard sign pattern"),
    (C, "if ((signs >> j) & 1u) xneg = !xneg;", "if ((signs >> (31 - j)) & 1u) xneg = !xneg;",
     ["test_oracle_rht.py"], "sign word bit order"),
    (C, "bound = big_const(1152, 2 * e + 266);", "bound = big_const(36, 2 * e + 266);",
     ["test_oracle_rht.py"], "rotation normalisation dropped from the scale bound"),
    (C, "static const uint32_t mid_k[7] = {1, 3, 5, 7, 10, 14, 20};",
     "static const uint32_t mid_k[7] = {1, 3, 5, 7, 10, 14, 21};", ["test_oracle_rht.py"],
     "rotated E2M1 midpoint 5 moved"),
    (C, "    return e - 1;\n}", "    return e;\n}", ["test_oracle_rht.py"], "bfloat16 exponent offset in the exact sums"),
    (C, "negative[i] = c < 0;", "negative[i] = c <= 0;", ["test_oracle_rht.py"], "sign of a zero rotated value"),
    (C, "    return orc_bf16_value(orc_bf16_from_double(v));", "    return v;", ["test_oracle_w4a16.py"],
     "W4A16 weight not rounded to bfloat16"),
    (C, "if (a == t) { m = (i % 2 == 0) ? i : i + 1; break; }", "if (a == t) { m = i; break; }",
     ["test_oracle_kv4.py"], "E1M2 ties always down"),
    (C, "if (amax <= 1568.0 * ldexp(1.0, k)) break;", "if (amax <= 1792.0 * ldexp(1.0, k)) break;",
     ["test_oracle_kv4.py"], "KV4 global scale constant (4 * 448)"),
    (C, "if (amax <= 3.5 * e4m3_pos_val[i] * g) return e4m3_pos_byte[i];",
     "if (amax <= 4.0 * e4m3_pos_val[i] * g) return e4m3_pos_byte[i];", ["test_oracle_kv4.py"],
     "KV4 block scale bound"),
    (C, "return shift ? v - shift[c] : v;", "return shift ? v + shift[c] : v;", ["test_oracle_kv4.py"],
     "KV4 shift sign"),
    (PY, "    q = 0.75 * (len(H) - 1)", "    q = 0.75 * len(H) - 1", ["test_oracle_sem.py"],
     "SEM percentile position"),
    (PY, "(H - hmin) / (tau - hmin + eps)", "(H - hmin) / (tau + eps)", ["test_oracle_sem.py"],
     "SEM weight denominator"),
    (PY, "    H = -(p * logp).sum(axis=1)", "    H = (p * logp).sum(axis=1)", ["test_oracle_sem.py"],
     "entropy sign"),
    (PY, "    g -= lam * np.asarray(w, np.float64)[:, None] * p * (logp + np.asarray(H, np.float64)[:, None])",
     "    g -= lam * np.asarray(w, np.float64)[:, None] * p * (logp - np.asarray(H, np.float64)[:, None])",
     ["test_oracle_sem.py"], "entropy gradient term"),
    (PY, "    return l_sft + lam * l_ent, l_sft, l_ent, w", "    return l_sft + l_ent, l_sft, l_ent, w",
     ["test_oracle_sem.py"], "SEM weight lambda dropped"),
]

TEST_FILES = ["__init__.py", "conftest.py", "indep.py", "test_oracle_formats.py", "test_oracle_tensor.py",
              "test_oracle_rht.py", "test_oracle_kv4.py", "test_oracle_sem.py", "test_oracle_w4a16.py"]


def _tree(base, mutation=None):
    """A copy of the oracle package (with `mutation` applied) and of the pin tests under `base`."""
    os.makedirs(os.path.join(base, "oracle"))
    for name in (C, PY):
        with open(os.path.join(ROOT, "oracle", name)) as f:
            src = f.read()
        if mutation is not None and mutation[0] == name:
            assert src.count(mutation[1]) == 1, "mutation site not unique: %r" % mutation[1][:60]
            src = src.replace(mutation[1], mutation[2])
        with open(os.path.join(base, "oracle", name), "w") as f:
            f.write(src)
    os.makedirs(os.path.join(base, "tests"))
    for name in TEST_FILES:
        shutil.copy(os.path.join(ROOT, "tests", name), os.path.join(base, "tests", name))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(base, "tests", "golden"))
    os.symlink(os.path.join(ROOT, "paper_2606_15682_amd"), os.path.join(base, "paper_2606_15682_amd"))


def _pins_pass(base, pins):
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        *[os.path.join("tests", p) for p in pins]],
                       cwd=base, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode == 0, r.stdout[-2000:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    base0 = str(tmp_path / "clean")
    _tree(base0)
    ok, out = _pins_pass(base0, sorted({p for m in MUTATIONS for p in m[3]}))
    assert ok, "the unmutated oracle copy fails its pins:\n" + out

    def one(i):
        m = MUTATIONS[i]
        base = str(tmp_path / ("m%02d" % i))
        _tree(base, m)
        passed, _ = _pins_pass(base, m[3])
        return m[4], passed

    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(one, range(len(MUTATIONS))))
    survivors = [name for name, passed in results if passed]
    assert not survivors, "planted mistakes no pin catches: %s" % survivors
