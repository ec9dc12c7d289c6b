"""The oracle's pins catch plausible mistakes.

Each mutant below is a copy of oracle/altr_oracle.c with one planted mistake
of the kind a careful reading could still miss (a dropped absolute value, a
flipped comparison, an off-by-one stride, a wrong row pitch, ...).  Every
mutant is compiled with gcc into a library of its own and the pin suite
(tests/test_oracle_pins.py) is run against it in a subprocess; the pins must
fail for every mutant.  The unmutated source, built the same way, must pass.
Everything runs on the CPU.
"""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "altr_oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# (name, text to replace, replacement): each text occurs exactly once.
MUTANTS = [
    # Eq. (3): the normaliser sums magnitudes
    ("normaliser_without_abs",
     "int D)\n{\n    double norm = 0.0;\n    for (int k = 0; k < D; ++k)\n"
     "        norm += fabs(elem(row, dtype, (size_t)k));\n    if (norm == 0.0)\n"
     "        return 0.0; /* reading: an all-zero row has H2 = 0 */",
     "int D)\n{\n    double norm = 0.0;\n    for (int k = 0; k < D; ++k)\n"
     "        norm += elem(row, dtype, (size_t)k);\n    if (norm == 0.0)\n"
     "        return 0.0; /* reading: an all-zero row has H2 = 0 */"),
    # Eq. (4): the sum of squared probabilities
    ("probabilities_not_squared", "        sum_p2 += p * p;", "        sum_p2 += p;"),
    ("entropy_sign", "    return -log(sum_p2);", "    return log(sum_p2);"),
    ("entropy_log2", "    return -log(sum_p2);", "    return -log2(sum_p2);"),
    ("zero_row_reading",
     "        return 0.0; /* reading: an all-zero row has H2 = 0 */",
     "        return log((double)D);"),
    # the Shannon variant
    ("shannon_sign", "            h -= q * log(q);", "            h += q * log(q);"),
    ("shannon_log_of_square", "            h -= q * log(q);", "            h -= q * log(q * q);"),
    ("shannon_without_abs", "        double q = fabs(elem(row, dtype, (size_t)j)) / norm;",
     "        double q = elem(row, dtype, (size_t)j) / norm;"),
    ("shannon_normaliser_without_abs",
     "        norm += fabs(elem(row, dtype, (size_t)k));\n    if (norm == 0.0)\n"
     "        return 0.0; /* reading: an all-zero row has H1 = 0 */",
     "        norm += elem(row, dtype, (size_t)k);\n    if (norm == 0.0)\n"
     "        return 0.0; /* reading: an all-zero row has H1 = 0 */"),
    ("entropy_variants_swapped", "            h2[i] = entropy == 1 ? altr_oracle_shannon(xr, dtype, D)",
     "            h2[i] = entropy == 2 ? altr_oracle_shannon(xr, dtype, D)"),
    # bf16 widening
    ("bf16_shift", "        uint32_t w = ((uint32_t)h) << 16;", "        uint32_t w = ((uint32_t)h) << 15;"),
    ("f64_rows_read_as_f32", "        return ((const double*)base)[i];",
     "        return (double)((const float*)base)[i];"),
    # the variance form used as a self-check
    ("sample_variance", "    v /= D;", "    v /= (D - 1);"),
    # Eq. (6)
    ("cosine_wrong_norm", "    return dot / sqrt(na * nb);", "    return dot / sqrt(na * na);"),
    ("cosine_abs_products", "        dot += u * w;", "        dot += fabs(u * w);"),
    ("cosine_zero_norm_reading",
     "    if (na == 0.0 || nb == 0.0)\n        return 0.0;",
     "    if (na == 0.0 || nb == 0.0)\n        return 1.0;"),
    ("state_rows_at_width_D",
     "            s[i] = altr_oracle_cosine((const char*)Xpre + (size_t)i * Dc * eb,",
     "            s[i] = altr_oracle_cosine((const char*)Xpre + (size_t)i * D * eb,"),
    # Algorithm 1, budget split and stride
    ("k1_rounded", "    int k1 = (int)floor(lambda * (double)K);", "    int k1 = (int)round(lambda * (double)K);"),
    ("k1_ceiling", "    int k1 = (int)floor(lambda * (double)K);", "    int k1 = (int)ceil(lambda * (double)K);"),
    ("stride_over_N", "    int r = N - k1;", "    int r = N;"),
    ("stride_ceiling", "        tt = r / k2;", "        tt = (r + k2 - 1) / k2;"),
    # Stage I order
    ("stage1_lowest_entropy",
     "    if (a->key > b->key) return -1;\n    if (a->key < b->key) return 1;\n"
     "    return (a->idx > b->idx) - (a->idx < b->idx);\n}\n\n/* Stage II",
     "    if (a->key < b->key) return -1;\n    if (a->key > b->key) return 1;\n"
     "    return (a->idx > b->idx) - (a->idx < b->idx);\n}\n\n/* Stage II"),
    ("stage1_ties_to_higher_index",
     "    if (a->key < b->key) return 1;\n    return (a->idx > b->idx) - (a->idx < b->idx);",
     "    if (a->key < b->key) return 1;\n    return (a->idx < b->idx) - (a->idx > b->idx);"),
    # Stage II order
    ("stage2_descending",
     "    if (a->key < b->key) return -1;\n    if (a->key > b->key) return 1;\n"
     "    return (a->idx > b->idx) - (a->idx < b->idx);\n}\n\n/* One image.",
     "    if (a->key > b->key) return -1;\n    if (a->key < b->key) return 1;\n"
     "    return (a->idx > b->idx) - (a->idx < b->idx);\n}\n\n/* One image."),
    ("stage2_unstable_ties",
     "    if (a->key > b->key) return 1;\n    return (a->idx > b->idx) - (a->idx < b->idx);",
     "    if (a->key > b->key) return 1;\n    return (a->idx < b->idx) - (a->idx > b->idx);"),
    ("remainder_keeps_imp", "            if (role[i] == 0) {", "            if (role[i] != 2) {"),
    # stride positions
    ("stride_last_of_interval", "                pos = (long)j * t;", "                pos = (long)(j + 1) * t - 1;"),
    ("stride_one_based", "                pos = (long)j * t;", "                pos = (long)j * t + (t > 1);"),
    ("real_stride_rounded",
     "                pos = (long)floor((double)j * (double)R / (double)K2);",
     "                pos = (long)round((double)j * (double)R / (double)K2);"),
    # output
    ("source_flag_inverted", "                out_src[k] = (uint8_t)(role[i] == 2);",
     "                out_src[k] = (uint8_t)(role[i] == 1);"),
    ("gather_without_image_offset",
     "                       (const char*)X + (size_t)(row0 + out_idx[out0 + k]) * D * eb,",
     "                       (const char*)X + (size_t)(out_idx[out0 + k]) * D * eb,"),
]


def _build(src_text: str, out_dir: str, name: str) -> str:
    c = os.path.join(out_dir, name + ".c")
    so = os.path.join(out_dir, "lib" + name + ".so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o", so, c, "-lm"])
    return so


def _pins_pass(lib: str) -> bool:
    env = dict(os.environ, ALTR_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", PINS], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    return r.returncode == 0


def _mutate(text: str, old: str, new: str) -> str:
    assert text.count(old) == 1, "mutation site not unique: %r" % old[:60]
    return text.replace(old, new)


def test_mutation_sites_exist():
    text = open(SRC).read()
    names = [m[0] for m in MUTANTS]
    assert len(names) == len(set(names))
    for name, old, new in MUTANTS:
        assert _mutate(text, old, new) != text, name


def test_every_mutant_fails_a_pin():
    text = open(SRC).read()
    with tempfile.TemporaryDirectory() as d:
        libs = {"unmutated": _build(text, d, "unmutated")}
        for name, old, new in MUTANTS:
            libs[name] = _build(_mutate(text, old, new), d, name)
        with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
            passed = dict(zip(libs, ex.map(_pins_pass, libs.values())))
    assert passed.pop("unmutated"), "the pins fail on the unmutated oracle built this way"
    survivors = sorted(n for n, ok in passed.items() if ok)
    assert not survivors, "mutants the pins do not catch: %s" % survivors
