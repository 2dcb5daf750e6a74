"""The oracle's pins catch plausible mistakes (CPU only).

Each case copies ``oracle/lpv_oracle.c`` to a temporary directory, plants one
mistake by text substitution (a dropped term, a flipped sign, a transposed
operand or index, a wrong decoder constant, ...), builds the copy and runs every
pin of ``pins.py`` against it in a child process.  The case passes when at least
one pin fails (or the mutant crashes).  The real oracle is never modified.
"""
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lpv_oracle.c")
HDR = os.path.join(ROOT, "oracle", "lpv_oracle.h")

MUTANTS = {
    "mask_index_transposed": ("mask[(n / b_r) * C + (k / b_c)]",
                              "mask[(k / b_c) * (N / b_r) + (n / b_r)]"),
    "block_sizes_swapped": ("mask[(n / b_r) * C + (k / b_c)]", "mask[(n / b_c) * C + (k / b_r)]"),
    "weight_transposed": ("dec_one(dtype, W, n * ldw + k)", "dec_one(dtype, W, k * ldw + n)"),
    "multiply_not_select": (
        "mask[(n / b_r) * C + (k / b_c)] ? dec_one(dtype, W, n * ldw + k) : 0.0",
        "dec_one(dtype, W, n * ldw + k) * (mask[(n / b_r) * C + (k / b_c)] ? 1.0 : 0.0)"),
    "bias_dropped": ("double v = acc[n] + j->b[n];", "double v = acc[n];"),
    "bias_reversed": ("double v = acc[n] + j->b[n];", "double v = acc[n] + j->b[j->N - 1 - n];"),
    "sign_flipped": ("acc[n] += xk * wk[n];", "acc[n] -= xk * wk[n];"),
    "last_k_dropped": ("for (int64_t k = 0; k < j->K; ++k) {\n            const double xk",
                       "for (int64_t k = 0; k < j->K - 1; ++k) {\n            const double xk"),
    "pack_cols_descending": ("for (int64_t c = 0; c < C; ++c) {\n            if (!mask[r * C + c])",
                             "for (int64_t c = C - 1; c >= 0; --c) {\n            if (!mask[r * C + c])"),
    "pack_block_stride": ("memcpy(dst + (int64_t)i * b_c * es, src",
                          "memcpy(dst + (int64_t)i * b_r * es, src"),
    "row_ptr_shifted": ("row_ptr[r + 1] = (int32_t)p;", "row_ptr[r + 1] = (int32_t)p - (r > 0);"),
    "unpack_wrong_column": ("char* dst = (char*)W_out + ((r * b_r + i) * ldw + c * b_c) * es;",
                            "char* dst = (char*)W_out + ((r * b_r + i) * ldw + c * b_r) * es;"),
    "gelu_tanh_form": ("0.5 * v * (1.0 + erf(v / sqrt(2.0)))",
                       "0.5 * v * (1.0 + tanh(0.7978845608028654 * (v + 0.044715 * v * v * v)))"),
    "gelu_wrong_scale": ("erf(v / sqrt(2.0))", "erf(v / 2.0)"),
    "f16_subnormal_scale": ("ldexp((double)f, -24)", "ldexp((double)f, -25)"),
    "f16_exponent_bias": ("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(1024 + f), e - 24)"),
    "bf16_shift": ("uint32_t u = (uint32_t)b << 16;", "uint32_t u = (uint32_t)b << 15;"),
    "score_abs_dropped": ("s += fabs(w * dec_one(dtype, G, n * ldg + k));",
                          "s += w * dec_one(dtype, G, n * ldg + k);"),
    "score_grid_transposed": ("scores[r * C + c] = G ? s / (double)(b_r * b_c) : s;",
                              "scores[c * R + r] = G ? s / (double)(b_r * b_c) : s;"),
    "score_last_column_dropped": ("for (int64_t k = c * b_c; k < (c + 1) * b_c; ++k) {",
                                  "for (int64_t k = c * b_c; k < (c + 1) * b_c - 1; ++k) {"),
    "score_not_averaged": ("scores[r * C + c] = G ? s / (double)(b_r * b_c) : s;",
                           "scores[r * C + c] = s;"),
    "keep_count_floor": ("return ((100 - (int64_t)sparsity_pct) * n_blocks + 99) / 100;",
                         "return ((100 - (int64_t)sparsity_pct) * n_blocks) / 100;"),
    "topk_ties_to_higher": ("return i < j ? -1 : (i > j ? 1 : 0);",
                            "return i < j ? 1 : (i > j ? -1 : 0);"),
    "gradx_mask_ignored": (
        "Wd[n * K + k] = mask[(n / b_r) * C + (k / b_c)] ? dec_one(dtype, W, n * ldw + k) : 0.0;",
        "Wd[n * K + k] = dec_one(dtype, W, n * ldw + k);"),
    "gradx_rows_reversed": ("const double* wn = j->Wd + n * j->K;",
                            "const double* wn = j->Wd + (j->N - 1 - n) * j->K;"),
    "gradx_sign_flipped": ("out[k] += g * wn[k];", "out[k] -= g * wn[k];"),
    "gradw_block_transposed": ("out[i * b_c + j] += g[i] * x[j];", "out[j * b_r + i] += g[i] * x[j];"),
    "gradw_last_token_dropped": ("for (int64_t m = 0; m < M; ++m) {\n                    for (int i = 0;",
                                 "for (int64_t m = 0; m < M - 1; ++m) {\n                    for (int i = 0;"),
    "gradw_wrong_g_stride": ("g[i] = dec_one(dtype, G, m * ldg + r * b_r + i);",
                             "g[i] = dec_one(dtype, G, m * ldg + r * b_c + i);"),
    "gradw_x_from_g": ("x[j] = dec_one(dtype, X, m * ldx + c * b_c + j);",
                       "x[j] = dec_one(dtype, G, m * ldg + c * b_c + j);"),
    "gradb_first_row_dropped": ("for (int64_t m = 0; m < M; ++m)\n            s += dec_one(dtype, G, m * ldg + n);",
                                "for (int64_t m = 1; m < M; ++m)\n            s += dec_one(dtype, G, m * ldg + n);"),
    "delta_half_dropped": ("delta[i] = lin + 0.5 * (kappa * sq", "delta[i] = lin + (kappa * sq"),
    "delta_change_sign": (": -dec_one(dtype, W, n * ldw + k);", ": dec_one(dtype, W, n * ldw + k);"),
    "delta_kept_blocks": ("? 0.0 : -dec_one(dtype, W, n * ldw + k);",
                          "? -dec_one(dtype, W, n * ldw + k) : 0.0;"),
    "delta_kappa_dropped": ("0.5 * (kappa * sq +", "0.5 * (0.0 * sq +"),
    "delta_fisher_not_averaged": ("fisher / (double)n_samples", "fisher"),
    "delta_linear_term_dropped": ("lin += dec_one(dtype, grad, e) * dw[e];", "lin += 0.0;"),
    "delta_l2_ranking": ("lpvo_block_scores(dtype, W, ldw, grad, K, N, K, b_r, b_c, scores)",
                         "lpvo_block_scores(dtype, W, ldw, NULL, K, N, K, b_r, b_c, scores)"),
    "topk_keeps_lowest": ("    if (si > sj)\n        return -1;\n    if (si < sj)\n        return 1;",
                          "    if (si > sj)\n        return 1;\n    if (si < sj)\n        return -1;"),
}

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
from pins import ALL_PINS
orc = oracle.Oracle({lib!r})
for pin in ALL_PINS:
    try:
        pin(orc)
    except AssertionError as e:
        print("CAUGHT", pin.__name__)
        sys.exit(0)
print("MISSED")
sys.exit(3)
"""


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, source):
    old, new = MUTANTS[name]
    assert source.count(old) >= 1, "mutation site for %s not found in the oracle" % name
    mutated = source.replace(old, new, 1)
    d = tempfile.mkdtemp(prefix="lpvo_mut_")
    try:
        src = os.path.join(d, "lpv_oracle.c")
        with open(src, "w") as f:
            f.write(mutated)
        shutil.copy(HDR, d)
        lib = os.path.join(d, "liblpv_oracle.so")
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fPIC", "-shared",
                               "-pthread", src, "-o", lib, "-lm"])
        code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
        p = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                           timeout=300)
        # a crash (negative return code) also means the mistake did not go unnoticed
        assert p.returncode != 3, "mutant %s passed every pin:\n%s%s" % (name, p.stdout, p.stderr)
        assert "ModuleNotFoundError" not in p.stderr and "ImportError" not in p.stderr, p.stderr
        assert ("CAUGHT" in p.stdout or p.returncode < 0
                or "Error" in p.stderr), (p.returncode, p.stdout, p.stderr)
    finally:
        shutil.rmtree(d, ignore_errors=True)
