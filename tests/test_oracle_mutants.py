"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of ``oracle/vdref.c`` (never in
the oracle itself), builds it with gcc into a temporary directory and runs the
pin checks of ``oracle_pins.py`` against it in a child process.  Every mutant
must fail at least one pin; a mutant that passes would mean the pins cannot
tell that mistake from the paper's definition.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "vdref.c")

# (name, text in vdref.c, replacement)
MUTANTS = [
    ("mean_divides_by_n_minus_1", "mean[c] = sum / (double)n;",
     "mean[c] = sum / (double)(n - 1);"),
    ("mean_skips_last_row", "for (int64_t i = 0; i < n; ++i)\n            sum +=",
     "for (int64_t i = 0; i < n - 1; ++i)\n            sum +="),
    ("l2_adds_mean", "double diff = get_elem(v, dtype, j * row_stride + c) - mean[c];",
     "double diff = get_elem(v, dtype, j * row_stride + c) + mean[c];"),
    ("l2_returns_square", "acc += diff * diff;\n            }\n            scores[j] = sqrt(acc);",
     "acc += diff * diff;\n            }\n            scores[j] = acc;"),
    ("norm_returns_square", "acc += x * x;\n            }\n            scores[j] = sqrt(acc);",
     "acc += x * x;\n            }\n            scores[j] = acc;"),
    ("dir_sign_flipped", "scores[j] = 1.0 - cosv;", "scores[j] = 1.0 + cosv;"),
    ("dir_zero_guard_cos_one", "double cosv = denom > 0.0 ? dot / denom : 0.0;",
     "double cosv = denom > 0.0 ? dot / denom : 1.0;"),
    ("dir_uses_squared_norm", "double denom = sqrt(vn2) * mean_norm;",
     "double denom = vn2 * mean_norm;"),
    ("tie_keeps_higher_index", "if (a->s < b->s)\n        return 1;\n    if (a->j < b->j)\n        return -1;",
     "if (a->s < b->s)\n        return 1;\n    if (a->j < b->j)\n        return 1;"),
    ("keeps_lowest_scores", "if (a->s > b->s)\n        return -1;\n    if (a->s < b->s)\n        return 1;",
     "if (a->s > b->s)\n        return 1;\n    if (a->s < b->s)\n        return -1;"),
    ("keeps_one_too_few", "by_score_desc_index_asc);\n    for (int64_t j = 0; j < n; ++j)\n        keep[j] = 0;\n    for (int64_t r = 0; r < N; ++r)",
     "by_score_desc_index_asc);\n    for (int64_t j = 0; j < n; ++j)\n        keep[j] = 0;\n    for (int64_t r = 0; r < N - 1; ++r)"),
    ("movers_start_past_budget", "int64_t next_mover = N;", "int64_t next_mover = N + 1;"),
    ("pos_not_moved", "pos[hole] = pos[next_mover];", "pos[hole] = pos[hole];"),
    ("k_not_moved", "if (k)\n            copy_row(k,", "if (0)\n            copy_row(k,"),
    ("bf16_wrong_shift", "uint32_t w = ((uint32_t)bits) << 16;", "uint32_t w = ((uint32_t)bits) << 15;"),
    ("unit_offset_wrong", "char *vu = (char *)v + (size_t)(u * cap * d) * es;",
     "char *vu = (char *)v + (size_t)(u * d) * es;"),
    ("sigma_sample_std", "*sigma = sqrt(var / (double)n);", "*sigma = sqrt(var / (double)(n - 1));"),
    ("dispersion_squared", "dist[i] = sqrt(acc);", "dist[i] = acc;"),
    ("bos_mean_includes_bos", "for (int64_t i = 1; i < n; ++i)\n                m +=",
     "for (int64_t i = 0; i < n; ++i)\n                m +="),
    ("sigma_k_of_v", "dispersion(k, dtype, n, d, row_stride, &out[2], &out[0]);",
     "dispersion(v, dtype, n, d, row_stride, &out[2], &out[0]);"),
    ("attn_no_max_shift", "\n        w[j] = exp(w[j] - top);", "\n        w[j] = exp(w[j]);"),
    ("attn_ignores_scale", "\n        w[j] = scale * dot;", "\n        w[j] = dot;"),
    ("attn_divides_by_n", "out[c] = acc / den;", "out[c] = acc / (double)n;"),
    ("attn_same_key_for_all", "dot += q[c] * get_elem(k, dtype, j * row_stride + c);",
     "dot += q[c] * get_elem(k, dtype, c);"),
    ("attn_values_from_keys", "acc += w[j] * get_elem(v, dtype, j * row_stride + c);",
     "acc += w[j] * get_elem(k, dtype, j * row_stride + c);"),
    ("key_side_scores_values", "vdref_score(key_side ? ku : vu, dtype",
     "vdref_score(vu, dtype"),
    ("key_norm_keeps_largest", "if (variant == VDREF_KEY_NORM)\n            vdref_select_smallest",
     "if (0)\n            vdref_select_smallest"),
    ("key_variant_maps_to_next_form", "variant -= VDREF_KEY_L2;", "variant -= VDREF_KEY_L2 - 1;"),
    ("smallest_tie_keeps_higher_index",
     "if (a->s > b->s)\n        return 1;\n    if (a->j < b->j)\n        return -1;",
     "if (a->s > b->s)\n        return 1;\n    if (a->j < b->j)\n        return 1;"),
    ("fastcaote_ratio_dropped", "? a[j] / (1.0 - a[j]) * dist[j]", "? a[j] * dist[j]"),
    ("fastcaote_heads_summed", "a[j] += w[j] / den / (double)G;", "a[j] += w[j] / den;"),
    ("fastcaote_no_max_shift", "w[j] = exp(w[j] - top);\n            den += w[j];",
     "w[j] = exp(w[j]);\n            den += w[j];"),
    ("fastcaote_ignores_scale", "w[j] = scale * dot;\n            if (w[j] > top)\n                top = w[j];\n        }\n        double den",
     "w[j] = dot;\n            if (w[j] > top)\n                top = w[j];\n        }\n        double den"),
]


def _build_and_check(name, old, new, tmp):
    with open(SRC) as fh:
        src = fh.read()
    assert src.count(old) == 1, f"mutation site of {name} not unique in vdref.c"
    path_c = os.path.join(tmp, f"{name}.c")
    path_so = os.path.join(tmp, f"lib{name}.so")
    with open(path_c, "w") as fh:
        fh.write(src.replace(old, new))
    subprocess.run(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", path_so,
                    path_c, "-lm"], check=True, capture_output=True)
    r = subprocess.run([sys.executable, os.path.join(HERE, "oracle_pins.py"), path_so,
                        "--fail-fast"], capture_output=True, text=True, timeout=300,
                       env={**os.environ, "OMP_NUM_THREADS": "1"})
    return r.returncode, r.stdout[-400:] + r.stderr[-400:]


def test_every_mutant_fails_a_pin():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
            futs = {m[0]: ex.submit(_build_and_check, *m, tmp) for m in MUTANTS}
            results = {k: f.result() for k, f in futs.items()}
    survivors = {k: out for k, (rc, out) in results.items() if rc == 0}
    assert not survivors, f"mutants not caught by any pin: {survivors}"


def test_unmutated_build_passes():
    with tempfile.TemporaryDirectory() as tmp:
        rc, out = _build_and_check("identity", "#define VDREF_OK 0", "#define VDREF_OK 0", tmp)
    assert rc == 0, out
