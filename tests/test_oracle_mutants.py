"""Mutation check of the oracle's pins.

Each case plants one plausible mistake in a temporary copy of oracle.c
(a dropped term, a wrong index or sign, a reversed tie-break, a transposed
layout offset, a missing normalisation), compiles it, and runs the pin suite
(tests/test_oracle.py) against it in a subprocess.  The suite must fail for
every mutant; the unmodified oracle must pass.  All of this runs on the CPU.
"""
import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = {
    "tie_break_reversed": ("return (a->j > b->j) - (a->j < b->j);",
                           "return (a->j < b->j) - (a->j > b->j);"),
    "keeps_smallest_scores": ("if (a->s > b->s) return -1;\n  if (a->s < b->s) return 1;",
                              "if (a->s > b->s) return 1;\n  if (a->s < b->s) return -1;"),
    "dot_drops_channel_0": ("for (int i = 0; i < d; ++i) s += a[i] * b[i];",
                            "for (int i = 1; i < d; ++i) s += a[i] * b[i];"),
    "gqa_head_map_modulo": ("int g = h / G;", "int g = h % p->Hkv;"),
    "softmax_not_normalised": ("double w = z[t] / Z;", "double w = z[t];"),
    "softmax_scale_dropped": ("z[t] = scale * dot(qbuf, kbuf, d);", "z[t] = dot(qbuf, kbuf, d);"),
    "budget_rounds_down": ("floor(x + 0.5)", "floor(x)"),
    "budget_no_lower_clamp": ("if (k < 1.0) k = 1.0;", ""),
    "group_sum_keeps_last_head": ("s += dot(qbuf, kbuf, p->d);", "s = dot(qbuf, kbuf, p->d);"),
    "paged_slot_off_by_one": ("int64_t slot = j % c->page_size;",
                              "int64_t slot = (j + 1) % c->page_size;"),
    "bf16_decoded_with_wrong_shift": ("uint32_t u = (uint32_t)((const uint16_t *)base)[off] << 16;",
                                      "uint32_t u = (uint32_t)((const uint16_t *)base)[off] << 15;"),
    "indices_left_in_score_order": ("qsort(idx, (size_t)k, sizeof(int32_t), by_int32_asc);", ""),
    "value_row_from_key_cache": ("load_vec(p->V->data, p->V->dtype, cache_row_offset(p->V,",
                                 "load_vec(p->K->data, p->K->dtype, cache_row_offset(p->K,"),
    "weights_squared": ("if (omega) z[t] *= (double)omega[t];",
                        "if (omega) z[t] *= (double)omega[t] * (double)omega[t];"),
    "weights_ignored": ("if (omega) z[t] *= (double)omega[t];", "if (omega) z[t] *= 1.0;"),
    "forced_sinks_compete_for_budget": ("int rc = oracle_select_row(scores + ns, mid, kh, kh, idx + ns, tau);",
                                        "int rc = oracle_select_row(scores, mid, kh, kh, idx + ns, tau);"),
    "local_window_off_by_one": ("idx[ns + kh + t] = (int32_t)(L - nl + t);",
                                "idx[ns + kh + t] = (int32_t)(L - nl + t - 1);"),
    "label_channel_ignored": ("for (int c = 0; c < p->nlab; ++c) s += qbuf[ch[c]] * kbuf[c];",
                              "for (int c = 0; c < p->nlab; ++c) s += qbuf[c] * kbuf[c];"),
    "label_channels_of_head_0": ("const int32_t *ch = p->channels + (int64_t)g * p->nlab;",
                                 "const int32_t *ch = p->channels;"),
    "row_scores_skip_last_position": ("for (int64_t j = 0; j < L; ++j) {\n    double s = 0.0;\n    if (p->lab)",
                                      "for (int64_t j = 0; j + 1 < L; ++j) {\n    double s = 0.0;\n    if (p->lab)"),
}


def _run_suite(lib_path):
    env = dict(os.environ, ORACLE_LIB_OVERRIDE=lib_path, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    return r.returncode, r.stdout[-2000:]


def _build(src_text, out_dir, name):
    c = os.path.join(out_dir, name + ".c")
    so = os.path.join(out_dir, name + ".so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-o", so, c, "-lm"],
                   check=True, capture_output=True)
    return so


def test_every_mutant_fails_the_pins():
    src = open(SRC).read()
    for name, (old, new) in MUTANTS.items():
        assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    with tempfile.TemporaryDirectory() as tmp:
        libs = {"unmodified": _build(src, tmp, "unmodified")}
        for name, (old, new) in MUTANTS.items():
            libs[name] = _build(src.replace(old, new), tmp, name)
        with cf.ThreadPoolExecutor(max_workers=4) as ex:
            results = dict(zip(libs, ex.map(_run_suite, libs.values())))
    rc, log = results.pop("unmodified")
    assert rc == 0, "the unmodified oracle must pass its pins:\n" + log
    survivors = [n for n, (rc, _) in results.items() if rc == 0]
    assert not survivors, f"mutants not caught by any pin: {survivors}"
