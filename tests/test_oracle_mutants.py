"""Planted mistakes in the oracle must each fail at least one pin.

Every mutant is a copy of oracle/oracle.c with one plausible mistake (a dropped term, a
wrong sign, a transposed operand, a flipped tie rule, a missing normalisation, an
off-by-one), compiled with gcc into a temporary library.  The real oracle is untouched.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "bwd_g_not_subtracted": (
        "for (int32_t e = 0; e < M; ++e) yb[e] = lg[e] * (pbar[e] - gt);",
        "for (int32_t e = 0; e < M; ++e) yb[e] = lg[e] * pbar[e];"),
    "bwd_P_not_normalised": (
        "lg[e] = exp(lg[e] - m[t]) / Z[t];  /* P */",
        "lg[e] = exp(lg[e] - m[t]);  /* P */"),
    "bwd_dz_reads_R2_transposed": (
        "for (int32_t e = 0; e < M; ++e) s += yb[e] * f2[(int64_t)i * M + e];",
        "for (int32_t e = 0; e < M; ++e) s += yb[e] * f2[((int64_t)e * r + i) % ((int64_t)r * M)];"),
    "bwd_dx_drops_last_rank_term": (
        "for (int32_t i = 0; i < r; ++i) s += dzt[i] * f1[(int64_t)c * r + i];",
        "for (int32_t i = 0; i < r - 1; ++i) s += dzt[i] * f1[(int64_t)c * r + i];"),
    "bwd_sparse_term_subtracted": (
        "if (e >= 0 && e < M) yb[e] += dtop[t * k + j];",
        "if (e >= 0 && e < M) yb[e] -= dtop[t * k + j];"),
    "bwd_invalid_id_counted": (
        "if (e >= 0 && e < M) yb[e] += dtop[t * k + j];",
        "if (e >= -1 && e < M) yb[e < 0 ? 0 : e] += dtop[t * k + j];"),
    "bwd_dR2_sparse_at_next_expert": (
        "if (e >= e0 && e < e1) yb[e - e0] += dtop[t * k + j];",
        "if (e + 1 >= e0 && e + 1 < e1) yb[e + 1 - e0] += dtop[t * k + j];"),
    "bwd_dR2_drops_last_token": (
        "for (int64_t t = 0; t < T; ++t) {\n                    const double* zt = zall",
        "for (int64_t t = 0; t < T - 1; ++t) {\n                    const double* zt = zall"),
    "bwd_dR1_uses_z": (
        "acc[(int64_t)(c - c0) * r + i] += xs[c - c0] * dzt[i];",
        "acc[(int64_t)(c - c0) * r + i] += xs[c - c0] * zall[t * r + i];"),
    "stats_no_max_shift_in_Z": (
        "zs += exp(lg[e] - mx);",
        "zs += exp(lg[e]);"),
    "stats_psum_not_normalised": (
        "pb[e] += exp(lg[e] - mx) / zs;",
        "pb[e] += exp(lg[e] - mx);"),
    "stats_max_is_minimum": (
        "mx = lg[e] > mx ? lg[e] : mx;",
        "mx = lg[e] < mx ? lg[e] : mx;"),
    "stats_Z_drops_last_expert": (
        "for (int32_t e = 0; e < M; ++e) zs += exp",
        "for (int32_t e = 0; e < M - 1; ++e) zs += exp"),
    "stats_last_token_block_dropped": (
        "for (int64_t b = 0; b < nb; ++b)\n            for (int32_t e = 0; e < M; ++e) psum[e]",
        "for (int64_t b = 0; b < nb - 1; ++b)\n            for (int32_t e = 0; e < M; ++e) psum[e]"),
    "dispatch_positions_reversed": (
        "    for (int64_t p = 0; p < N; ++p) {\n        const int32_t key = dispatch_key(idx[p], M);",
        "    for (int64_t p = N - 1; p >= 0; --p) {\n        const int32_t key = dispatch_key(idx[p], M);"),
    "dispatch_offsets_inclusive": (
        "for (int32_t e = 0; e <= M; ++e) offsets[e] = start[e];",
        "for (int32_t e = 0; e <= M; ++e) offsets[e] = start[e + 1];"),
    "dispatch_invalid_ids_to_expert_0": (
        "return (e >= 0 && e < M) ? e : M;",
        "return (e >= 0 && e < M) ? e : 0;"),
    "z_drops_last_hidden_term": (
        "for (int32_t j = 0; j < h; ++j) {\n                    const double* r1row",
        "for (int32_t j = 0; j < h - 1; ++j) {\n                    const double* r1row"),
    "logit_drops_last_rank_term": (
        "for (int32_t i = 0; i < r; ++i) {\n                    const double* r2row",
        "for (int32_t i = 0; i < r - 1; ++i) {\n                    const double* r2row"),
    "R2_read_transposed": (
        "logit[e] += z[i] * r2row[e];",
        "logit[e] += z[i] * r2[(int64_t)e * r + i];"),
    "R1_read_transposed": (
        "z[i] += xrow[j] * r1row[i];",
        "z[i] += xrow[j] * r1[((int64_t)i * h + j) % ((int64_t)h * r)];"),
    "selects_smallest": (
        "if (a->value > b->value) return -1;\n    if (a->value < b->value) return 1;",
        "if (a->value > b->value) return 1;\n    if (a->value < b->value) return -1;"),
    "ties_prefer_larger_index": (
        "if (a->expert < b->expert) return -1;\n    if (a->expert > b->expert) return 1;",
        "if (a->expert < b->expert) return 1;\n    if (a->expert > b->expert) return -1;"),
    "softmax_sign_flipped": (
        "gate[j] = exp(work[j].value - top);",
        "gate[j] = exp(top - work[j].value);"),
    "softmax_not_normalised": (
        "for (int32_t j = 0; j < k; ++j) gate[j] /= denom;",
        "for (int32_t j = 0; j < k; ++j) gate[j] /= (denom + 0.0 * gate[j]) * 1.0 + 0.01;"),
    "next_is_kth_itself": (
        "*next = (k < M) ? work[k].value : -INFINITY;",
        "*next = (k < M) ? work[k - 1].value : -INFINITY;"),
    "selection_off_by_one": (
        "idx[j] = work[j].expert;\n        topval[j] = work[j].value;",
        "idx[j] = work[j + (j + 1 < M)].expert;\n        topval[j] = work[j + (j + 1 < M)].value;"),
    "fullrank_drops_last_hidden_term": (
        "for (int32_t j = 0; j < h; ++j) {\n                const double* wrow",
        "for (int32_t j = 0; j < h - 1; ++j) {\n                const double* wrow"),
    "logits_at_drops_last_hidden_term": (
        "for (int32_t i = 0; i < r; ++i) z[i] += xrow[j] * w1[i];",
        "for (int32_t i = 0; i < r; ++i) z[i] += (j + 1 < h) * xrow[j] * w1[i];"),
    "logits_at_wrong_expert_column": (
        "l += z[i] * r2[(int64_t)i * M + e];",
        "l += z[i] * r2[(int64_t)i * M + (e + 1) % M];"),
    "fullrank_logits_at_transposed_W": (
        "const double wv = bf16_bits_to_double(W[(int64_t)q * M + e]);",
        "const double wv = bf16_bits_to_double(W[((int64_t)e * h + q) % ((int64_t)h * M)]);"),
    "histogram_off_by_one": (
        "counts[idx[i]] += 1;",
        "counts[(idx[i] + 1) % M] += 1;"),
}


def _build_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor for %s not found exactly once" % name
    path = tmp_path / (name + ".c")
    path.write_text(src.replace(old, new))
    lib_path = tmp_path / ("lib" + name + ".so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", str(lib_path),
                    str(path), "-lm"], check=True)
    return oracle.load_library(str(lib_path))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    lib = _build_mutant(name, tmp_path)
    failed = []
    for check in oracle_pins.ALL_CHECKS:
        try:
            check(lib=lib)
        except (AssertionError, ValueError):
            failed.append(check.__name__)
    assert failed, "planted mistake %r passed every pin" % name
