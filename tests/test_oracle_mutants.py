"""Each plausible mistake planted in a copy of the oracle fails at least one pin.

The mutants are built from the oracle's C source with one textual change each
and loaded in place of the real oracle for the duration of one check run (CPU
only; the real oracle is restored afterwards).
"""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import oracle_pins as P  # noqa: E402
from oracle import build as obuild  # noqa: E402

MUTANTS = {
    "silu_sign": ("return v / (1.0 + exp(-v));", "return v / (1.0 + exp(v));"),
    "drop_private_slice": ("for (int c = 0; c < h; ++c) out[c] += q[c];",
                           "for (int c = 0; c < h; ++c) out[c] += 0.0 * q[c];"),
    "sigma_missing_down": ("sigma_vec(cfg, b, d);                          /* sigma((A_d)^T v)",
                           "/* sigma((A_d)^T v)"),
    "gelu_unscaled_erf": ("erf(v / sqrt(2.0))", "erf(v)"),
    "rmsnorm_sum_not_mean": ("sqrt(ss / d + OREF_RMS_EPS)", "sqrt(ss + OREF_RMS_EPS)"),
    "cover_one_short": ("if (D >= cfg->top_k_dept) break;", "if (D >= cfg->top_k_dept - 1) break;"),
    "cover_victim_highest_rank": ("for (int r = k - 1; r >= 0 && victim < 0; --r)",
                                  "for (int r = 0; r < k && victim < 0; ++r)"),
    "cover_no_rerank": ("for (int r = 1; r < k; ++r)\n        for (int q = r;",
                        "for (int r = k; r < k; ++r)\n        for (int q = r;"),
    "gate_up_swapped": ("matvec(&s->M[3], i, G, a);", "matvec(&s->M[4], i, G, a);"),
    "tie_break_high_id": ("(la == lb && a < b)", "(la == lb && a > b)"),
    "dept_of_expert_modulo": ("j = i / (cfg->n_experts / cfg->n_depts);",
                              "j = i % cfg->n_depts;"),
    "route_scale_dropped": ("w[r] *= cfg->route_scale;", "w[r] *= 1.0;"),
    "sigmoid_sign": ("w[r] = 1.0 / (1.0 + exp(-(double)l[ids[r]]));",
                     "w[r] = 1.0 / (1.0 + exp((double)l[ids[r]]));"),
    "group_score_min": ("if (l[e] > gs[j]) gs[j] = l[e];", "if (l[e] < gs[j]) gs[j] = l[e];"),
    "bias_ignored": ("l[e] = l[e] + b;", "l[e] = l[e] + 0.0f * b;"),
    "fp8_subnormal_exponent": ("ldexp((double)m / 8.0, -6)", "ldexp((double)m / 8.0, -7)"),
    "fp8_scale_transposed": ("r / 128) * cb + c / 128]", "c / 128) * cb + r / 128]"),
    "softmax_renorm_over_all": ("for (int r = 0; r < k; ++r) den += exp((double)l[ids[r]] - mx);",
                                "for (int e = 0; e < n; ++e) den += exp((double)l[e] - mx);"),
    "shared_expert_dropped": ("yt[c] += o[c];\n    }\n    free(xv);",
                              "yt[c] += 0.0 * o[c];\n    }\n    free(xv);"),
    "dept_bytes_two_matrices": ("int64_t dept = 3 * matrix_bytes(wt, d, h);",
                                "int64_t dept = 2 * matrix_bytes(wt, d, h);"),
    "fp8_scale_bytes_missing": ("if (w_dtype == OREF_FP8) b += ((R + 127) / 128) * ((C + 127) / 128) * 4;",
                                "if (w_dtype == OREF_FP8) b += 0;"),
    "two_stage_dept_weight_one": ("y[(size_t)t * h + c] += Pj * o[c];",
                                  "y[(size_t)t * h + c] += o[c];"),
    "dept_list_descending": ("for (int t = 0; t < T; ++t)\n      for (int r = 0; r < out->tok_ndept[t]; ++r)",
                             "for (int t = T - 1; t >= 0; --t)\n      for (int r = 0; r < out->tok_ndept[t]; ++r)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(os.path.join(obuild.HERE, "deamoe_oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = obuild.build(src=str(path), out=str(tmp_path / "libmutant.so"))
    saved = oracle._lib
    oracle._lib = oracle._open(lib)
    failed = []
    try:
        for check in P.ALL_CHECKS:
            try:
                check()
            except AssertionError:
                failed.append(check.__name__)
                break
    finally:
        oracle._lib = saved
    assert failed, f"no pin catches mutant {name}"
