"""Planted mistakes in the oracle must each be caught by at least one pin.

Each mutant is the oracle's C source with one plausible slip (a wrong group map, a transposed
index, a dropped term, a scatter turned into a store at the wrong place ...), compiled on the CPU
into a temporary library.  Every planted access stays in bounds for the pins' shapes.
"""
import os

import pytest

import oracle
import oracle_pins as P

SRC = open(oracle.SRC).read()

MUTANTS = {
    "group_map_mod": ("const int64_t g = l / G;                 /* g(l)", "const int64_t g = l % (L / G); /* g(l)"),
    "idx_transposed_fwd": ("const int64_t f = idx[g * F_in + t];\n                z +=",
                           "const int64_t f = idx[t * (L / G) + g];\n                z +="),
    "bias_dropped": ("double z = bias ? (double)bias[l] : 0.0;\n            for (int64_t t = 0; t < F_in; ++t) {",
                     "double z = 0.0;\n            for (int64_t t = 0; t < F_in; ++t) {"),
    "fwd_last_slot_dropped": ("for (int64_t t = 0; t < F_in; ++t) {\n                const int64_t f = idx[g * F_in + t];\n                z +=",
                              "for (int64_t t = 0; t + 1 < F_in; ++t) {\n                const int64_t f = idx[g * F_in + t];\n                z +="),
    "bwd_w_slot_not_feature": ("s += ld(dY, b * L + l, dtype) * ld(X, b * F_s + f, dtype);",
                               "s += ld(dY, b * L + l, dtype) * ld(X, b * F_s + t, dtype);"),
    "bwd_w_sign": ("s += ld(dY, b * L + l, dtype) * ld(X, b * F_s + f, dtype);",
                   "s -= ld(dY, b * L + l, dtype) * ld(X, b * F_s + f, dtype);"),
    "dbias_wrong_row": ("for (int64_t b = 0; b < B; ++b) s += ld(dY, b * L + l, dtype);",
                        "for (int64_t b = 0; b < B; ++b) s += ld(dY, l, dtype);"),
    "bwd_x_scatter_to_slot": ("row[idx[g * F_in + t]] += d * ld(W, l * F_in + t, dtype);",
                              "row[t] += d * ld(W, l * F_in + t, dtype);"),
    "bwd_x_dy_transposed": ("const double d = ld(dY, b * L + l, dtype);",
                            "const double d = ld(dY, l * B + b, dtype);"),
    "bwd_x_group_of_slot": ("row[idx[g * F_in + t]] += d * ld(W, l * F_in + t, dtype);",
                            "row[idx[g * F_in + t]] += d * ld(W, g * F_in + t, dtype);"),
    "head_w_transposed": ("z += ld(X, b * F_s + f, dtype) * ld(Wh, h * F_s + f, dtype);",
                          "z += ld(X, b * F_s + f, dtype) * ld(Wh, f * H + h, dtype);"),
    "head_dw_dy_transposed": ("s += ld(dYh, b * H + h, dtype) * ld(X, b * F_s + f, dtype);",
                              "s += ld(dYh, h * B + b, dtype) * ld(X, b * F_s + f, dtype);"),
    "head_dx_w_transposed": ("s += ld(dYh, b * H + h, dtype) * ld(Wh, h * F_s + f, dtype);",
                             "s += ld(dYh, b * H + h, dtype) * ld(Wh, f * H + h, dtype);"),
    "bce_target_added": ("if (c >= 0 && c < N) dY[b * N + c] = sigmoid(Z[b * N + c]) - 1.0;",
                         "if (c >= 0 && c < N) dY[b * N + c] -= 1.0;"),
    "bce_sigmoid_sign": ("static double sigmoid(double z) { return 1.0 / (1.0 + exp(-z)); }",
                         "static double sigmoid(double z) { return 1.0 / (1.0 + exp(z)); }"),
    "bce_at_target_ignored": ("if (pos[bs[i] * P + p] == ns[i]) y = 1.0;", "if (pos[bs[i] * P + p] == ns[i]) y = 0.0;"),
    "sgd_momentum_dropped": ("m[i] = momentum * m[i] + (grad[i] + weight_decay * w);",
                             "m[i] = (grad[i] + weight_decay * w);"),
    "sgd_decay_sign": ("m[i] = momentum * m[i] + (grad[i] + weight_decay * w);",
                       "m[i] = momentum * m[i] + (grad[i] - weight_decay * w);"),
    "sgd_step_uses_grad": ("W_next[i] = w - lr * m[i];", "W_next[i] = w - lr * grad[i];"),
    "rewire_ties_reversed": ("return (x->i > y->i) - (x->i < y->i);", "return (x->i < y->i) - (x->i > y->i);"),
    "rewire_largest": ("if (x->s < y->s) return -1;\n    if (x->s > y->s) return 1;",
                       "if (x->s > y->s) return -1;\n    if (x->s < y->s) return 1;"),
    "rewire_m_ceil": ("(int64_t)floor((double)K * (double)F * rho)", "(int64_t)ceil((double)K * (double)F * rho)"),
    "rewire_kept_not_excluded": ("if (!mask[k * F + j]) { used[idx[k * F + j]] = 1; ++n_used; }",
                                 "if (!mask[k * F + j]) { ++n_used; }"),
    "rewire_column_not_moved": ("tmp[p] = ld(W, l * F + j, dtype);", "tmp[p] = ld(W, l * F + p, dtype);"),
    "group_least_similar": ("if (x->sim != y->sim) return x->sim > y->sim ? -1 : 1;",
                            "if (x->sim != y->sim) return x->sim < y->sim ? -1 : 1;"),
    "group_assign_argmin": ("if (best < 0 || v > bv) { bv = v; best = c; }", "if (best < 0 || v < bv) { bv = v; best = c; }"),
    "group_assign_raw_dot": ("const double v = (double)dot / cn[c];", "const double v = (double)dot;"),
    "group_centre_int8": ("memcpy(cs + c * D, sum, (size_t)D * sizeof(int64_t));\n            cn[c] = nrm;",
                          "for (int64_t d = 0; d < D; ++d) cs[c * D + d] = (int64_t)rint(127.0 * (double)sum[d] / nrm);\n"
                          "            cn[c] = exact_norm(cs + c * D, D);"),
    "group_sim_raw_dot": ("cand[nc].sim = (double)dot8(e, E + (int64_t)s * D, D) / sqrt((double)(ni * ns));",
                          "cand[nc].sim = (double)dot8(e, E + (int64_t)s * D, D) + 0.0 * (double)(ni * ns);"),
    "group_seed_index": ("const int32_t s = a[r];", "const int32_t s = a[nu - 1 - r];"),
    "group_seed_tie_not_lower": ("return (x->id > y->id) - (x->id < y->id);\n}\n\nstatic int by_id",
                                 "return (x->id < y->id) - (x->id > y->id);\n}\n\nstatic int by_id"),
    "rewire_reinit_zero": ("v = (double)((float)((int64_t)(2 * n) - (1LL << 24)) * scale);", "v = 0.0 * (double)n;"),
    "rewire_reinit_one_sided": ("(float)((int64_t)(2 * n) - (1LL << 24)) * scale", "(float)((int64_t)n) * scale"),
    "rewire_reinit_scale_1_over_F": ("const float a = (float)(1.0 / sqrt((double)F));", "const float a = (float)(1.0 / (double)F);"),
    "group_centre_negated": ("for (int64_t d = 0; d < D; ++d) sum[d] += E[l * D + d]; }",
                             "for (int64_t d = 0; d < D; ++d) sum[d] -= E[l * D + d]; }"),
    "bf16_decode_shift": ("uint32_t u = ((uint32_t)((const uint16_t *)p)[i]) << 16;",
                          "uint32_t u = ((uint32_t)((const uint16_t *)p)[i]) << 15;"),
}


def _caught(o):
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, ValueError, FloatingPointError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert SRC.count(old) >= 1, f"mutation site for {name} not found"
    src = tmp_path / f"{name}.c"
    src.write_text(SRC.replace(old, new, 1))
    lib = oracle.build(str(src), str(tmp_path / f"lib{name}.so"))
    failed = _caught(oracle.Oracle(lib))
    assert failed, f"planted mistake {name} passed every pin"
