"""Planted mistakes in the oracle must be caught by its pins.

Each mutant is a copy of the oracle source with one plausible slip (a dropped
term, a flipped sign, a wrong index or condition -- at every place the
mutated line occurs), compiled on the CPU into a temporary library.  The pins of tests/oracle_pins.py are run against it and at
least one must fail; otherwise the pins would not be strong enough to trust
the oracle as the parity reference.
"""
import os
import subprocess

import pytest

from oracle import oracle as O
from tests import oracle_pins as P

MUTANTS = {
    "step_ahead_plus": ("xh[(int64_t)k * d_pad + j] = x[j] - e[", "xh[(int64_t)k * d_pad + j] = x[j] + e["),
    "drop_local_error": ("ek[j] = fmaf(lr, gk[j], ek[j]);", "ek[j] = fmaf(lr, gk[j], 0.0f);"),
    "lr_dropped": ("ek[j] = fmaf(lr, gk[j], ek[j]);", "ek[j] = gk[j] + ek[j];"),
    "sign_zero_minus": ("return v >= 0.0f ? 1 : 0;", "return v > 0.0f ? 1 : 0;"),
    "scale_wrong_count": ("double mean = S64 / (double)n;", "double mean = S64 / (double)(n + 1);"),
    "residual_plus": ("err[i] = v[i] - message_value(scale, bit);", "err[i] = v[i] + message_value(scale, bit);"),
    "drop_server_error": ("e_srv[off[l] + i] = e_srv[off[l] + i] + a;", "e_srv[off[l] + i] = a;"),
    "reupdate_plus": ("x[off[l] + i] = x[off[l] + i] - message_value(srv_scales[l], bit);",
                      "x[off[l] + i] = x[off[l] + i] + message_value(srv_scales[l], bit);"),
    "sc_plus": ("x[off[l] + i] = x[off[l] + i] - a;", "x[off[l] + i] = x[off[l] + i] + a;"),
    "average_when_t_divisible": ("(t + 1) % period == 0", "t % period == 0"),
    "server_mean_wrong_k": ("float a = (float)(acc / (double)K);", "float a = (float)(acc / (double)(K + 1));"),
    "error_mean_wrong_k": ("float mean = (float)(acc / (double)K);", "float mean = (float)(acc / (double)(K + 1));"),
    "bit_index_shift": ("return (int)((words[off / 64 + i / 64] >> (i % 64)) & 1u);",
                        "return (int)((words[off / 64 + i / 64] >> ((i + 1) % 64)) & 1u);"),
    "l1_rounds_not_floors": ("S += (u128)scaled;", "S += (u128)(scaled + 0.5);"),
    "decode_swapped": ("return bit ? scale : -scale;", "return bit ? -scale : scale;"),
    "worker_stride": ("float* ek = e + (int64_t)k * d_pad;", "float* ek = e + (int64_t)(K - 1 - k) * d_pad;"),
    "mismatch_drops_server_error": ("double u = (e_srv != NULL ? (double)e_srv[j] : 0.0) + ebar;",
                                    "double u = ebar;"),
    "mismatch_mean_not_divided": ("double ebar = sum / (double)K;", "double ebar = sum;"),
    "mismatch_saef_not_divided": ("saef[l] = b / (double)K;", "saef[l] = b;"),
    "mismatch_sign": ("double dk = u - (double)e[", "double dk = u + (double)e["),
    "mismatch_ef_not_squared": ("a += u * u;", "a += fabs(u);"),
    "ef_variant_steps_ahead": ("if (variant == 1) /* SAEF: one step ahead */",
                               "if (variant >= 0) /* SAEF: one step ahead */"),
    "topk_keeps_smallest": ("if (ma > mb) return -1;\n    if (ma < mb) return 1;",
                            "if (ma < mb) return -1;\n    if (ma > mb) return 1;"),
    "topk_tie_high_index": ("return (a < b) ? -1 : (a > b) ? 1 : 0;",
                            "return (a < b) ? 1 : (a > b) ? -1 : 0;"),
    "topk_error_keeps_value": ("err[i] = v[i] - c;", "err[i] = v[i];"),
    "topk_rank_shifted": ("rank[off / 64 + w] = (uint32_t)count;",
                          "rank[off / 64 + w] = (uint32_t)(count > 0 ? count - 1 : 0);"),
    "topk_reupdate_plus": ("applied_to[i] = applied_to[i] - c;", "applied_to[i] = applied_to[i] + c;"),
    "topk_mean_wrong_k": ("mean[j] = (float)(acc[j] / (double)K);",
                          "mean[j] = (float)(acc[j] / (double)(K + 1));"),
    "topk_value_magnitude": ("vals[count++] = v[i];", "vals[count++] = fabsf(v[i]);"),
    "topk_momentum_dropped": ("mk[j] = fmaf(mu, mk[j], gk[j]);\n                    delta[j]",
                              "mk[j] = gk[j];\n                    delta[j]"),
    "momentum_dropped": ("mk[j] = fmaf(mu, mk[j], gk[j]);", "mk[j] = gk[j];"),
    "momentum_swapped": ("mk[j] = fmaf(mu, mk[j], gk[j]);", "mk[j] = fmaf(mu, gk[j], mk[j]);"),
    "momentum_lr_dropped": ("ek[j] = fmaf(lr, mk[j], ek[j]);", "ek[j] = mk[j] + ek[j];"),
    "step_ahead_skips_worker": ("for (int32_t k = 0; k < K; ++k)\n        for (int32_t l = 0; l < L; ++l)\n            for (int64_t i = 0; i < n[l]; ++i) {\n                int64_t j = off[l] + i;\n                /* x^(k)",
                                "for (int32_t k = 0; k < K - (K > 1); ++k)\n        for (int32_t l = 0; l < L; ++l)\n            for (int64_t i = 0; i < n[l]; ++i) {\n                int64_t j = off[l] + i;\n                /* x^(k)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(O.SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    msrc = tmp_path / "saef_oracle.c"
    msrc.write_text(src.replace(old, new))
    (tmp_path / "saef_oracle.h").write_text(open(os.path.join(O.HERE, "saef_oracle.h")).read())
    lib = str(tmp_path / f"liboracle_{name}.so")
    O.build(src=str(msrc), out=lib, werror=False)
    caught = []
    for pin in P.QUICK_PINS:
        try:
            pin(lib)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutant {name}"
