"""The pins are strong enough to catch plausible mistakes: each case below plants
one error in a temporary copy of the oracle source, builds it, and requires at
least one pin to fail against that build (CPU only; the real oracle is untouched)."""
import os
import subprocess

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "ress_oracle.c")

MUTATIONS = {
    "restore_gain_sign": ("dG = -2.0 * dkMg + s[k] * s[k];", "dG = 2.0 * dkMg + s[k] * s[k];"),
    "drop_gain_no_s2": ("dG = 2.0 * dkMg + s[k] * s[k];", "dG = 2.0 * dkMg;"),
    "key_no_renorm": ("key[j] = s[j] / (den > eps ? den : eps);", "key[j] = s[j];"),
    "tie_to_higher_index": ("return (a->j < b->j) ? -1 : (a->j > b->j);",
                            "return (a->j > b->j) ? -1 : (a->j < b->j);"),
    "schedule_off_by_one": ("ldexp(1.0, -(r + 1))", "ldexp(1.0, -r)"),
    "no_track_best": ("if (maximise ? J > Jb : J < Jb) {", "if (1) {"),
    "max_keeps_smallest_J": ("if (maximise ? J > Jb : J < Jb) {", "if (J < Jb) {"),
    "max_without_gain_flip": ("            for (int j = 0; j < nkb; ++j) dJ[j] = -dJ[j];\n", "            ;\n"),
    "probability_ranks_by_key": ("rank[j] = criterion == 1 ? P[j] :", "rank[j] = criterion == 1 ? key[j] :"),
    "cdf_one_block_too_many": ("            while (n < cnt && mass < cdf_tau) mass += it[n++].v;\n",
                               "            while (n < cnt && mass < cdf_tau) mass += it[n++].v;\n            if (n < cnt) ++n;\n"),
    "cdf_ignores_forced_mass": ("                    mass += P[j];\n", ""),
    "drift_without_prob": ("g[d] += P[j] * (vbar_i[d] - vbar[(size_t)j * D + d]);",
                           "g[d] += (vbar_i[d] - vbar[(size_t)j * D + d]);"),
    "pooled_logit_unscaled": ("    double scale = 1.0 / sqrt((double)D);\n    for (int j = 0; j < nkb; ++j) {",
                              "    double scale = 1.0;\n    for (int j = 0; j < nkb; ++j) {"),
    "pool_divides_by_block": ("sum / (double)(hi - lo)", "sum / (double)b"),
    "attn_unscaled": ("lg[ns] = dot * scale;", "lg[ns] = dot;"),
    "mass_sign": ("double K = 1.0 - mass;", "double K = 1.0 + mass;"),
    "margin_always_zero": ("    *margin = mrg;\n", "    *margin = 0.0;\n"),
    "margin_ignores_rounds": ("        mrg = min2(mrg, gap_r / jden);\n        mrg = min2(mrg, gap_d / jden);\n", ""),
    "margin_ignores_track_best": (
        "        if (memcmp(inD, best, nkb) != 0) mrg = min2(mrg, fabs(J - Jb) / (Jb > 0.0 ? Jb : 1e-300));\n", ""),
    "margin_initial_unnormalised": ("gap / (vmax > 0.0 ? vmax : 1e-300)", "gap"),
    "margin_cdf_ignored": ("                mrg = min2(mrg, min2(mass - cdf_tau, cdf_tau - before) / cdf_tau);\n", ""),
    "drop_gain_uses_plus_u": ("dG = 2.0 * dkMg + s[k] * s[k];\n            u = -P[k];",
                              "dG = 2.0 * dkMg + s[k] * s[k];\n            u = P[k];"),
}


def _build_mutant(tmp_path, name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib_{name}.so"
    subprocess.run(["gcc", "-std=c99", "-O1", "-fopenmp", "-fPIC", "-shared", str(path), "-o", str(lib),
                    "-lm"], check=True)
    return str(lib)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch(name, tmp_path):
    lib = _build_mutant(tmp_path, name)
    caught = []
    with oracle.use_library(lib):
        for check in pins.ALL:
            try:
                check()
            except AssertionError:
                caught.append(check.__name__)
    assert caught, f"no pin caught the planted error {name}"
    print(name, "caught by", caught)
