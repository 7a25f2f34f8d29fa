"""The oracle's pins must catch plausible mistakes.

Each case copies the oracle source, plants one mistake by text substitution,
builds the copy with the host compiler into a temporary directory, and runs
the pin suites against it in a child process; at least one pin must fail.
Nothing here touches the GPU or the HIP library.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "osd_ref.cpp")

MUTATIONS = {
    "residual_without_q": ("double diff = P[(size_t)j] - Q[(size_t)j];",
                           "double diff = P[(size_t)j];"),
    "ratio_inverted": ("ratio = py / qy;", "ratio = qy / py;"),
    "bonus_row_off_by_one": ("b * tstride + (int64_t)kb * V, V);",
                             "b * tstride + (int64_t)(kb - 1) * V, V);"),
    "cdf_non_strict": ("if (C > c) {", "if (C >= c) {"),
    "accept_continues_after_reject": ("                    a = i;\n                    rejected = true;\n                    break;",
                                      "                    a = i;\n                    rejected = true;"),
    "rkl_grad_missing_kl_term": ("(logQ[(size_t)j] - logP[(size_t)j] - D) /",
                                 "(logQ[(size_t)j] - logP[(size_t)j]) /"),
    "jsd_mixture_swapped": ("std::log(wp * P[(size_t)j] + wq * Q[(size_t)j]);",
                            "std::log(wp * Q[(size_t)j] + wq * P[(size_t)j]);"),
    "fkl_grad_missing_tau": ("g[j] = (Q[(size_t)j] - P[(size_t)j]) / tau;",
                             "g[j] = (Q[(size_t)j] - P[(size_t)j]);"),
    "fkl_sign_flipped": ("D += P[(size_t)j] * (logP[(size_t)j] - logQ[(size_t)j]);",
                         "D += P[(size_t)j] * (logQ[(size_t)j] - logP[(size_t)j]);"),
    "verify_temperature_ignored": ("const double T = (double)temperature;\n    const int64_t tstride",
                                   "const double T = 1.0;\n    const int64_t tstride"),
    "tree_temperature_ignored": ("const double T = (double)temperature;\n    const int64_t stride",
                                 "const double T = 1.0;\n    const int64_t stride"),
    "distill_temperature_ignored": ("bool ok = temperature_softmax(t, tau, P, logP) &&\n                      temperature_softmax(s, tau, Q, logQ);",
                                    "bool ok = temperature_softmax(t, 1.0, P, logP) &&\n                      temperature_softmax(s, 1.0, Q, logQ);"),
    "argmax_last_on_ties": ("if (z[j] > bv) {", "if (z[j] >= bv) {"),
    "bf16_round_truncates": ("double r = std::nearbyint(v / q) * q;",
                             "double r = std::trunc(v / q) * q;"),
    "sample_mixture_weights_swapped": ("if (use_p) w += beta * P[(size_t)j];",
                                       "if (use_p) w += (1.0 - beta) * P[(size_t)j];"),
    "sample_temperature_ignored": ("const double temp = (double)temperature;", "const double temp = 1.0;"),
    "jsd_endpoint_zero_times_inf": ("""                if (wp > 0.0)
                    for (int j = 0; j < V; ++j)
                        if (P[(size_t)j] > 0.0)
                            kl_pm += P[(size_t)j] * (logP[(size_t)j] - logM[(size_t)j]);
                if (wq > 0.0)
                    for (int j = 0; j < V; ++j)
                        if (Q[(size_t)j] > 0.0)
                            kl_qm += Q[(size_t)j] * (logQ[(size_t)j] - logM[(size_t)j]);
                D = 0.0;
                if (wp > 0.0) D += wp * kl_pm;
                if (wq > 0.0) D += wq * kl_qm;""",
                                    """                for (int j = 0; j < V; ++j)
                    if (P[(size_t)j] > 0.0)
                        kl_pm += P[(size_t)j] * (logP[(size_t)j] - logM[(size_t)j]);
                for (int j = 0; j < V; ++j)
                    if (Q[(size_t)j] > 0.0)
                        kl_qm += Q[(size_t)j] * (logQ[(size_t)j] - logM[(size_t)j]);
                D = wp * kl_pm + wq * kl_qm;"""),
    "jsd_endpoint_grad_weight_ignored": ("g[j] = (wq > 0.0 && Q[(size_t)j] > 0.0)", "g[j] = (Q[(size_t)j] > 0.0)"),
    "cdf_margin_divided_by_z": ("*margin = a < b ? a : b;", "*margin = (a < b ? a : b) / Z;"),
    "tree_residual_not_updated": ("for (int j = 0; j < V; ++j) R[(size_t)j] = r[(size_t)j] / Z;", "(void)0;"),
    "tree_tested_against_p": ("const double rc = R[(size_t)tok[c]], qc", "const double rc = P[(size_t)tok[c]], qc"),
    "tree_extra_from_p": ("extra = inverse_cdf(last_r, last_Z, u_resample[b], &m);",
                          "extra = inverse_cdf(P, 1.0, u_resample[b], &m);"),
    "tree_children_last_first": ("if (par[n] == v) kids.push_back(n);", "if (par[n] == v) kids.insert(kids.begin(), n);"),
    "sample_row_stride_ignored": ("temperature_softmax(load_row(q, dtype, (int64_t)n * q_stride, V), temp, Q, logQ)",
                                  "temperature_softmax(load_row(q, dtype, (int64_t)n * V, V), temp, Q, logQ)"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not found exactly once: {name}"
    mutated = tmp_path / "osd_ref_mut.cpp"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libosd_ref_mut.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-fPIC", "-shared", "-I",
                    os.path.join(ROOT, "oracle"), "-o", str(lib), str(mutated)],
                   check=True)
    env = dict(os.environ, OSD_REF_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_verify_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_distill_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_sample_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_tree_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"pins did not catch mutation {name}:\n{r.stdout[-2000:]}"
