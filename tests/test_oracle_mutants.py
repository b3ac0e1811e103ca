"""Every plausible mistake planted in a copy of the oracle must fail a pin.

Each mutant is a textual edit of dla_oracle.c (a dropped term, a wrong sign or
index, a transposed operand, a wrong reading of an algorithm step), compiled
to a temporary library.  The pins of tests/pins.py are run against it and at
least one must fail; otherwise the pins would not catch that mistake.  CPU only.
"""
import os
import subprocess
import tempfile

import pytest

from tests import pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "dla_oracle.c")

MUTANTS = {
    # the delta-rule form (Sec. 2.2, eq. delta_rule_rnn)
    "delta_u_without_erase_term": ("u_out[t * dv + c] = beta ? beta[t] * (vt[c] - y[c]) : vt[c];",
                                   "u_out[t * dv + c] = beta ? beta[t] * vt[c] : vt[c];"),
    "delta_u_unscaled": ("u_out[t * dv + c] = beta ? beta[t] * vt[c] : vt[c];",
                         "u_out[t * dv + c] = vt[c];"),
    "delta_erase_sign": ("S[a * dv + c] -= beta * k[a] * u[c];", "S[a * dv + c] += beta * k[a] * u[c];"),
    "delta_erase_without_key": ("u[c] += k[a] * S[a * dv + c];", "u[c] += S[a * dv + c];"),
    "delta_erase_skipped": ("      if (beta) delta_erase(So, kt, beta[t], dk, dv, y);\n", "\n"),
    "delta_write_unscaled": ("      for (int64_t i = 0; i < D; ++i) s[i] *= beta[t];\n", "      ;\n"),
    "delta_on_closing_state": ("      memcpy(S + (int64_t)m * D, s, sizeof(double) * D);",
                               "      if (beta && m > 0) delta_erase(S + (int64_t)(m - 1) * D, kt, beta[t], dk, dv, y);\n"
                               "      memcpy(S + (int64_t)m * D, s, sizeof(double) * D);"),
    "no_decay": ("S[j * D + i] *= alpha;", "S[j * D + i] *= 1.0;"),
    "decay_only_newest": ("for (int32_t j = full ? 0 : (m > 0 ? m - 1 : 0); j < m; ++j)",
                          "for (int32_t j = (m > 0 ? m - 1 : 0); j < m; ++j)"),
    "score_sign": ("const double d = ns[i] - nS[i];", "const double d = ns[i] + nS[i];"),
    "no_rmsnorm_on_state": ("nS[i] = S[i] / rS;", "nS[i] = S[i];"),
    "score_denominator_token": ("return sqrt(dd) / (frob(nS, D) + eps);",
                                "return sqrt(dd) / (frob(ns, D) + eps);"),
    "rms_not_mean": ("const double rS = sqrt(SS / (double)D + eps_rms);",
                     "const double rS = sqrt(SS + eps_rms);"),
    "threshold_strict": ("b = (I >= tau) ? 1 : 0;", "b = (I > tau) ? 1 : 0;"),
    "argmax": ("if (dens[i] < dens[best]) best = i;", "if (dens[i] > dens[best]) best = i;"),
    "argmin_last_tie": ("if (dens[i] < dens[best]) best = i;",
                        "if (dens[i] <= dens[best]) best = i;"),
    "density_product": ("(double)(n[i] + n[i + 1]);", "(double)(n[i] * n[i + 1]);"),
    "density_no_count": ("dens[i] = (ibar[i] + ibar[i + 1]) / (double)(n[i] + n[i + 1]);",
                         "dens[i] = (ibar[i] + ibar[i + 1]);"),
    "merge_overwrites": ("S[best * D + i] += S[(best + 1) * D + i];",
                         "S[best * D + i] = S[(best + 1) * D + i];"),
    "merge_counts_not_summed": ("n[best] += n[best + 1];", "n[best] += 0;"),
    "new_state_score_zero": ("ibar[m] = I;", "ibar[m] = 0.0;"),
    "accumulate_score_dropped": ("ibar[m - 1] += I;", "ibar[m - 1] += 0.0;"),
    # Alg. 1 read literally: the token is merged into the newest state and also appended
    "double_count_token": ("      memcpy(S + (int64_t)m * D, s, sizeof(double) * D);",
                           "      if (m > 0)\n"
                           "        for (int64_t i = 0; i < D; ++i) S[(int64_t)(m - 1) * D + i] += s[i];\n"
                           "      memcpy(S + (int64_t)m * D, s, sizeof(double) * D);"),
    "readout_transposed": ("y[c] += qt[a] * Sj[a * dv + c];", "y[c] += qt[a] * Sj[c * dk + a];"),
    "lambda_recency_index": ("lam[t * C + j]", "lam[t * C + (m - 1 - j)]"),
    "readout_skips_newest": ("for (int32_t j = 0; j < m; ++j) {\n        const double lj",
                             "for (int32_t j = 0; j + 1 < m; ++j) {\n        const double lj"),
    "token_state_outer_swapped": ("s[a * dv + c] = kt[a] * vt[c];",
                                  "s[a * dv + c] = kt[c % dk] * vt[a % dv];"),
    # the just-closed state left out of the merge candidates
    "candidates_exclude_closed": ("for (int32_t i = 0; i + 1 < C; ++i) {\n          dens[i]",
                                  "for (int32_t i = 0; i + 2 < C; ++i) {\n          dens[i]"),
    # the near-tie margins that decide where the parity protocol hands the GPU
    # the oracle's decision, and the merge override
    "margin_b_zero": ("margin_b[t] = free_b ? fabs(I - tau) : INFINITY;",
                      "margin_b[t] = free_b ? 0.0 : INFINITY;"),
    "margin_b_forced_counted": ("margin_b[t] = free_b ? fabs(I - tau) : INFINITY;",
                                "margin_b[t] = fabs(I - tau);"),
    "margin_b_against_zero": ("margin_b[t] = free_b ? fabs(I - tau) : INFINITY;",
                              "margin_b[t] = free_b ? fabs(I) : INFINITY;"),
    "margin_m_zero": ("mgap = (second - d1) / (fabs(d1) > 0.0 ? fabs(d1) : 1e-300);",
                      "mgap = 0.0;"),
    "margin_m_largest_pair": ("if (i != best && dens[i] < second) second = dens[i];",
                              "if (i != best && (second == INFINITY || dens[i] > second)) "
                              "second = dens[i];"),
    "margin_m_relative_to_second": ("mgap = (second - d1) / (fabs(d1) > 0.0 ? fabs(d1) : 1e-300);",
                                    "mgap = (second - d1) / second;"),
    "margin_m_for_forced_merge": ("        } else if (C > 2) {\n          const double d1",
                                  "        }\n        if (C > 2) {\n          const double d1"),
    "merge_override_ignored": ("best = m_ovr[t];", "best = best;"),
    "merge_override_below_capacity": (
        "      if (m == C) {\n        /* Alg. 2",
        "      if (m == C || (m_ovr && m_ovr[t] >= 0 && m >= 2)) {\n        /* Alg. 2"),
    # (accepted and clamped into range, so the mutant never indexes outside the cache)
    "merge_override_out_of_range_accepted": (
        "          if (m_ovr[t] < 0 || m_ovr[t] > C - 2) {\n            rc = ORACLE_BAD_MERGE_OVERRIDE;\n"
        "            break;\n          }\n          best = m_ovr[t];",
        "          best = m_ovr[t] < 0 ? 0 : (m_ovr[t] > C - 2 ? C - 2 : m_ovr[t]);"),
    # the size of the readout's terms (the rounding scale of stored states)
    "magnitude_signed_lambda": ("mag += fabs(lj) * frob(Sj, D);", "mag += lj * frob(Sj, D);"),
    "magnitude_last_state_only": ("mag += fabs(lj) * frob(Sj, D);", "mag = fabs(lj) * frob(Sj, D);"),
    "magnitude_without_query": ("mag_out[t] = mag * frob(qt, dk);", "mag_out[t] = mag;"),
    "c1_not_forced": ("      if (C == 1) {\n        b = 0;", "      if (C == 0) {\n        b = 0;"),
}


@pytest.fixture(scope="module")
def src():
    with open(SRC) as fh:
        return fh.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_fails_a_pin(name, src, tmp_path):
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new, 1)
    c = tmp_path / "mut.c"
    c.write_text(mutated)
    lib = str(tmp_path / "libmut.so")
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-shared", "-fPIC", str(c), "-o", lib,
                    "-lm"], check=True)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(lib_path=lib)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
