"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of the oracle's C source (a dropped
term, a wrong sign or index, an off-by-one mask, a transposed operand, a wrong
tie-break), builds it with gcc into a temporary library and runs the pins against it
in a child process.  At least one pin must fail for every mutant; otherwise the pins
would let that mistake through.
"""
import json
import os
import subprocess
import sys

import pytest

import oracle

MUTANTS = {
    "causal_mask_minus_one": ("? ctx + i + 1 : ctx + B", "? ctx + i : ctx + B"),
    "causal_mask_plus_one": ("? ctx + i + 1 : ctx + B", "? ctx + i + 2 : ctx + B"),
    "bidir_mask_short": ("? ctx + i + 1 : ctx + B;", "? ctx + i + 1 : ctx + B - 1;"),
    "gqa_modulo_map": ("const int g = h / G;", "const int g = h % Hkv;"),
    "scale_dropped": ("score[j] = scale * acc;", "score[j] = acc;"),
    "normaliser_dropped": ("o[d] /= den;", "o[d] /= 1.0;"),
    "max_not_subtracted_wrong": ("double w = exp(score[j] - mx);", "double w = exp(score[j] - mx) * (j + 1);"),
    "value_row_transposed": ("o[d] += w * (double)vb[(size_t)j * D + d];",
                             "o[d] += w * (double)vb[(size_t)d * D + j % D];"),
    "argmax_highest_tie": ("if (x[v] > x[best]) best = v;", "if (x[v] >= x[best]) best = v;"),
    "accept_le": ("if (!(u < rho)) break;", "if (!(u <= rho)) break;"),
    "accept_always": ("if (!(u < rho)) break;", "if (0) break;"),
    "ratio_inverted": ("p[d] / qd[d] : INFINITY", "qd[d] / p[d] : INFINITY"),
    "residual_is_p": ("r[v] = p[v] - qd[v];", "r[v] = p[v];"),
    "residual_sign": ("r[v] = p[v] - qd[v];", "r[v] = qd[v] - p[v];"),
    "temperature_ignored": ("p[v] = exp(((double)x[v] - mx) / T);", "p[v] = exp(((double)x[v] - mx));"),
    "cdf_ge": ("if (c > target) return v;", "if (c >= target) return v;"),
    "final_uniform_slot": ("const double ustar = (double)uniforms[off + n];",
                           "const double ustar = (double)uniforms[off + a];"),
    "greedy_next_row_shift": ("next_token[s] = argmax_lowest(target + (size_t)(off + a) * V, V);",
                              "next_token[s] = argmax_lowest(target + (size_t)(off + (a ? a - 1 : 0)) * V, V);"),
    # the parity harness's near-tie outputs
    "accept_margin_rho_unclamped": ("fabs(u - (rho < 1.0 ? rho : 1.0))", "fabs(u - rho)"),
    "accept_margin_last_tested": ("if (m < accept_margin[s]) accept_margin[s] = m;", "accept_margin[s] = m;"),
    "accept_margin_untested_too": ("if (!(u < rho)) break; /* R7 */",
                                   "if (!(u < rho)) { for (int k = a + 1; k < n; ++k) { const double uk = "
                                   "(double)uniforms[off + k]; if (fabs(uk - 0.5) < accept_margin[s]) "
                                   "accept_margin[s] = fabs(uk - 0.5); } break; }"),
    "sample_margin_zero": ("sample_margin[s] = m1 < m2 ? m1 : m2;", "sample_margin[s] = 0;"),
    "sample_margin_unscaled": ("double m1 = (tgt - below) / tot, m2 = (below + r[x] - tgt) / tot;",
                               "double m1 = (tgt - below), m2 = (below + r[x] - tgt);"),
    "sample_margin_far_edge": ("sample_margin[s] = m1 < m2 ? m1 : m2;", "sample_margin[s] = m1 > m2 ? m1 : m2;"),
    "band_whole_vocab": ("double lo_t = tgt - band * tot, hi_t = tgt + band * tot;", "double lo_t = 0, hi_t = tot;"),
    "band_unscaled": ("double lo_t = tgt - band * tot, hi_t = tgt + band * tot;",
                      "double lo_t = tgt - band, hi_t = tgt + band;"),
    "band_whole_and_margin_zero": ("double lo_t = tgt - band * tot, hi_t = tgt + band * tot;\n",
                                   "double lo_t = 0, hi_t = tot; m1 = m2 = 0; sample_margin[s] = 0;\n"),
    "tie_p_band_only": ("ptie += w < 2.0 * band ? w : 2.0 * band;", "ptie += w > 0 ? 2.0 * band : 0.0;"),
    "tie_p_mass_only": ("ptie += w < 2.0 * band ? w : 2.0 * band;", "ptie += w;"),
}

_RUNNER = r"""
import json, sys
sys.path.insert(0, sys.argv[1]); sys.path.insert(0, sys.argv[2])
import oracle, oracle_pins
orc = oracle.Oracle(sys.argv[3])
print("RESULT " + json.dumps(oracle_pins.run_all(orc)))
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    src = open(oracle.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation site for {name} not found; update the mutant table"
    mutated = src.replace(old, new, 1)
    c_path = tmp_path / "mutant.c"
    c_path.write_text(mutated)
    so_path = str(tmp_path / "libmutant.so")
    oracle.compile_oracle(str(c_path), so_path)
    here = os.path.dirname(os.path.abspath(__file__))
    root = os.path.dirname(here)
    env = dict(os.environ, OMP_NUM_THREADS=os.environ.get("OMP_NUM_THREADS", "4"))
    proc = subprocess.run([sys.executable, "-c", _RUNNER, root, here, so_path], capture_output=True,
                          text=True, timeout=600, env=env)
    line = [l for l in proc.stdout.splitlines() if l.startswith("RESULT ")]
    if not line:
        # the mutant crashed the child process: that is a detected mistake too
        assert proc.returncode != 0
        return
    res = json.loads(line[0][len("RESULT "):])
    failed = [k for k, v in res.items() if v is not None]
    assert failed, f"mutant {name} passed every pin"
