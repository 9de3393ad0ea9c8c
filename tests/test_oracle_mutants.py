"""Planted mistakes: each build of the oracle below carries one plausible
error (dropped term, wrong sign, wrong index, swapped operand, ...), planted
in a temporary copy of the C source on the CPU.  The pin battery must reject
every one of them, and must accept the unmodified source."""
import os
import shutil
import subprocess

import pytest

import oracle
from tests import oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "pi_oracle.c")

MUTANTS = {
    "prior_dropped": [("double dl = z + (s < nw ? log_local : log_skip);", "double dl = z;")],
    "priors_swapped": [("(s < nw ? log_local : log_skip)", "(s < nw ? log_skip : log_local)")],
    "skip_prior_sign": [("log_skip = log1p(-at);", "log_skip = -log1p(-at);")],
    "eps_clip_dropped": [("return ORACLE_EPS + (1.0 - 2.0 * ORACLE_EPS) * a;", "return a;")],
    "sigmoid_sign": [("double a = 1.0 / (1.0 + exp(-g));", "double a = 1.0 / (1.0 + exp(g));")],
    "scale_dropped": [("z *= scale;", ";")],
    "window_short_by_one": [("int lo = t - k > 0 ? t - k : 0;", "int lo = t - k + 1 > 0 ? t - k + 1 : 0;")],
    "partner_off_by_one": [("slot[nw] = t - pi; ++cnt;", "slot[nw] = t - pi + 1; ++cnt;")],
    "partner_not_deduplicated": [
        ("return window_slots(k, causal) + (pi > k ? (causal ? 1 : 2) : 0);",
         "return window_slots(k, causal) + (pi > 0 ? (causal ? 1 : 2) : 0);"),
        ("if (pi > k && t - pi >= 0)", "if (pi > 0 && t - pi >= 0)"),
        ("if (!causal && pi > k && t + pi < n)", "if (!causal && pi > 0 && t + pi < n)")],
    # bidirectional mode
    "bidir_forward_partner_dropped": [("if (!causal && pi > k && t + pi < n) { slot[nw + 1] = t + pi; ++cnt; }", ";")],
    "bidir_window_left_only": [("int hi = causal ? t : (t + k < n - 1 ? t + k : n - 1);", "int hi = t;")],
    "bidir_window_right_short": [("int hi = causal ? t : (t + k < n - 1 ? t + k : n - 1);",
                                  "int hi = causal ? t : (t + k - 1 < n - 1 ? t + k - 1 : n - 1);")],
    "bidir_forward_partner_local_prior": [("(s < nw ? log_local : log_skip)", "(s < nw || s == nw + 1 ? log_local : log_skip)")],
    "bidir_forward_partner_mirrored": [("slot[nw + 1] = t + pi;", "slot[nw + 1] = t - pi;")],
    "keys_values_swapped": [("const float *kj = krows + (int64_t)slot[s] * D;",
                             "const float *kj = vrows + (int64_t)slot[s] * D;")],
    "values_from_keys": [("const float *vj = vrows + (int64_t)slot[s] * D;",
                          "const float *vj = krows + (int64_t)slot[s] * D;")],
    "softmax_unnormalised": [("if (slot[s] >= 0) Z += exp(delta[s] - mu);",
                              "if (slot[s] >= 0) Z += exp(delta[s]);")],
    "max_not_subtracted_in_lse": [("return mu + log(Z);", "return log(Z);")],
    # backward
    "bwd_softmax_mean_dropped": [("double dd = p[s] * (dp[s] - mean);", "double dd = p[s] * dp[s];")],
    "bwd_dv_weighted_by_logit_grad": [("dvb[(int64_t)j * D + d] += p[s] * (double)gt[d];",
                                       "dvb[(int64_t)j * D + d] += dd * (double)gt[d];")],
    "bwd_dk_scale_dropped": [("dkb[(int64_t)j * D + d] += scale * dd * (double)qt[d];",
                              "dkb[(int64_t)j * D + d] += dd * (double)qt[d];")],
    "bwd_dq_from_query": [("dqb[(int64_t)t * D + d] += scale * dd * (double)kj[d];",
                           "dqb[(int64_t)t * D + d] += scale * dd * (double)qt[d];")],
    "bwd_dp_from_keys": [("const float *vj = vb + (int64_t)slot[s] * D;\n                    for (int d = 0; d < D; ++d) dp[s]",
                          "const float *vj = kb + (int64_t)slot[s] * D;\n                    for (int d = 0; d < D; ++d) dp[s]")],
    "bwd_gate_skip_sign": [("double dg_skip = -(1.0 - 2.0 * ORACLE_EPS)", "double dg_skip = (1.0 - 2.0 * ORACLE_EPS)")],
    "bwd_gate_sigmoid_chain_dropped": [
        ("double dg_local = (1.0 - 2.0 * ORACLE_EPS) * a * (1.0 - a) / at;",
         "double dg_local = (1.0 - 2.0 * ORACLE_EPS) / at;"),
        ("double dg_skip = -(1.0 - 2.0 * ORACLE_EPS) * a * (1.0 - a) / (1.0 - at);",
         "double dg_skip = -(1.0 - 2.0 * ORACLE_EPS) / (1.0 - at);")],
    "bwd_gate_priors_swapped": [("dgt += dd * (s < nw ? dg_local : dg_skip);", "dgt += dd * (s < nw ? dg_skip : dg_local);")],
    "bwd_bidir_gate_partner_as_local": [("dgt += dd * (s < nw ? dg_local : dg_skip);",
                                         "dgt += dd * (s < nw || s == nw + 1 ? dg_local : dg_skip);")],
    "bwd_clamp_not_cut": [("if (clamp > 0.0 && fabs(delta[s]) >= clamp) dd = 0.0;", ";")],
}


def _build(tmp_path, name, edits):
    src = open(SRC).read()
    for old, new in edits:
        assert src.count(old) == 1, f"{name}: pattern must occur exactly once: {old!r}"
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    c.write_text(src)
    so = str(tmp_path / f"lib{name}.so")
    oracle.build(str(c), so)
    return oracle.load_library(so)


def _failures(L):
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(L)
        except (AssertionError, ValueError, FloatingPointError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_unmodified_source_passes(tmp_path):
    assert _failures(_build(tmp_path, "control", [])) == []


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_rejected(tmp_path, name):
    failed = _failures(_build(tmp_path, name, MUTANTS[name]))
    assert failed, f"planted mistake {name!r} passed every pin"
