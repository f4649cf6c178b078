"""The pins must catch plausible slips in the oracle.

Each case plants one mistake in a temporary copy of oracle.c (a source
substitution, compiled on the CPU into a throw-away library), reruns the pin
suite against it and requires at least one pin to fail.  The real oracle is
never modified.
"""
import os
import subprocess

import pytest

import oracle
import sys
sys.path.insert(0, os.path.dirname(__file__))
from oracle import build as obuild

import test_oracle_pins as pins

MUTATIONS = {
    "bias_dropped": ("+ pb->bias[at_bias(pb->g, qi, k) * H + hh];", ";"),
    "bias_transposed_starting": ("return qi * g.n + k; /* B[q][k] */", "return k * g.n + qi;"),
    "ending_key_axis_swapped": ("return k * g.n + row;                              /* [k][j], j = row */",
                                "return row * g.n + k;"),
    "ending_mask_transposed": ("return k * g.n + row;                              /* mask[k][j] */",
                               "return row * g.n + k;"),
    "scale_missing": ("s[k] = pb->scale * dot +", "s[k] = dot +"),
    "gate_not_applied": ("out[e] = sigmoid(gate[e]) * a[c];", "out[e] = a[c];"),
    "ds_sign": ("const double ds = p[kk] * (dp - dsum);", "const double ds = p[kk] * (dsum - dp);"),
    "d_term_dropped": ("dsum += da[c] * a[c]; /* D = rowsum(dA * A) */", ";"),
    "dq_scale_missing": ("dq[e0 + c] += scale * ds * k[ek + c];", "dq[e0 + c] += ds * k[ek + c];"),
    "dv_uses_dout": ("dv[ek + c] += p[kk] * da[c];", "dv[ek + c] += p[kk] * dout[e0 + c];"),
    "dgate_wrong": ("dg[e0 + c] = dout[e0 + c] * a[c] * sg * (1.0 - sg);",
                    "dg[e0 + c] = dout[e0 + c] * a[c] * sg;"),
    "db_drops_d": ("acc[kk] += p[kk] * (dp - dsum);", "acc[kk] += p[kk] * dp;"),
    "lse_without_max": ("const double lse = mx + log(z);", "const double lse = log(z);"),
    "mask_ignored": ("int valid = pb->mask == NULL || pb->mask[at_mask(pb->g, row, k)] != 0;",
                     "int valid = 1;"),
}

PIN_TESTS = [
    (pins.test_forward_matches_sdpa_starting, dict(seed=1)),
    (pins.test_backward_matches_sdpa_autograd_starting, dict(seed=3)),
    (pins.test_backward_matches_central_finite_differences, dict(node=0)),
    (pins.test_backward_matches_central_finite_differences, dict(node=1)),
    (pins.test_ending_is_transposed_starting, dict(node=0)),
    (pins.test_closed_forms_zero_query_and_constant_bias, dict(node=1)),
    (pins.test_closed_form_single_valid_key, dict(node=1)),
    (pins.test_fully_masked_queries, dict(node=1)),
    (pins.test_hand_derived_fixture, dict()),
]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    bad = tmp_path / "oracle_mut.c"
    bad.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", str(bad), "-o",
                    str(lib), "-lm"], check=True)
    prev = oracle.use_library(oracle.load(str(lib)))
    caught = []
    try:
        for fn, kw in PIN_TESTS:
            try:
                fn(**kw)
            except AssertionError:
                caught.append(fn.__name__)
    finally:
        oracle.use_library(prev)
    assert caught, f"no pin caught mutation {name}"


# ---- the fused layer-norm + linear oracle (ln_linear.c) -------------------------------

import test_oracle_ln_linear as lnl_pins  # noqa: E402

LNL_MUTATIONS = {
    "unbiased_variance": ("  var /= (double)K;", "  var /= (double)(K - 1);"),
    "mean_not_subtracted": ("    xhat[k] = (x[k] - mean) * rstd;", "    xhat[k] = x[k] * rstd;"),
    "beta_dropped": ("    o1[k] = xhat[k] * gamma[k] + beta[k];", "    o1[k] = xhat[k] * gamma[k];"),
    "c1_dropped": ("rstd * (wdy[k] - c1 * xhat[k] - c2)", "rstd * (wdy[k] - c2)"),
    "c2_dropped": ("rstd * (wdy[k] - c1 * xhat[k] - c2)", "rstd * (wdy[k] - c1 * xhat[k])"),
    "rstd_missing_in_dx": ("rstd * (wdy[k] - c1 * xhat[k] - c2)", "(wdy[k] - c1 * xhat[k] - c2)"),
    "gamma_missing_in_wdy": ("      wdy[k] = d1 * gamma[k];", "      wdy[k] = d1;"),
    "dw_uses_xhat": ("        dw[k * N + n] += o1 * do2[m * N + n];",
                     "        dw[k * N + n] += xhat * do2[m * N + n];"),
    "dgamma_uses_o1": ("      dg += d1 * xhat;", "      dg += d1 * o1;"),
    "w_transposed_in_do1": ("      for (int64_t n = 0; n < N; ++n) d1 += do2[m * N + n] * w[k * N + n];",
                            "      for (int64_t n = 0; n < N; ++n) d1 += do2[m * N + n] * w[n * K + k % N];"),
}

LNL_PIN_TESTS = [
    (lnl_pins.test_forward_and_backward_match_torch, dict(m=5, k=4, n=3, seed=0)),
    (lnl_pins.test_backward_matches_central_finite_differences, dict()),
    (lnl_pins.test_row_shift_and_scale_invariance, dict()),
    (lnl_pins.test_zero_gamma_gives_beta_projection_and_no_input_gradient, dict()),
    (lnl_pins.test_closed_form_two_features, dict()),
]


@pytest.mark.parametrize("name", sorted(LNL_MUTATIONS))
def test_lnl_pins_catch_mutation(name, tmp_path):
    old, new = LNL_MUTATIONS[name]
    src = open(obuild.SRC_LNL).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    bad = tmp_path / "ln_linear_mut.c"
    bad.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", obuild.SRC,
                    str(bad), "-o", str(lib), "-lm"], check=True)
    prev = oracle.use_library(oracle.load(str(lib)))
    caught = []
    try:
        for fn, kw in LNL_PIN_TESTS:
            try:
                fn(**kw)
            except AssertionError:
                caught.append(fn.__name__)
    finally:
        oracle.use_library(prev)
    assert caught, f"no pin caught mutation {name}"
