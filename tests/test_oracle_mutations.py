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
