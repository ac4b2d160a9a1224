"""Mutation check of the oracle's conditioning pins (CPU only).

Each case plants one plausible mistake in a temporary copy of the oracle's
C source (a dropped term, a missing absolute value, a wrong summation range,
K in place of K'), builds it, binds the oracle module to that build and runs
the pins that cover the output: at least one must fail. The same pins pass on
the real oracle (tests/test_oracle_conditioning.py and the conv-vs-dense pin
in tests/test_oracle_pins.py).
"""
import os
import tempfile

import pytest

import oracle
from tests import test_oracle_conditioning as tc
from tests import test_oracle_pins as tp

SRC = os.path.join(os.path.dirname(oracle.__file__), "dstd_oracle.c")

_CONV_CS = dict(C_in=3, H=8, W=6, C_out=2, KH=3, KW=3, stride=1, pad=1, pool_in=2)


def _dense_vabs():
    for row in [(1.0, 0.3), (0.5, 0.5), (float("inf"), 0.4)]:
        tc.test_dstd_vabs_and_emass_are_direct_sums(*row)


def _dense_margin():
    tc.test_dstd_margin_earlier_interval_term_binds()
    tc.test_dstd_margin_right_end_term_binds()
    for row in [(1.0, 0.3), (2.0, 0.4), (0.5, 0.5)]:
        tc.test_dstd_margin_and_interval_match_superposition(*row)


def _dense_backward():
    for row in [(1.0, 0.3), (float("inf"), float("inf"))]:
        tc.test_dstd_backward_abs_and_error_sums_are_direct_sums(*row)


def _conv():
    tp.test_conv_equals_dense_layer_with_conv_connectivity(_CONV_CS)


def _exact_fwd():
    tc.test_exact_margin_earlier_interval_term_binds()
    for row in [(1.0, 0.3), (0.5, 0.5)]:
        tc.test_exact_margin_vabs_emass_match_direct_sums(*row)


def _exact_bwd():
    tc.test_exact_backward_abs_and_error_sums_are_direct_sums(1.0, 0.3)


# (name, original text, planted text, pins expected to catch it)
MUTATIONS = [
    ("vabs summed over every grid point instead of m <= q*",
     "for (int m = 0; m <= (q < 0 ? -1 : q); ++m)\n                    va +=",
     "for (int m = 0; m <= M; ++m)\n                    va +=", _dense_vabs),
    ("vabs without the absolute value of the event terms",
     "wabs[ev[j].m[k]] += fabs(wr[j] * ev[j].s[k]);",
     "wabs[ev[j].m[k]] += wr[j] * ev[j].s[k];", _dense_vabs),
    ("emass over every grid point for a firing neuron",
     "for (int m = 0; m <= (q < 0 ? M : q); ++m) em += wabs[m];\n                emass[o] = em;",
     "for (int m = 0; m <= M; ++m) em += wabs[m];\n                emass[o] = em;", _dense_vabs),
    ("margin drops the earlier-interval term",
     "double m = pre;\n            m = fmin(m, fabs(peak - p->theta));",
     "double m = INFINITY;\n            m = fmin(m, fabs(peak - p->theta));", _dense_margin),
    # No case drops |v(T_q*) - theta|: v^ is continuous, so theta minus the
    # previous interval's peak (its closed-interval supremum) already bounds
    # it; the two differ only at q* = 0, where v^(T_0) = 0 and the term is
    # theta, far from any ambiguity threshold. That mutant is equivalent.
    ("margin drops |v(T_q*+1) - theta|",
     "if (q < p->M) m = fmin(m, fabs(pv(&pc, hi) - p->theta));", "(void)hi;", _dense_margin),
    ("dW |term| sum without the absolute value",
     "double term = G[g] * e->s[k];\n                        acc += term;\n                        aabs += fabs(term);",
     "double term = G[g] * e->s[k];\n                        acc += term;\n                        aabs += term;",
     _dense_backward),
    ("error weight takes K in place of K'",
     "delta[o] * fabs(kern_dt(p.tv, p.ti, u)));\n            }\n        }\n    }\n    if (grad_t_in) {",
     "delta[o] * fabs(kern(p.tv, p.ti, u)));\n            }\n        }\n    }\n    if (grad_t_in) {",
     _dense_backward),
    ("error weight drops |gamma|",
     "GE[o * (M + 1) + m] = fabs(gam) * (rho[o]", "GE[o * (M + 1) + m] = (rho[o]", _dense_backward),
    ("conv vabs without the absolute value",
     "wabs[e->m[k]] += fabs(w * e->s[k]);", "wabs[e->m[k]] += w * e->s[k];", _conv),
    ("conv dW error sum drops the pooling factor",
     "dWel[widx] += GE[e->m[k]] * fabs(e->s[k]) / g.P;", "dWel[widx] += GE[e->m[k]] * fabs(e->s[k]);",
     _conv),
    ("exact margin drops the earlier-interval term",
     "mg = fmin(pre, fabs(peak - theta));", "mg = fabs(peak - theta);", _exact_fwd),
    ("exact vabs without the absolute value",
     "va += fabs(s[j].w * kern(tv, ti, root - s[j].t));", "va += s[j].w * kern(tv, ti, root - s[j].t);",
     _exact_fwd),
    ("exact dt_in error bound drops the K'' term",
     "(rho[o] * fabs(kd) + delta[o] * k2);", "(rho[o] * fabs(kd));", _exact_bwd),
]


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new,pins", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(name, old, new, pins):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site not found exactly once: {name}"
    with tempfile.TemporaryDirectory(prefix="oracle_mut_") as d:
        path = os.path.join(d, "dstd_oracle_mut.c")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        lib = oracle.compile_oracle(path, os.path.join(d, "libmut.so"))
        with oracle.use_library(lib):
            with pytest.raises(AssertionError):
                pins()


def test_pins_pass_on_the_oracle():
    for pins in {m[3] for m in MUTATIONS}:
        pins()
