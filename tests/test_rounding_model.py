"""The kernels' precision rules on large-norm inputs, checked with the CPU
rounding model (tests/rounding_model.py) on the sweep's regression
configurations (skewed: log-normal cube-mean norms):
- with the first rules (two-term products only on block pairs that touch a
  block with a value above 8, O divided by the sum of the unrounded
  probabilities) each of the first six misses the bar, as the GPU measured
  (dK up to 2.14x, dQ up to 1.27x the 2e-2 bar, or dQ relative-L2 above
  1e-2);
- with the kernels' rules (threshold 7; two-term P on every pair of a row
  that touches a flagged block; two-term dS on every pair of such a row and
  of a row with |Delta| above 16; O divided by the sum of the rounded
  probabilities) every one stays within it;
- with those rules but the threshold at 8, the near-threshold configuration
  (a query block with values up to 7.06) misses it again;
- the last two configurations (found on the GPU in a sweep of 300 skewed
  ones) miss it without the Delta rule (dK 1.21x) or, on the GPU, with P
  two-term only on the flagged pairs (dQ 1.15x; the model, which leaves
  out the fp32 accumulation order, puts that one at 0.98x, against 0.04x
  under the kernels' rules)."""
import pytest

from rounding_model import model_errors
from sweep_cases import REGRESSION

CASES = {w.name: w for w in REGRESSION}


def _over(e):
    return e[0] > 1.0 or e[1] > 1.0 or e[2] > 1e-2 or e[3] > 1e-2


FIRST = [w.name for w in REGRESSION[:6]]


@pytest.mark.parametrize("name", FIRST)
def test_first_rules_miss_the_bar(name):
    e = model_errors(CASES[name], tau=8.0, row_rule=False, rounded_sum=False, p_row_rule=False, delta_tau=None)
    print("%s: dQ %.2f dK %.2f of the bar, rel-L2 dQ %.2e dK %.2e" % ((name,) + e))
    assert _over(e)


@pytest.mark.parametrize("name", list(CASES))
def test_kernel_rules_stay_within_the_bar(name):
    e = model_errors(CASES[name])
    print("%s: dQ %.2f dK %.2f of the bar, rel-L2 dQ %.2e dK %.2e" % ((name,) + e))
    assert not _over(e)


def test_threshold_8_misses_the_near_threshold_case():
    assert _over(model_errors(CASES["near-threshold-cap2"], tau=8.0))


def test_pair_rule_for_p_misses_the_flagged_row_case():
    # the GPU measured dQ at 1.15x the bar under the pair rule; the model,
    # which leaves out the fp32 accumulation order, puts it just under
    w = CASES["one-term-p-in-flagged-row"]
    pair_rule, kernel_rules = model_errors(w, p_row_rule=False), model_errors(w)
    print("dQ share: pair rule %.3f, kernel rules %.3f" % (pair_rule[0], kernel_rules[0]))
    assert pair_rule[0] > 0.9 and kernel_rules[0] < 0.1


def test_no_delta_rule_misses_the_large_delta_case():
    assert _over(model_errors(CASES["large-delta-unflagged-row"], delta_tau=None))
