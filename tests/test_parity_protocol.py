"""The parity protocol's host side, without a GPU: the bound on decisions
pinned from the oracle, and the pinned counts of the small parity cases (the
oracle alone decides them, so they are known before any GPU run)."""
import numpy as np
import pytest

from tests import harness as H
from paper_2606_10650_amd.workloads import WORKLOADS, make_inputs


def test_bound_rejects_a_margin_that_pins_everything():
    """A margin that came out zero would pin every decision and leave the
    kernels' decision logic untested; the bound turns that into a failure."""
    T = 400
    ref = {"b": np.ones((1, T), np.int8), "merge": np.full((1, T), -1, np.int32),
           "margin_b": np.zeros((1, T)), "margin_m": np.full((1, T), np.inf)}
    with pytest.raises(AssertionError, match="near-tie decisions pinned"):
        H.near_tie_overrides(ref, what="all pinned")
    ref["margin_b"][:] = 1.0
    ref["margin_b"][0, :2] = 1e-6   # two near ties out of 400 free decisions: allowed
    bo, mo, nb, nm = H.near_tie_overrides(ref, what="two pinned")
    assert nb == 2 and nm == 0 and (bo[0, :2] == 1).all() and (bo[0, 2:] == -1).all()


# the small cases of tests/test_gpu_parity.py (same workloads, same sizes)
SMALL = [
    ("cfg1", {}, None, None),
    ("cfg1_iid", {}, None, None),
    ("cfg1", {}, 1, None),
    ("cfg1", dict(T=300), 300, 0.0),
    ("cfg2", dict(B=1, H=4, T=1000, C=12), None, None),
    ("cfg3", dict(B=1, H=3, T=2600, C=24, span_mean=200.0), None, None),
    ("cfg4", dict(B=1, H=2, T=3000, C=40, n_seg=200), None, None),
    ("cfg2", dict(B=1, H=2, T=700, C=9, dk=64, dv=128), None, None),
    ("cfg2", dict(B=1, H=1, T=1100, dk=128, dv=128), 1024, 0.0),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_cases_pin_few_decisions(case):
    name, kw, C, tau = SMALL[case]
    w = WORKLOADS[name].replace(**kw) if kw else WORKLOADS[name]
    w = w.replace(C=C or w.C, tau=w.tau if tau is None else tau)
    x = make_inputs(w)
    ref = H.run_oracle(w, {k: x[k] for k in ("k", "v", "g")}, full=False)
    H.near_tie_overrides(ref, what=w.label)   # asserts the bound
