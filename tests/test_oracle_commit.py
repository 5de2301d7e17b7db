"""Pins for the commitment decision, case by case from Section 3.2.

  * timing-based eligibility: a claim may commit once its estimated laxity
    TTU - TTR has reached zero or gone below it, or as soon as retrieval of
    its KV is requested;
  * positive laxity predicts early readiness: not eligible, decision deferred;
  * a protected commitment needs the claim's full footprint within the
    protected-capacity budget; bytes that an earlier commitment already
    protects are not reserved again ("Shared staging and resource lifecycle");
  * without sufficient capacity the claim stays PLANNED (here BLOCKED);
  * a claim whose retrieval is requested but which cannot be protected is
    read through the ordinary retrieval path instead, uncommitted (ORDINARY).
"""
import itertools
import math

import pytest

import oracle
from oracle import BLOCKED, COMMIT, DEFER, EINVAL, ORDINARY

GiB = 1 << 30


@pytest.mark.parametrize("laxity_sign,fits,requested",
                         list(itertools.product([-1, 0, 1], ["yes", "budget", "free"], [False, True])))
def test_truth_table(laxity_sign, fits, requested):
    ttr = 2.0
    ttu = ttr + 0.5 * laxity_sign
    budget, free, total, new = 50 * GiB, 10 * GiB, 8 * GiB, 4 * GiB
    if fits == "budget":
        total = 60 * GiB            # footprint larger than the whole budget
    elif fits == "free":
        new = 12 * GiB              # newly reserved bytes exceed free protected capacity
        total = 16 * GiB
    d = oracle.commit_should_stage(ttu, ttr, free, new, total, budget, requested)
    eligible = laxity_sign <= 0 or requested
    if not eligible:
        assert d == DEFER
    elif fits == "yes":
        assert d == COMMIT
    elif requested:
        assert d == ORDINARY
    else:
        assert d == BLOCKED


def test_exactly_zero_laxity_is_eligible():
    assert oracle.commit_should_stage(1.25, 1.25, GiB, 1, 1, GiB, False) == COMMIT


def test_fits_at_the_boundaries():
    assert oracle.commit_should_stage(0.0, 1.0, 5, 5, 9, 9, False) == COMMIT
    assert oracle.commit_should_stage(0.0, 1.0, 4, 5, 9, 9, False) == BLOCKED
    assert oracle.commit_should_stage(0.0, 1.0, 5, 5, 10, 9, True) == ORDINARY


def test_shared_bytes_already_covered_need_no_free_capacity():
    # Every byte of the claim is already protected for another claim: nothing
    # new to reserve, so it commits even with no free protected capacity.
    assert oracle.commit_should_stage(0.0, 3.0, 0, 0, 8 * GiB, 50 * GiB, False) == COMMIT


def test_infinite_estimates():
    inf = math.inf
    assert oracle.commit_should_stage(1.0, inf, GiB, 1, 1, GiB, False) == COMMIT   # never ready in time
    assert oracle.commit_should_stage(inf, 1.0, GiB, 1, 1, GiB, False) == DEFER    # no retrieval expected
    assert oracle.commit_should_stage(inf, 1.0, GiB, 1, 1, GiB, True) == COMMIT
    assert oracle.commit_should_stage(-inf, 1.0, GiB, 1, 1, GiB, False) == COMMIT


def test_invalid_inputs():
    assert oracle.commit_should_stage(math.nan, 1.0, 1, 1, 1, 1, False) == EINVAL
    assert oracle.commit_should_stage(1.0, math.nan, 1, 1, 1, 1, True) == EINVAL
    assert oracle.commit_should_stage(0.0, 1.0, 10, 5, 4, 10, False) == EINVAL    # new > total
