"""Pins of the plain reference of intent signalling and action timing
(oracle/staging.py): the Poisson quantile against scipy, Algorithm 1's
update rules as closed forms, and hand-worked scenarios of the intent
states (inactive, active, expired) on a small local store."""
import math

import pytest
import scipy.stats as st

from oracle.staging import StagingOracle, action_timing, poisson_cdf, poisson_quantile

MUS = [1e-5, 1e-4, 0.01, 0.5, 1.0, 2.0, 7.3, 20.0, 100.0, 1234.5, 5000.0]
PS = [0.5, 0.9, 0.99, 0.9999]


@pytest.mark.parametrize("mu", MUS)
@pytest.mark.parametrize("p", PS)
def test_poisson_quantile_is_scipy_ppf(mu, p):
    assert poisson_quantile(mu, p) == int(st.poisson.ppf(p, mu))


@pytest.mark.parametrize("mu", [0.3, 20.0, 800.0])
def test_poisson_cdf_is_scipy_cdf(mu):
    for k in (0, 1, int(mu), int(mu + 3 * math.sqrt(mu)) + 1):
        assert poisson_cdf(k, mu) == pytest.approx(st.poisson.cdf(k, mu), rel=1e-11, abs=1e-300)


def test_poisson_quantile_zero_iff_no_event_is_likely_enough():
    """Q(mu, p) = 0 exactly when P(X = 0) = e^-mu >= p, i.e. mu <= -ln p."""
    p = 0.9999
    edge = -math.log(p)
    assert poisson_quantile(edge * 0.999, p) == 0
    assert poisson_quantile(edge * 1.001, p) == 1
    assert poisson_quantile(0.0, p) == 0


def test_first_round_from_the_paper_defaults():
    """lambda_0 = 10, alpha = 0.1, p = 0.9999, no clock yet: the estimate
    stays 10 and intents starting before 0 + Q(20, 0.9999) = 39 are acted upon."""
    lam, h = action_timing(10.0, 0, 0)
    assert lam == 10.0 and h == 39


def test_no_update_when_the_clock_did_not_move():
    lam, h = action_timing(3.25, 17, 17, alpha=0.1)
    assert lam == 3.25
    assert h == 17 + poisson_quantile(6.5, 0.9999)


def test_constant_rate_converges_in_closed_form():
    """Delta constant: lambda_t = Delta + (lambda_0 - Delta)(1 - alpha)^t."""
    lam, c, delta, alpha = 10.0, 0, 3, 0.1
    for t in range(1, 40):
        lam, _ = action_timing(lam, c, c + delta, alpha)
        c += delta
        assert lam == pytest.approx(delta + (10.0 - delta) * (1 - alpha) ** t, rel=1e-12)


def test_a_jump_above_the_estimate_uses_the_jump():
    """Delta = 100 after an estimate of 10: smoothing gives 19, but the
    decision uses max(19, 100) = 100."""
    lam, h = action_timing(10.0, 50, 150, alpha=0.1)
    assert lam == pytest.approx(19.0)
    assert h == 150 + poisson_quantile(200.0, 0.9999)
    assert h > 150 + poisson_quantile(38.0, 0.9999)


# ------------------------------------------------------------------ intent states
def test_data_loader_pattern_of_figure_2():
    """Intent(P_i, i, i+1) for batches 1..4 signalled up front; a round at
    clock 0 acts on all four (horizon 39); keys leave once their last
    intent has expired."""
    o = StagingOracle(100, [0], [100])
    P = {1: [1, 2, 3], 2: [3, 4], 3: [5, 1], 4: [6]}
    for i, keys in P.items():
        o.intent(keys, i, i + 1)
    staged, evicted = o.round()
    assert o.last_horizon == 39 and evicted == []
    assert sorted(staged) == [1, 2, 3, 4, 5, 6]
    o.advance_clock()                   # clock 1: batch 1 active, nothing forced
    assert o.forced == 0
    o.advance_clock()                   # clock 2: P_1's intent expired
    staged, evicted = o.round()
    assert staged == [] and sorted(evicted) == [2]   # 1 is wanted again at 3, 3 at 2
    o.advance_clock()
    o.round()                           # clock 3: P_2 expired, 3 and 4 leave
    assert o.resident() == {1, 5, 6}
    o.advance_clock()
    o.advance_clock()
    staged, evicted = o.round()         # clock 5: everything expired
    assert o.resident() == set() and sorted(evicted) == [1, 5, 6]


def test_late_intent_is_forced_when_it_becomes_active():
    o = StagingOracle(10, [0], [10])
    o.intent([7, 8], 1, 2)
    o.advance_clock()                   # no round ran: act at once
    assert o.forced == 1 and o.resident() == {7, 8}


def test_small_rate_defers_action_until_the_horizon_reaches_the_intent():
    """lambda_0 = 1, p = 0.5: Q(2, 0.5) = 2, so at clock C only intents with
    C_start < C + 2 are acted upon."""
    o = StagingOracle(10, [0], [10], p=0.5, lambda0=1.0)
    assert poisson_quantile(2.0, 0.5) == 2
    o.intent([3], 3, 4)
    o.round()                           # clock 0: horizon 2 (estimate 1, Delta 0)
    assert o.resident() == set()
    o.advance_clock()
    o.round()                           # clock 1: Delta 1, estimate 1, horizon 3: 3 < 3 is false
    assert o.resident() == set() and o.last_horizon == 3
    o.advance_clock()
    o.round()                           # clock 2: horizon 4
    assert o.resident() == {3} and o.forced == 0


def test_capacity_limits_acting_per_range_in_order():
    """Two ranges of capacity 2 each; the round stops at the first key whose
    range is full and continues once expiries free slots."""
    o = StagingOracle(20, [0, 10], [2, 2])
    o.intent([1, 2, 3], 1, 2)           # range 0 needs 3 slots
    o.intent([11], 1, 2)
    o.intent([4], 2, 3)
    staged, _ = o.round()
    assert staged == [1, 2] and o.resident() == {1, 2}
    o.advance_clock()                   # forced: still full, nothing more
    assert o.resident() == {1, 2} and o.forced == 1
    o.advance_clock()                   # clock 2: 1 and 2 expired; intent (1,2) dropped; 4 forced in
    assert o.resident() == {4}


def test_out_of_range_keys_and_expired_intents_are_ignored():
    o = StagingOracle(5, [0], [5])
    o.advance_clock()
    o.advance_clock()
    o.intent([1], 0, 2)                 # already expired at clock 2
    o.intent([-1, 2, 5, 99], 3, 4)
    o.round()
    assert o.resident() == {2}


def test_overlapping_intents_extend_residency():
    o = StagingOracle(5, [0], [5])
    o.intent([1], 1, 3)
    o.intent([1], 2, 6)
    o.round()
    for _ in range(5):
        o.advance_clock()
        o.round()
        assert (1 in o.resident()) == (o.clock < 6)
