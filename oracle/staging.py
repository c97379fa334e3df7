"""Plain reference of intent signalling and adaptive action timing for one
worker whose parameters live in a large home store and are staged into a
smaller local store (Section 3, "Intent signaling"; Section 4.2,
"Adaptive Action Timing", Algorithm 1).

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product path.
It shares nothing with the store's planner; it follows the paper's
definitions step by step in plain Python.

Definitions used (Section 3): an intent (keys, C_start, C_end) of the worker
is inactive while its clock C < C_start, active while C_start <= C < C_end
and expired once C_end <= C.  The worker raises C by one per advance.

Readings taken where the paper, written for several nodes, is silent about
one worker with one local store:
  * Acting on an intent makes its keys resident in the local store (a copy
    from the home store for keys not resident yet).  With one worker exactly
    one party has intent, so of the paper's techniques only relocation
    applies.
  * A resident key stays resident until every intent acted upon for it has
    expired (the largest such C_end <= C); the next round, or the next
    forced action, writes it back and frees its slot.
  * Rounds act on pending intents in order of C_start, ties in signal order,
    and on an intent's keys in the order given.  A key range whose local
    capacity is used up stops the acting for that round; the intent stays
    pending with the keys not reached.
  * An intent that is still pending when the clock reaches its C_start is
    acted upon at once (a forced action, the analogue of the remote access
    the paper falls back to when action comes too late).  Forced actions do
    not update the rate estimate.
  * Intents signalled already expired are ignored, and so is the rest of a
    pending intent that expires before capacity lets it be acted upon; keys
    outside [0, num_keys) are skipped.
"""
from __future__ import annotations

import math


def poisson_cdf(k: int, mu: float) -> float:
    """P(X <= k) for X ~ Poisson(mu): the sum of e^-mu mu^j / j!, each term
    formed in log space so that large mu does not underflow e^-mu."""
    if mu == 0.0:
        return 1.0
    total = 0.0
    for j in range(k + 1):
        total += math.exp(-mu + j * math.log(mu) - math.lgamma(j + 1))
    return total


def poisson_quantile(mu: float, p: float) -> int:
    """Q_Poiss(mu, p): the smallest k >= 0 with P(X <= k) >= p (Section 4.2)."""
    if mu == 0.0:
        return 0
    k = 0
    total = math.exp(-mu)
    while total < p:
        k += 1
        total += math.exp(-mu + k * math.log(mu) - math.lgamma(k + 1))
    return k


def smoothed_rate(estimate: float, advance: int, alpha: float) -> float:
    """The clocks-per-round estimate of adaptive action timing (Section 4.2):
    an exponential moving average, with weight alpha, of how far the worker
    clock moved between consecutive rounds.  A round that saw no clock
    movement carries no information and leaves the estimate as it was."""
    return (1.0 - alpha) * estimate + alpha * advance if advance > 0 else estimate


def action_timing(lam_prev: float, c_prev: int, c_now: int, alpha: float = 0.1, p: float = 0.9999):
    """Section 4.2 (Algorithm 1) for one round at clock c_now after a round at
    c_prev: returns (new estimate, horizon).  The next round is expected
    within Poisson-many clocks; the bound takes the p-quantile of a Poisson
    variable whose mean is twice the larger of the estimate and the last
    observed advance, so an intent is acted upon now iff its C_start lies
    below the horizon c_now + that quantile."""
    est = smoothed_rate(lam_prev, c_now - c_prev, alpha)
    reach = poisson_quantile(2.0 * max(est, float(c_now - c_prev)), p)
    return est, c_now + reach


class StagingOracle:
    """One worker, its clock, and a local store with a slot capacity per key
    range (range r holds keys [begin[r], begin[r+1]); the last range ends at
    num_keys).  Tracks which keys are resident after every event."""

    def __init__(self, num_keys, range_begin, range_capacity, alpha=0.1, p=0.9999, lambda0=10.0):
        self.num_keys = num_keys
        self.begin = list(range_begin)
        self.cap = list(range_capacity)
        self.alpha, self.p = alpha, p
        self.lam = lambda0
        self.clock = 0
        self.round_clock = 0           # C at the previous (non-forced) round
        self.pending = []              # [C_start, seq, C_end, keys, next index]
        self.seq = 0
        self.until = {}                # resident key -> largest C_end of intents acted upon
        self.count = [0] * len(self.begin)   # resident keys per range
        self.staged_total = 0
        self.evicted_total = 0
        self.forced = 0
        self.last_horizon = None

    def range_of(self, key):
        r = 0
        while r + 1 < len(self.begin) and key >= self.begin[r + 1]:
            r += 1
        return r

    def intent(self, keys, c_start, c_end):
        if c_end <= self.clock or c_end <= c_start:
            return
        self.pending.append([c_start, self.seq, c_end, list(keys), 0])
        self.seq += 1

    def _evict_expired(self):
        gone = [k for k, u in self.until.items() if u <= self.clock]
        for k in gone:
            del self.until[k]
            self.count[self.range_of(k)] -= 1
        self.evicted_total += len(gone)
        return gone

    def _act(self, horizon):
        """Act on pending intents with C_start < horizon, in order."""
        staged = []
        self.pending.sort(key=lambda e: (e[0], e[1]))
        while self.pending and self.pending[0][0] < horizon:
            c_start, _, c_end, keys, i = self.pending[0]
            if c_end <= self.clock:      # expired while pending: nothing to act upon
                self.pending.pop(0)
                continue
            while i < len(keys):
                k = keys[i]
                if 0 <= k < self.num_keys:
                    if k in self.until:
                        self.until[k] = max(self.until[k], c_end)
                    else:
                        r = self.range_of(k)
                        if self.count[r] >= self.cap[r]:
                            self.pending[0][4] = i
                            return staged
                        self.until[k] = c_end
                        self.count[r] += 1
                        staged.append(k)
                        self.staged_total += 1
                i += 1
            self.pending.pop(0)
        return staged

    def round(self):
        """A communication round: Algorithm 1, then expiries, then actions."""
        self.lam, horizon = action_timing(self.lam, self.round_clock, self.clock, self.alpha, self.p)
        self.round_clock = self.clock
        self.last_horizon = horizon
        evicted = self._evict_expired()
        staged = self._act(horizon)
        return staged, evicted

    def advance_clock(self):
        """The worker raises its clock; intents now active but not acted upon
        are acted upon at once."""
        self.clock += 1
        if any(e[0] <= self.clock for e in self.pending):
            self.forced += 1
            self._evict_expired()
            self._act(self.clock + 1)

    def resident(self):
        return set(self.until)
