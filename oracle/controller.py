"""Oracle of the runtime-adaptive proposal-length controller -- TEST
INFRASTRUCTURE ONLY (only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may use it).

Section 3.2, "Runtime-adaptive proposal-length controller", Eq. (1): for an
eligible retrieval of similarity s, pick the proposal length l in
0..l_max (proposals are also cut at their sequence boundary, so at most the
retrieved length) that minimises  T(l) / (A(l, s) + 1),  where T is the
predicted decoding-iteration latency and A the expected number of accepted
proposal tokens; the +1 is the model's own token that every iteration adds.
l = 0 is an ordinary greedy pass. After each iteration both estimators learn
from what was observed, online; now and then the controller tries a length
next to the best one.

The paper names the estimator families but not their features, step sizes or
exploration rule. The readings taken here (each is a documented choice):

* acceptance: two online logistic regressions over the features
  phi(j, s) = (1, s, j / l_max), j the 1-based position of a proposal token:
  P1(s) = sigmoid(w_first . phi(1, s)) is the probability that the first
  token is accepted, Pc(j, s) = sigmoid(w_cont . phi(j, s)) the probability
  that token j >= 2 is accepted given that token j - 1 was. Acceptance is a
  prefix, so A(l, s) = sum_{j=1..l} prod_{i=1..j} q_i with q_1 = P1 and
  q_i = Pc(i, s). Each model takes one stochastic-gradient step of the
  log-likelihood per sample (w += lr * (y - p) * x), the samples of an
  iteration that proposed l tokens and accepted a of them being: the first
  token (y = [a >= 1]) when l >= 1, and tokens j = 2..min(l, a + 1)
  (y = [a >= j]); tokens after the first rejection carry no information
  about the conditional probability and are not used;
* latency: log T(l) = theta . psi(l), psi(l) = (1, u, u^2), u = l / l_max,
  T in milliseconds, fitted by recursive least squares with forgetting
  factor `forget` (weights forget^age on past samples) from theta = 0 and
  covariance prior_var * I, i.e. the exponentially weighted ridge regression
  of log T on psi;
* exploration: every `explore_every`-th choice (0: never) takes a length
  next to the best one, alternately one above and one below (the other side
  where that one is out of range);
* ties of the objective go to the shorter length; an iteration with no
  eligible retrieval is a greedy pass (l = 0) whose latency is still learned.

All arithmetic is Python float (IEEE fp64), written out in plain loops.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List


def sigmoid(z: float) -> float:
    """Logistic function, evaluated without overflow on either side."""
    if z >= 0.0:
        return 1.0 / (1.0 + math.exp(-z))
    e = math.exp(z)
    return e / (1.0 + e)


@dataclass
class ControllerParams:
    l_max: int = 64
    lr: float = 0.05
    forget: float = 0.98
    prior_var: float = 100.0
    explore_every: int = 16


@dataclass
class Controller:
    """Estimator states and the choice rule of Eq. (1)."""
    params: ControllerParams = field(default_factory=ControllerParams)
    w_first: List[float] = field(default_factory=lambda: [0.0, 0.0, 0.0])
    w_cont: List[float] = field(default_factory=lambda: [0.0, 0.0, 0.0])
    theta: List[float] = field(default_factory=lambda: [0.0, 0.0, 0.0])
    P: List[List[float]] = None
    n_choose: int = 0
    n_explore: int = 0
    n_observe: int = 0

    def __post_init__(self):
        if self.P is None:
            v = self.params.prior_var
            self.P = [[v if r == c else 0.0 for c in range(3)] for r in range(3)]

    # ------------------------------------------------------------ features
    def phi(self, j: int, s: float) -> List[float]:
        return [1.0, s, j / self.params.l_max]

    def psi(self, l: int) -> List[float]:
        u = l / self.params.l_max
        return [1.0, u, u * u]

    # ------------------------------------------------------------ estimators
    def p_first(self, s: float) -> float:
        return sigmoid(_dot(self.w_first, self.phi(1, s)))

    def p_cont(self, j: int, s: float) -> float:
        return sigmoid(_dot(self.w_cont, self.phi(j, s)))

    def accept_prob(self, j: int, s: float) -> float:
        """q_j: token j accepted given that every earlier token was."""
        return self.p_first(s) if j == 1 else self.p_cont(j, s)

    def expected_accepted(self, l: int, s: float) -> float:
        """A(l, s): the sum over j of the probability that the first j
        proposal tokens are all accepted."""
        total = 0.0
        for j in range(1, l + 1):
            prefix = 1.0
            for i in range(1, j + 1):
                prefix *= self.accept_prob(i, s)
            total += prefix
        return total

    def latency(self, l: int) -> float:
        """T(l) in ms, the exponential of the fitted quadratic."""
        return math.exp(_dot(self.theta, self.psi(l)))

    def objective(self, l: int, s: float) -> float:
        """Eq. (1): predicted latency per token the iteration adds."""
        return self.latency(l) / (self.expected_accepted(l, s) + 1.0)

    # ------------------------------------------------------------ choice
    def best_length(self, s: float, avail: int) -> int:
        L = max(0, min(self.params.l_max, avail))
        best, best_j = 0, self.objective(0, s)
        for l in range(1, L + 1):
            j = self.objective(l, s)
            if j < best_j:
                best, best_j = l, j
        return best

    def choose(self, s: float, avail: int) -> int:
        """Length for this iteration: the argmin, or a neighbour of it on an
        exploring call."""
        L = max(0, min(self.params.l_max, avail))
        best = self.best_length(s, avail)
        self.n_choose += 1
        every = self.params.explore_every
        if every > 0 and L > 0 and self.n_choose % every == 0:
            up = self.n_explore % 2 == 0
            nb = best + 1 if up else best - 1
            if nb < 0 or nb > L:
                nb = best - 1 if up else best + 1
            self.n_explore += 1
            return nb
        return best

    # ------------------------------------------------------------ learning
    def _sgd(self, w: List[float], x: List[float], y: float) -> None:
        p = sigmoid(_dot(w, x))
        g = self.params.lr * (y - p)
        for k in range(3):
            w[k] += g * x[k]

    def _rls(self, x: List[float], y: float) -> None:
        lam = self.params.forget
        Px = [sum(self.P[r][c] * x[c] for c in range(3)) for r in range(3)]
        den = lam + _dot(x, Px)
        gain = [Px[r] / den for r in range(3)]
        err = y - _dot(self.theta, x)
        for r in range(3):
            self.theta[r] += gain[r] * err
        self.P = [[(self.P[r][c] - gain[r] * Px[c]) / lam for c in range(3)] for r in range(3)]

    def observe(self, l: int, s: float, accepted: int, latency_ms: float) -> None:
        """Learn from one iteration that proposed l tokens at similarity s,
        accepted `accepted` of them and took latency_ms."""
        if not (0 <= accepted <= l) or not latency_ms > 0.0:
            raise ValueError("observation out of range")
        if l >= 1:
            self._sgd(self.w_first, self.phi(1, s), 1.0 if accepted >= 1 else 0.0)
            for j in range(2, min(l, accepted + 1) + 1):
                self._sgd(self.w_cont, self.phi(j, s), 1.0 if accepted >= j else 0.0)
        self._rls(self.psi(l), math.log(latency_ms))
        self.n_observe += 1


def _dot(a, b) -> float:
    t = 0.0
    for x, y in zip(a, b):
        t += x * y
    return t
