"""Pins of the oracle's proposal-length controller (Section 3.2,
"Runtime-adaptive proposal-length controller", Eq. (1)).

Each check ties the oracle to something other than its own formulas: the
geometric closed form of the expected accepted length, the expectation taken
over the distribution of the accepted length and by simulation, the
continuous minimiser of the objective for latencies whose optimum is known
in closed form, the batch weighted ridge regression that recursive least
squares must equal, exact recovery of a noise-free log-quadratic, hand
values of the first gradient step, and the fixed point of the logistic
updates under a known Bernoulli rate."""
import math

import numpy as np
import pytest

from oracle.controller import Controller, ControllerParams, sigmoid


def _ctl(**kw):
    return Controller(ControllerParams(**kw))


# ------------------------------------------------------- expected acceptance

def test_expected_accepted_geometric_closed_form():
    c = _ctl(l_max=64)
    for a, b in ((0.3, -0.7), (2.0, 1.5), (-1.0, 3.0)):
        c.w_first = [a, 0.0, 0.0]
        c.w_cont = [b, 0.0, 0.0]
        p, q = 1.0 / (1.0 + math.exp(-a)), 1.0 / (1.0 + math.exp(-b))
        for l in (0, 1, 2, 7, 64):
            ref = p * (1.0 - q ** l) / (1.0 - q)
            assert abs(c.expected_accepted(l, 0.4) - ref) < 1e-12


def test_expected_accepted_from_distribution_and_simulation():
    # position- and similarity-dependent probabilities: the expectation of the
    # accepted length over its distribution (accept k, then reject token k+1)
    c = _ctl(l_max=16)
    c.w_first = [0.8, 1.2, 0.0]
    c.w_cont = [1.5, 0.5, -2.0]
    s, l = 0.6, 12
    q = [None] + [1.0 / (1.0 + math.exp(-(c.w_first[0] + c.w_first[1] * s + c.w_first[2] / 16)))]
    for j in range(2, l + 1):
        q.append(1.0 / (1.0 + math.exp(-(c.w_cont[0] + c.w_cont[1] * s + c.w_cont[2] * j / 16))))
    mean = 0.0
    for k in range(l + 1):
        pk = 1.0
        for i in range(1, k + 1):
            pk *= q[i]
        if k < l:
            pk *= 1.0 - q[k + 1]
        mean += k * pk
    assert abs(c.expected_accepted(l, s) - mean) < 1e-12
    # and by simulation
    rng = np.random.default_rng(5)
    n = 200000
    u = rng.random((n, l))
    acc = np.zeros(n, np.int64)
    alive = np.ones(n, bool)
    for j in range(1, l + 1):
        alive &= u[:, j - 1] < q[j]
        acc += alive
    sim = acc.mean()
    assert abs(sim - c.expected_accepted(l, s)) < 4 * acc.std() / math.sqrt(n)


# ------------------------------------------------------------ Eq. (1) argmin

def _sure_accept(c):
    # sigmoid(60) rounds to exactly 1.0 in fp64: every token is accepted, A(l) = l
    c.w_first = [60.0, 0.0, 0.0]
    c.w_cont = [60.0, 0.0, 0.0]
    assert c.expected_accepted(9, 0.0) == 9.0


def test_argmin_exponential_latency():
    # T = exp(b * l / l_max), A = l: minimise b l / l_max - log(l + 1), which
    # is convex with its stationary point at l = l_max / b - 1
    c = _ctl(l_max=64)
    _sure_accept(c)
    for target in (3, 9, 31):
        c.theta = [0.7, 64.0 / (target + 1), 0.0]
        assert c.best_length(0.5, 64) == target


def test_argmin_gaussian_latency():
    # T = exp(k u^2), u = l / l_max, A = l: stationary point where
    # l (l + 1) = l_max^2 / (2 k)
    c = _ctl(l_max=64)
    _sure_accept(c)
    for target in (15, 40):
        k = 64.0 ** 2 / (2.0 * target * (target + 1))
        c.theta = [-0.2, 0.0, k]
        assert c.best_length(0.1, 64) == target


def test_argmin_special_cases():
    c = _ctl(l_max=32)
    # flat latency and positive acceptance: A increases with l -> the longest
    # (q = sigmoid(3) keeps every increment of A far above rounding)
    c.w_first, c.w_cont = [0.0, 0.0, 0.0], [3.0, 0.0, 0.0]
    c.theta = [1.0, 0.0, 0.0]
    assert c.best_length(0.3, 100) == 32
    assert c.best_length(0.3, 5) == 5     # cut at the retrieved length
    assert c.best_length(0.3, 0) == 0
    # nothing is ever accepted and latency grows: a greedy pass
    c.w_first = [-800.0, 0.0, 0.0]
    c.theta = [1.0, 0.5, 0.0]
    assert c.expected_accepted(32, 0.3) == 0.0
    assert c.best_length(0.3, 32) == 0
    # all objectives equal: the shortest
    c.theta = [1.0, 0.0, 0.0]
    assert c.best_length(0.3, 32) == 0


def test_similarity_moves_the_choice():
    # acceptance rising with similarity, latency rising with length: a higher
    # similarity never gives a shorter proposal
    c = _ctl(l_max=64)
    c.w_first = [-2.0, 6.0, 0.0]
    c.w_cont = [-1.0, 5.0, 0.0]
    c.theta = [0.9, 0.4, 0.6]
    ls = [c.best_length(s, 64) for s in np.linspace(-1.0, 1.0, 21)]
    assert ls == sorted(ls) and ls[0] == 0 and ls[-1] > 8


# ------------------------------------------------------------ latency fit

@pytest.mark.parametrize("forget", [1.0, 0.9])
def test_rls_equals_weighted_ridge(forget):
    rng = np.random.default_rng(11)
    c = _ctl(l_max=64, forget=forget, prior_var=7.0)
    ls = rng.integers(0, 65, 40)
    ts = rng.uniform(1.0, 6.0, 40)
    for l, t in zip(ls, ts):
        c.observe(int(l), 0.0, 0, float(t))
    n = len(ls)
    X = np.stack([[1.0, l / 64, (l / 64) ** 2] for l in ls])
    y = np.log(ts)
    wts = forget ** (n - 1 - np.arange(n))
    A = (X * wts[:, None]).T @ X + forget ** n / 7.0 * np.eye(3)
    b = (X * wts[:, None]).T @ y
    theta = np.linalg.solve(A, b)
    assert np.allclose(c.theta, theta, rtol=1e-9, atol=1e-10)
    assert np.allclose(np.array(c.P), np.linalg.inv(A), rtol=1e-8, atol=1e-12)


def test_rls_recovers_noise_free_log_quadratic():
    c = _ctl(l_max=64, forget=1.0, prior_var=1e10)
    a, b, k = 0.9, 0.3, 0.45
    for l in [0, 4, 8, 16, 32, 64] * 3:
        u = l / 64
        c.observe(l, 0.0, 0, math.exp(a + b * u + k * u * u))
    assert np.allclose(c.theta, [a, b, k], atol=1e-6)
    assert abs(c.latency(24) - math.exp(a + b * 0.375 + k * 0.375 ** 2)) < 1e-6


# ------------------------------------------------------------ acceptance fit

def test_first_gradient_step_by_hand():
    # from zero weights every probability is 1/2, so the first step of each
    # model is lr * (y - 1/2) * x
    c = _ctl(l_max=8, lr=0.5)
    c.observe(2, 0.2, 1, 3.0)
    assert c.w_first == [0.25, 0.05, 0.03125]            # y = 1, x = (1, .2, 1/8)
    assert c.w_cont == [-0.25, -0.05, -0.0625]           # y = 0, x = (1, .2, 2/8)
    # nothing proposed: only the latency model learns
    c2 = _ctl(l_max=8, lr=0.5)
    c2.observe(0, 0.9, 0, 2.0)
    assert c2.w_first == [0.0] * 3 and c2.w_cont == [0.0] * 3
    assert c2.theta[0] != 0.0


def test_conditional_samples():
    # l = 5, a = 3: continuation samples at j = 2, 3 (accepted) and 4
    # (rejected); j = 5 comes after the first rejection and is not a sample.
    # With a tiny step the update is lr * sum_j (y_j - 1/2) x_j to first order
    lr, s, lm = 1e-9, 0.3, 16
    c = _ctl(l_max=lm, lr=lr)
    c.observe(5, s, 3, 2.0)
    ref = [0.5, 0.5 * s, 0.5 * (2 + 3 - 4) / lm]
    assert np.allclose(np.array(c.w_cont) / lr, ref, rtol=1e-6)
    assert np.allclose(np.array(c.w_first) / lr, [0.5, 0.5 * s, 0.5 / lm], rtol=1e-6)
    # everything accepted: j = 2..5, all positive
    c = _ctl(l_max=lm, lr=lr)
    c.observe(5, s, 5, 2.0)
    assert np.allclose(np.array(c.w_cont) / lr, [2.0, 2.0 * s, 0.5 * 14 / lm], rtol=1e-6)
    # first token rejected: no continuation sample at all
    c = _ctl(l_max=lm, lr=lr)
    c.observe(5, s, 0, 2.0)
    assert c.w_cont == [0.0] * 3


def test_logistic_fixed_point():
    # Bernoulli(0.3) labels at one feature vector: the stochastic gradient's
    # fixed point is the rate itself
    rng = np.random.default_rng(3)
    c = _ctl(l_max=8, lr=0.01)
    ys = rng.random(30000) < 0.3
    for y in ys:
        c.observe(1, 0.5, int(y), 1.0)
    assert abs(c.p_first(0.5) - 0.3) < 0.03


def test_observe_rejects_bad_input():
    c = _ctl()
    for args in ((3, 0.0, 4, 1.0), (3, 0.0, -1, 1.0), (3, 0.0, 1, 0.0), (3, 0.0, 1, float("nan"))):
        with pytest.raises(ValueError):
            c.observe(*args)


# ------------------------------------------------------------ exploration

def test_exploration_schedule():
    c = _ctl(l_max=16, explore_every=3)
    _sure_accept(c)
    c.theta = [0.0, 16.0 / 6, 0.0]          # best length 5 (exponential case)
    assert c.best_length(0.0, 16) == 5
    got = [c.choose(0.0, 16) for _ in range(9)]
    assert got == [5, 5, 6, 5, 5, 4, 5, 5, 6]
    assert c.n_explore == 3
    # at the top of the range the upward step turns down, at zero the
    # downward step turns up
    c = _ctl(l_max=16, explore_every=1)
    _sure_accept(c)
    c.theta = [0.0, 0.0, 0.0]               # flat latency: best is the cap
    assert [c.choose(0.0, 4) for _ in range(2)] == [3, 3]
    c.w_first = [-800.0, 0.0, 0.0]          # best is 0
    c.theta = [0.0, 1.0, 0.0]
    assert [c.choose(0.0, 4) for _ in range(2)] == [1, 1]
    # no range to explore
    assert c.choose(0.0, 0) == 0
    # never exploring
    c = _ctl(l_max=16, explore_every=0)
    _sure_accept(c)
    assert {c.choose(0.0, 16) for _ in range(40)} == {16}


def test_sigmoid_extremes():
    assert sigmoid(0.0) == 0.5
    assert sigmoid(-800.0) == 0.0 and sigmoid(800.0) == 1.0
    assert abs(sigmoid(math.log(3.0)) - 0.75) < 1e-15
