"""Parity of the library's proposal-length controller (host C++, fp64) with
the oracle's (Section 3.2, "Runtime-adaptive proposal-length controller",
Eq. (1)), through the C ABI. Host code only: runs without a GPU.

Estimator states must agree to 1e-12 relative after every observation; the
objective rows likewise. Where the oracle's best objective beats the
runner-up by more than 1e-9 relative, the chosen length must be the same;
closer than that, it must lie among the near-tied lengths."""
import math

import numpy as np
import pytest

import paper_2609_32166_amd as pf
from oracle.controller import Controller, ControllerParams

TOL = 1e-12


def _pair(**kw):
    prm = ControllerParams(**kw)
    lib_ctl = pf.pf_ctl_create(prm.l_max, prm.explore_every, prm.lr, prm.forget, prm.prior_var)
    return lib_ctl, Controller(prm)


def _close(a, b, tol=TOL):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return np.all(np.abs(a - b) <= tol * np.maximum(1.0, np.abs(b)))


def _same_state(lib_ctl, orc):
    st = pf.pf_ctl_get_state(lib_ctl)
    assert _close(list(st.w_first), orc.w_first)
    assert _close(list(st.w_cont), orc.w_cont)
    assert _close(list(st.theta), orc.theta)
    assert _close(list(st.P), [v for row in orc.P for v in row], 1e-11)
    assert (st.n_choose, st.n_explore, st.n_observe) == (orc.n_choose, orc.n_explore,
                                                         orc.n_observe)


def _same_choice(lib_l, orc, s, avail, orc_l, exploring):
    L = max(0, min(orc.params.l_max, avail))
    J = np.array([orc.objective(l, s) for l in range(L + 1)])
    if exploring:
        assert lib_l == orc_l
        return
    order = np.sort(J)
    if len(J) == 1 or order[1] - order[0] > 1e-9 * order[0]:
        assert lib_l == orc_l
    else:
        assert J[lib_l] <= order[0] * (1 + 1e-9)


def _latency(l, rng):
    # a synthetic iteration latency: flat while the rows fit one 16-row tile,
    # then a step per extra tile plus a linear part, with 2% noise
    return (2.4 + 0.25 * ((l + 15) // 16) + 0.012 * l) * (1.0 + 0.02 * rng.standard_normal())


@pytest.mark.parametrize("l_max,every,lr,forget,prior", [(64, 16, 0.05, 0.98, 100.0),
                                                         (16, 3, 0.2, 1.0, 5.0),
                                                         (7, 0, 0.01, 0.9, 1e4),
                                                         (1, 2, 0.1, 0.95, 10.0)])
def test_stream_parity(l_max, every, lr, forget, prior):
    rng = np.random.default_rng(l_max * 7 + every)
    lib_ctl, orc = _pair(l_max=l_max, explore_every=every, lr=lr, forget=forget, prior_var=prior)
    for it in range(300):
        s = float(rng.uniform(-1.0, 1.0))
        avail = int(rng.integers(0, l_max + 3))
        # objective rows without side effects
        J_lib, best_lib = pf.pf_ctl_objective(lib_ctl, s, avail)
        L = max(0, min(l_max, avail))
        J_orc = [orc.objective(l, s) for l in range(L + 1)]
        assert _close(J_lib, J_orc)
        n_explore = orc.n_explore
        l_orc = orc.choose(s, avail)
        l_lib = pf.pf_ctl_choose(lib_ctl, s, avail)
        _same_choice(l_lib, orc, s, avail, l_orc, orc.n_explore != n_explore)
        assert best_lib == orc.best_length(s, avail) or _close(J_orc[best_lib], min(J_orc), 1e-9)
        # observe the oracle's choice on both sides so the streams stay equal
        l = l_orc
        q = 1.0 / (1.0 + math.exp(-(3.0 * s)))
        acc = 0
        while acc < l and rng.random() < q:
            acc += 1
        t = _latency(l, rng)
        orc.observe(l, s, acc, t)
        pf.pf_ctl_observe(lib_ctl, l, s, acc, t)
        _same_state(lib_ctl, orc)


def test_closed_form_minimisers_through_the_abi():
    # every token accepted (sigmoid(60) is 1.0 in fp64), T = exp(b l / l_max):
    # the optimum sits at l = l_max / b - 1
    lib_ctl, _ = _pair(l_max=64)
    for target in (0, 3, 9, 31, 63):
        st = pf.pf_ctl_get_state(lib_ctl)
        st.w_first[:] = [60.0, 0.0, 0.0]
        st.w_cont[:] = [60.0, 0.0, 0.0]
        st.theta[:] = [0.3, 64.0 / (target + 1), 0.0]
        pf.pf_ctl_set_state(lib_ctl, st)
        J, best = pf.pf_ctl_objective(lib_ctl, 0.2, 64)
        assert best == target, (target, best)
        assert abs(J[9] - math.exp(0.3 + 9 / (target + 1)) / 10.0) < 1e-12 * J[9]
    # the cap at the retrieved length
    J, best = pf.pf_ctl_objective(lib_ctl, 0.2, 5)
    assert len(J) == 6 and best == 5


def test_learns_the_best_length():
    # acceptance q(s) per token, latency from the tile staircase: after a few
    # hundred iterations the library's choice is within 3% of the best
    # objective computed from the true model
    rng = np.random.default_rng(9)
    lib_ctl, _ = _pair(l_max=64, explore_every=16, lr=0.05, forget=0.98, prior_var=100.0)

    def true_obj(l, q):
        A = sum(q ** j for j in range(1, l + 1))
        return (2.4 + 0.25 * ((l + 15) // 16) + 0.012 * l) / (A + 1.0)

    for s, q in ((0.9, 0.97), (0.2, 0.6)):
        for it in range(400):
            l = pf.pf_ctl_choose(lib_ctl, s, 64)
            acc = 0
            while acc < l and rng.random() < q:
                acc += 1
            pf.pf_ctl_observe(lib_ctl, l, s, acc, _latency(l, rng))
        _, best = pf.pf_ctl_objective(lib_ctl, s, 64)
        opt = min(true_obj(l, q) for l in range(65))
        assert true_obj(best, q) <= 1.03 * opt, (s, best, true_obj(best, q), opt)


def test_argument_errors():
    with pytest.raises(pf.PfError) as e:
        pf.pf_ctl_create(l_max=0)
    assert e.value.status == -1
    for kw in (dict(l_max=65), dict(lr=0.0), dict(forget=1.5), dict(forget=0.0),
               dict(prior_var=-1.0), dict(explore_every=-1)):
        with pytest.raises(pf.PfError):
            pf.pf_ctl_create(**kw)
    c = pf.pf_ctl_create(l_max=8)
    for args in ((9, 0.0, 0, 1.0), (3, 0.0, 4, 1.0), (3, 0.0, -1, 1.0), (-1, 0.0, 0, 1.0),
                 (2, 0.0, 1, 0.0), (2, 0.0, 1, float("inf")), (2, float("nan"), 1, 1.0)):
        with pytest.raises(pf.PfError) as e:
            pf.pf_ctl_observe(c, *args)
        assert e.value.status == -1
    with pytest.raises(pf.PfError):
        pf.pf_ctl_choose(c, float("nan"), 4)
    st = pf.pf_ctl_get_state(c)
    st.theta[1] = float("inf")
    with pytest.raises(pf.PfError):
        pf.pf_ctl_set_state(c, st)
    # nothing above changed the state
    st2 = pf.pf_ctl_get_state(c)
    assert list(st2.theta) == [0.0, 0.0, 0.0] and st2.n_observe == 0
    assert list(st2.P) == [100.0, 0, 0, 0, 100.0, 0, 0, 0, 100.0]
