"""Pins of the oracle's WSP simulation (HetPipe Sec. 4 and Sec. 5).

The worked examples of the paper are literal fixtures (tests/golden); the
staleness and clock bounds the paper derives are checked as invariants over
many schedules; two special cases are compared with independent textbook
recursions (sequential SGD and delayed SGD) and one (D = 0) with an exact
rational brute force built from the paper's description of which updates a
minibatch includes.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import seeded_inputs as si
from oracle import wsp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "wsp_worked_examples.json")


def quad_grad(a):
    """Gradient of f_{n,q}(w) = 1/2 |w - a[n, q]|^2."""
    return lambda n, q, w: w - a[(n, q)]


def targets(N, Q, dim, seed=5, dtype=np.float32):
    out = {}
    for n in range(N):
        for q in range(1, Q + 1):
            out[(n, q)] = si.normal(si.stream_key(seed, n, q, si.T_Y), dim).astype(dtype)
    return out


def run(N, s_local, D, waves, periods=None, dim=3, lr=0.1, record=False, dtype=np.float32):
    W = s_local + 1
    a = targets(N, waves * W, dim, dtype=np.float64 if dtype is np.float64 else np.float32)
    w0 = np.zeros(dim, dtype)
    sim = wsp.WSP(w0, N, s_local, D, lr, quad_grad(a), periods=periods, dtype=dtype, record=record)
    sim.run(waves)
    return sim


def mb_events(sim):
    return {(e[1], e[2]): e[3] for e in sim.events if e[0] == "mb"}


# ------------------------------------------------------------ worked examples

def test_worked_examples_from_the_paper():
    ex = json.load(open(GOLDEN))["examples"]
    for e in ex:
        if "own_updates" in e:
            sim = run(e["N"], e["s_local"], e["D"], 3)
            V = mb_events(sim)[(e["vw"], e["q"])]
            assert V[e["vw"]] == e["own_updates"], e["cite"]
        elif "minibatches" in e:
            W = e["s_local"] + 1
            c = e["wave"]
            assert list(range(c * W + 1, (c + 1) * W + 1)) == e["minibatches"], e["cite"]
            sim = run(1, e["s_local"], 0, 3)
            pushes = [ev for ev in sim.events if ev[0] == "push"]
            # the second push closes wave 1 and directly follows minibatch 8
            i = sim.events.index(pushes[1])
            assert sim.events[i - 1][:3] == ("mb", 0, e["minibatches"][-1]), e["cite"]
        elif "min_updates_every_vw" in e:
            sim = run(e["N"], e["s_local"], e["D"], 4, periods=[1, 2][:e["N"]])
            V = mb_events(sim)[(e["vw"], e["q"])]
            assert min(V) >= e["min_updates_every_vw"], (e["cite"], V)
            if "push_after" in e:
                ev = sim.events
                first_push = next(i for i, x in enumerate(ev) if x[0] == "push" and x[1] == e["vw"])
                assert ev[first_push - 1][:3] == ("mb", e["vw"], e["push_after"]), e["cite"]
        elif "s_global" in e:
            assert wsp.s_global(e["D"], e["s_local"]) == e["s_global"], e["cite"]
        elif "first_pull_after_wave" in e:
            sim = run(e["N"], e["s_local"], e["D"], 6, periods=[1, 3])
            W = e["s_local"] + 1
            # no pull before the VW has completed wave D (clock D+1)
            clock = {n: 0 for n in range(e["N"])}
            for ev in sim.events:
                if ev[0] == "push":
                    clock[ev[1]] = ev[2]
                if ev[0] == "pull":
                    assert clock[ev[1]] >= e["first_pull_after_wave"] + 1, e["cite"]
            assert any(ev[0] == "pull" for ev in sim.events)
            del W


# ------------------------------------------------------------------ invariants

SCHEDULES = [
    # N, s_local, D, waves, periods
    (1, 0, 0, 4, None),
    (1, 3, 0, 4, None),
    (2, 3, 0, 4, None),
    (2, 3, 0, 5, [1, 2]),
    (3, 2, 1, 6, [1, 1, 3]),
    (4, 3, 1, 5, [1, 1, 1, 2]),
    (4, 1, 2, 7, [1, 2, 3, 5]),
    (3, 4, 0, 4, [2, 3, 1]),
    (2, 0, 3, 8, [1, 4]),
]


@pytest.mark.parametrize("sched", SCHEDULES)
def test_local_staleness_is_exact(sched):
    """I1: minibatch q holds exactly the own updates 1 .. q - W (Sec. 4)."""
    N, s_local, D, waves, periods = sched
    W = s_local + 1
    sim = run(N, s_local, D, waves, periods)
    for (n, q), V in mb_events(sim).items():
        assert V[n] == max(0, q - W), (n, q, V)


@pytest.mark.parametrize("sched", SCHEDULES)
def test_global_staleness_bound(sched):
    """I2: for q > (D+1)W + s_local every VW's updates 1 .. q - (s_global+1) are in
    w_q (Sec. 5); before that only own updates may be present."""
    N, s_local, D, waves, periods = sched
    W = s_local + 1
    sg = wsp.s_global(D, s_local)
    sim = run(N, s_local, D, waves, periods)
    attained = False
    for (n, q), V in mb_events(sim).items():
        if q > (D + 1) * W + s_local:
            for m in range(N):
                assert V[m] >= q - (sg + 1), (n, q, V)
                if m != n and V[m] == q - (sg + 1):
                    attained = True
        else:
            assert all(V[m] == 0 for m in range(N) if m != n), (n, q, V)
    if N > 1 and waves * W > (D + 1) * W + s_local + W:
        assert attained


@pytest.mark.parametrize("sched", SCHEDULES)
def test_clock_distance_bound(sched):
    """I3: a VW continues past a wave end only within D clocks of c_g; local
    clocks never spread more than D+1 apart (the +1 is the wave just pushed
    while waiting)."""
    N, s_local, D, waves, periods = sched
    sim = run(N, s_local, D, waves, periods)
    clock = [0] * N
    g = [0] * N
    blocked = [False] * N
    for ev in sim.events:
        if ev[0] == "push":
            clock[ev[1]] = ev[2]
            assert ev[3] == min(clock)
        elif ev[0] == "pull":
            g[ev[1]] = ev[2]
            blocked[ev[1]] = False
        elif ev[0] == "block":
            blocked[ev[1]] = True
        elif ev[0] == "mb":
            n = ev[1]
            assert not blocked[n]
            assert clock[n] - g[n] <= D, ev
        assert max(clock) - min(clock) <= D + 1


@pytest.mark.parametrize("sched", SCHEDULES)
def test_push_is_sum_of_wave_updates_and_server_is_sum_of_pushes(sched):
    """I4 (u~ = sum of the wave's W updates, Sec. 5) and I5 (w_g = w_0 + sum of
    pushes in push order)."""
    N, s_local, D, waves, periods = sched
    W = s_local + 1
    sim = run(N, s_local, D, waves, periods, record=True, dtype=np.float64)
    for n, c, ut in sim.pushes:
        s = sum(sim.updates[(n, q)] for q in range(c * W + 1, (c + 1) * W + 1))
        np.testing.assert_allclose(ut, s, rtol=1e-14, atol=1e-15)
    total = sum(ut for _, _, ut in sim.pushes)
    np.testing.assert_allclose(sim.wg, total, rtol=1e-13, atol=1e-15)
    assert len(sim.pushes) == N * waves


# -------------------------------------------- special cases with closed forms

def test_single_vw_no_pipelining_is_sequential_sgd():
    """I6: N = 1, s_local = 0 is plain sequential SGD (Sec. 4, N_m = 1)."""
    lr, Q, dim = 0.3, 12, 4
    sim = run(1, 0, 0, Q, lr=lr, dim=dim, dtype=np.float64)
    a = targets(1, Q, dim, dtype=np.float64)
    w = np.zeros(dim)
    for q in range(1, Q + 1):
        w = w - lr * (w - a[(0, q)])
    np.testing.assert_allclose(sim.wg, w, rtol=1e-13)
    np.testing.assert_allclose(sim.ring[0][0], w, rtol=1e-13)


@pytest.mark.parametrize("s_local,D", [(1, 0), (3, 0), (3, 2), (4, 1)])
def test_single_vw_is_delayed_sgd(s_local, D):
    """I6: with one VW, minibatch q runs at w_0 + sum_{j <= q-W} u_j whatever D is."""
    lr, waves, dim = 0.2, 5, 3
    W = s_local + 1
    sim = run(1, s_local, D, waves, lr=lr, dim=dim, dtype=np.float64, record=True)
    a = targets(1, waves * W, dim, dtype=np.float64)
    u = {}
    for q in range(1, waves * W + 1):
        wq = np.zeros(dim) + sum((u[j] for j in range(1, q - W + 1)), np.zeros(dim))
        u[q] = -lr * (wq - a[(0, q)])
        np.testing.assert_allclose(sim.updates[(0, q)], u[q], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(sim.wg, sum(u.values()), rtol=1e-12)


@pytest.mark.parametrize("N,s_local,periods", [(2, 3, [1, 2]), (3, 1, [3, 1, 2]), (3, 2, [1, 1, 1])])
def test_bsp_like_D0_exact_rational_brute_force(N, s_local, periods):
    """I8: with D = 0 (Sec. 5: BSP-like) the weights of minibatch q of VW n hold
    exactly its own updates 1..q-W plus every other VW's updates of the waves
    completed before its last pull, i.e. 1 .. W*(floor(q/W)-1).  Built from that
    description alone in exact rationals, independent of the schedule."""
    W = s_local + 1
    waves, dim = 4, 2
    lr = Fraction(1, 5)
    a64 = targets(N, waves * W, dim, dtype=np.float64)
    a = {k: [Fraction(float(v)) for v in arr] for k, arr in a64.items()}
    u = {}
    V_expect = {}
    for q in range(1, waves * W + 1):
        for n in range(N):
            other = W * max(0, q // W - 1)
            inc = [(n, j) for j in range(1, q - W + 1)]
            inc += [(m, j) for m in range(N) if m != n for j in range(1, other + 1)]
            w = [sum((u[k][d] for k in inc), Fraction(0)) for d in range(dim)]
            u[(n, q)] = [-lr * (w[d] - a[(n, q)][d]) for d in range(dim)]
            V_expect[(n, q)] = tuple(max(0, q - W) if m == n else other for m in range(N))
    # the oracle in exact rational arithmetic
    sim = wsp.WSP(np.array([Fraction(0)] * dim, dtype=object), N, s_local, 0, lr,
                  lambda n, q, w: np.array([w[d] - a[(n, q)][d] for d in range(dim)], dtype=object),
                  periods=periods, dtype=object, record=True)
    sim.run(waves)
    assert mb_events(sim) == V_expect
    for k, uk in u.items():
        assert list(sim.updates[k]) == uk
    wg = [sum((u[k][d] for k in u), Fraction(0)) for d in range(dim)]
    assert list(sim.wg) == wg


def test_event_log_is_deterministic():
    s1 = run(4, 3, 1, 5, [1, 1, 1, 2])
    s2 = run(4, 3, 1, 5, [1, 1, 1, 2])
    assert s1.events == s2.events
    blocks = [e for e in s1.events if e[0] == "block"]
    assert len(blocks) > 0


def test_equal_periods_with_D1_never_block():
    sim = run(4, 3, 1, 5)
    assert not any(e[0] == "block" for e in sim.events)


def test_stopped_worker_deadlocks_the_others():
    W = 4
    a = targets(3, 40, 2)
    sim = wsp.WSP(np.zeros(2, np.float32), 3, 3, 0, 0.1, quad_grad(a))
    with pytest.raises(wsp.DeadlockError):
        sim.run(10, stop_vw=2, stop_after=W + 2)
    # the other VWs got at most D+1 waves ahead of the stopped one before blocking
    assert all(sim.blocked[n] for n in (0, 1))
    del W


# ---------------------------------------------------------------- optimizer variants

def test_theorem1_schedule_numbers_updates_across_workers():
    # Theorem 1: eta_t = sigma / sqrt(t); the updates of all VWs form one
    # sequence taking the VWs in turn (minibatch q of VW n is update (q-1)N+n+1)
    lr = wsp.theorem1_schedule(0.6, 3)
    assert lr(0, 1) == pytest.approx(0.6)
    assert lr(2, 1) == pytest.approx(0.6 / np.sqrt(3))
    assert lr(0, 2) == pytest.approx(0.3)
    assert lr(1, 5) == pytest.approx(0.6 / np.sqrt(14))


def test_schedule_single_worker_is_plain_sgd():
    # N = 1, s_local = 0: w_{t+1} = w_t - sigma/sqrt(t) * grad(w_t)
    a = np.array([0.5, -1.0, 2.0], np.float32)
    w0 = np.array([1.0, 2.0, -3.0], np.float32)
    lr = wsp.theorem1_schedule(0.3, 1)
    sim = wsp.WSP(w0, 1, 0, 0, lr, lambda n, q, w: w - a)
    sim.run(6)
    w = w0.copy()
    for t in range(1, 7):
        w = w + (-np.float32(0.3 / np.sqrt(t))) * (w - a)
    np.testing.assert_array_equal(sim.ring[0][0], w)


def test_momentum_matches_heavy_ball_matrix_power():
    # f(w) = a w^2 / 2, N = 1, no staleness: heavy ball is the linear map
    # (w, v) -> (w - eta (mu v + a w), mu v + a w); k steps = k-th matrix power
    a, eta, mu, w0 = Fraction(3, 2), Fraction(1, 5), Fraction(2, 3), Fraction(7, 4)
    sim = wsp.WSP(np.array([w0], dtype=object), 1, 0, 0, eta,
                   lambda n, q, w: np.array([a * w[0]], dtype=object), dtype=object,
                   momentum=mu)
    sim.run(7)
    Mx = [[1 - eta * a, -eta * mu], [a, mu]]

    def mul(A, B):
        return [[sum(A[i][k] * B[k][j] for k in range(2)) for j in range(2)] for i in range(2)]
    Pw = [[1, 0], [0, 1]]
    for _ in range(7):
        Pw = mul(Mx, Pw)
    assert sim.ring[0][0][0] == Pw[0][0] * w0
    assert sim.vel[0][0] == Pw[1][0] * w0


def test_momentum_with_local_staleness_brute_force():
    # N = 1, W = 3: minibatch q reads w0 + sum of u_1..u_{q-3}; velocity and
    # steps follow completion order.  Written directly from those two rules.
    a, eta, mu = Fraction(1, 2), Fraction(1, 3), Fraction(1, 2)
    w0 = Fraction(5)
    sim = wsp.WSP(np.array([w0], dtype=object), 1, 2, 0, eta,
                   lambda n, q, w: np.array([a * w[0] - 1], dtype=object), dtype=object,
                   momentum=mu)
    sim.run(4)
    us, v = [], Fraction(0)
    for q in range(1, 13):
        wq = w0 + sum(us[:max(0, q - 3)])
        v = mu * v + (a * wq - 1)
        us.append(-eta * v)
    assert sim.wg[0] == w0 + sum(us)
    assert sim.vel[0][0] == v
