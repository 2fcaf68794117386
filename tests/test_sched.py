"""Slice scheduling across GPUs (Greedy-Least-Loaded) and bursty preemption
caps: the oracle pinned by hand-worked cases and by the competitive bound the
paper states (Appendix C: peak slice load under GLL at most (m+3)/2 times an
offline optimum), checked against brute-force optima on tiny traces; the
library's ema_sched_* against the oracle on random traces.
"""
import itertools

import numpy as np
import pytest

import oracle


def _lib():
    from paper_2609_27040_amd import ema
    return ema


# ---- oracle pins -------------------------------------------------------------------

def test_gll_hand_worked():
    s = oracle.SchedOracle(3, 4, 0)
    assert s.place(0, 0, 3, 0) == [1, 2, 1]      # tie -> lowest peer, then the emptier slice
    assert s.place(1, 0, 2, 0) == [2, 2]         # {1,0} holds 2 of GPU 0's units
    # {2,0} holds 1 (GPU 0's), {2,1} holds 2 (GPU 1's): 0; then 2 vs 2, tie: 0; then 3 vs 2: 1
    assert s.place(2, 7, 3, 0) == [0, 0, 1]
    # full slices refuse: {0,1} and {0,2} at 4
    s2 = oracle.SchedOracle(3, 2, 0)
    assert s2.place(0, 0, 5, 0) == [1, 2, 1, 2, -1]
    s2.release(0, 0, 2)                          # most recent first: the units on 2 and 1
    assert s2.use[0][1] == 1 and s2.use[0][2] == 1


def test_release_is_per_request_and_lifo():
    s = oracle.SchedOracle(4, 10, 0)
    a = s.place(0, 1, 3, 0)
    b = s.place(0, 2, 2, 0)
    s.release(0, 1, 1)                            # the last unit of request 1
    assert s.held[(0, 1)] == a[:2] and s.held[(0, 2)] == b
    with pytest.raises(ValueError):
        s.release(0, 2, 3)


def test_preemption_cap_hand_worked():
    T = 10
    s = oracle.SchedOracle(2, 10, T)              # one slice {0, 1}
    s.place(0, 0, 7, 0)
    s.preempted(0, 1, 5)                          # 7 of 10 > half: capped at 7 until tick 15
    s.release(0, 0, 3)                            # 4 held
    assert s.place(0, 0, 5, 6) == [1, 1, 1, -1, -1]   # back up to the cap only
    s.release(0, 0, 2)                            # 5 held
    s.preempted(0, 1, 12)                         # 5 of 10 is not above half: nothing changes
    assert s.active_cap(0, 1, 12) == 7
    s.place(0, 0, 1, 12)                          # 6 held
    s.preempted(0, 1, 13)                         # lower level within the window: cap 6 until 23
    assert s.active_cap(0, 1, 22) == 6 and s.active_cap(0, 1, 23) is None
    assert s.place(0, 0, 1, 20) == [-1]
    assert s.place(0, 0, 2, 23) == [1, 1]         # the window passed: cap lifted
    s0 = oracle.SchedOracle(2, 10, 0)             # window 0: no caps at all
    s0.place(0, 0, 9, 0)
    s0.preempted(0, 1, 0)
    assert s0.active_cap(0, 1, 0) is None


def _unit_trace(rng, m, n_units, horizon):
    """Unit jobs (gpu, arrival, departure), arrivals in time order."""
    jobs = []
    for _ in range(n_units):
        a = int(rng.integers(0, horizon))
        jobs.append((int(rng.integers(0, m)), a, a + 1 + int(rng.integers(0, horizon))))
    return sorted(jobs, key=lambda j: j[1])


def _peak(m, jobs, choice):
    """Peak total load over slices and ticks when job k sits on {gpu_k, choice[k]}."""
    horizon = max(d for _, _, d in jobs)
    peak = 0
    for t in range(horizon + 1):
        load = {}
        for (g, a, d), j in zip(jobs, choice):
            if a <= t < d:
                e = (min(g, j), max(g, j))
                load[e] = load.get(e, 0) + 1
        peak = max([peak] + list(load.values()))
    return peak


def _gll_choices(m, jobs):
    """GLL with unlimited capacity, events processed tick by tick (releases of
    a tick before its arrivals), one request per unit."""
    s = oracle.SchedOracle(m, 10 ** 9, 0)
    horizon = max(d for _, _, d in jobs)
    choice = [None] * len(jobs)
    for t in range(horizon + 1):
        for k, (g, a, d) in enumerate(jobs):
            if d == t and choice[k] is not None:
                s.release(g, k, 1)
        for k, (g, a, d) in enumerate(jobs):
            if a == t:
                choice[k] = s.place(g, k, 1, t)[0]
    return choice


@pytest.mark.parametrize("m,n_units,seed", [(3, 8, s) for s in range(6)] +
                                           [(4, 6, s) for s in range(6)])
def test_gll_peak_within_the_stated_bound_of_the_offline_optimum(m, n_units, seed):
    rng = np.random.default_rng(100 * m + seed)
    jobs = _unit_trace(rng, m, n_units, horizon=5)
    gll = _peak(m, jobs, _gll_choices(m, jobs))
    peers = [[j for j in range(m) if j != g] for g, _, _ in jobs]
    opt = min(_peak(m, jobs, c) for c in itertools.product(*peers))
    assert opt >= 1 and gll <= (m + 3) / 2 * opt, (gll, opt)


def test_gll_on_an_adversarial_pile_up():
    # three GPUs; GPU 0's early units spread over both slices, later GPU 1 and
    # GPU 2 load the slice GPU 0 could have avoided: GLL stays within the bound
    m = 3
    jobs = [(0, 0, 9), (0, 0, 9), (1, 1, 9), (1, 1, 9), (2, 2, 9), (2, 2, 9)]
    gll = _peak(m, jobs, _gll_choices(m, jobs))
    peers = [[j for j in range(m) if j != g] for g, _, _ in jobs]
    opt = min(_peak(m, jobs, c) for c in itertools.product(*peers))
    assert gll <= (m + 3) / 2 * opt


# ---- library against the oracle ----------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_library_scheduler_matches_oracle_on_random_traces(seed):
    ema = _lib()
    rng = np.random.default_rng(seed)
    m, units, T = int(rng.integers(2, 7)), int(rng.integers(3, 30)), int(rng.integers(0, 8))
    lib = ema.Scheduler(m, units, T)
    st = oracle.SchedOracle(m, units, T)
    try:
        reqs = {}
        for t in range(300):
            op = rng.choice(["place", "place", "release", "preempt"])
            g = int(rng.integers(0, m))
            if op == "place":
                r, n = int(rng.integers(0, 5)), int(rng.integers(1, 6))
                assert lib.place(g, r, n, t) == st.place(g, r, n, t)
                reqs[(g, r)] = len(st.held.get((g, r), []))
            elif op == "release":
                held = [(k, v) for k, v in reqs.items() if v > 0]
                if held:
                    (g, r), h = held[int(rng.integers(0, len(held)))]
                    n = int(rng.integers(1, h + 1))
                    lib.release(g, r, n)
                    st.release(g, r, n)
                    reqs[(g, r)] = h - n
            else:
                j = int(rng.integers(0, m - 1))
                j = j if j < g else j + 1
                lib.preempted(g, j, t)
                st.preempted(g, j, t)
            use, cap = lib.usage(t)
            assert use.tolist() == st.use
            want = [[-1 if st.active_cap(i, j, t) is None else st.active_cap(i, j, t)
                     for j in range(m)] for i in range(m)]
            assert cap.tolist() == want
    finally:
        lib.close()


def test_library_scheduler_errors():
    ema = _lib()
    with pytest.raises(ema.EmaError):
        ema.Scheduler(1, 4)
    s = ema.Scheduler(3, 4)
    try:
        with pytest.raises(ema.EmaError):
            s.place(3, 0, 1)
        with pytest.raises(ema.EmaError):
            s.release(0, 0, 1)                  # holds nothing
        with pytest.raises(ema.EmaError):
            s.preempted(0, 0, 0)                # a GPU has no slice with itself
    finally:
        s.close()
