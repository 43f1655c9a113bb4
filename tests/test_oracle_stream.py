"""Pins of the oracle's streaming-buffer simulation (§II-C Eqns 2 and 3, the
buffer policies and batch rule of §IV, Table II).

Checked against: the closed form of Eqn 2 (exact for a continuous stream as
long as every iteration can take its full batch), Eqn 3 with the printed
entries of Table II, the two statements of the text about the first
iterations, conservation of samples, the truncation bound, and a brute-force
simulation that moves individual samples through a FIFO queue.
"""
import collections
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")
P, TR = 0, 1


def arrivals_until(S, t_us, T):
    return S * t_us * T // 1_000_000


def brute_force(rates, iter_us, b_min, b_max, policy, T):
    """Every sample is an object in a FIFO queue: the device trains on the
    oldest ones; truncation keeps only the newest samples of the iteration."""
    K = len(rates)
    queued = np.zeros((T + 1, K), dtype=np.uint64)
    batch = np.zeros((T, K), dtype=np.uint64)
    dropped = np.zeros(K, dtype=np.uint64)
    for j, (S, t_us) in enumerate(zip(rates, iter_us)):
        b = min(max(S, b_min), b_max)
        q = collections.deque(range(S))          # sample ids, the first second of the stream
        next_id = S
        lost = 0
        queued[0, j] = len(q)
        for t in range(T):
            used = 0
            while used < b and q:
                q.popleft()
                used += 1
            batch[t, j] = used
            new = list(range(next_id, next_id + arrivals_until(S, t_us, t + 1) - arrivals_until(S, t_us, t)))
            next_id += len(new)
            if policy == P:
                q.extend(new)
            else:
                lost += len(q)
                keep = new[len(new) - min(len(new), S):]
                lost += len(new) - len(keep)
                q = collections.deque(keep)
                assert all(a < b_ for a, b_ in zip(keep, keep[1:]))
            queued[t + 1, j] = len(q)
        dropped[j] = lost
    return queued, batch, dropped


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("policy", [P, TR])
def test_brute_force_fifo(orc, seed, policy):
    rng = np.random.default_rng(seed)
    K = int(rng.integers(1, 6))
    rates = [int(x) for x in rng.integers(0, 300, K)]
    iter_us = [int(x) for x in rng.integers(1, 3_000_000, K)]
    b_min, b_max = sorted(int(x) for x in rng.integers(0, 400, 2))
    T = int(rng.integers(0, 40))
    want = brute_force(rates, iter_us, b_min, b_max, policy, T)
    got = orc.stream_run(rates, iter_us, b_min, b_max, policy, T)
    for w, g in zip(want, got):
        assert np.array_equal(w, g)


@pytest.mark.parametrize("S,t_us,b", [(100, 1_200_000, 100), (600, 1_600_000, 600), (250, 2_000_000, 64),
                                      (37, 1_000_000, 37), (1000, 3_500_000, 800)])
def test_eqn2_closed_form(orc, S, t_us, b):
    # Eqn 2: Q = (t S - b) T + S whenever t S >= b, here with t S a whole number
    T = 500
    q, used, _ = orc.stream_run([S], [t_us], b, b, P, T)
    tS = S * t_us // 1_000_000
    assert tS * 1_000_000 == S * t_us and tS >= b
    for step in range(T + 1):
        assert int(q[step, 0]) == (tS - b) * step + S
    assert np.all(used == b)
    # the text's first iteration: (S - b) + t S samples at ts = 1
    assert int(q[1, 0]) == (S - b) + tS
    # Eqn 2 at ts = 2 (the text's own sum for ts = 2 has an extra S; Eqn 2 is followed)
    assert int(q[2, 0]) == 2 * tS - 2 * b + S


def test_eqn2_fractional_arrivals(orc):
    # a continuous stream whose arrivals per iteration are not whole: the
    # buffer is S + floor(S t T) - b T exactly, never drifting from Eqn 2 by a sample
    S, t_us, b, T = 333, 1_234_567, 300, 2000
    q, _, _ = orc.stream_run([S], [t_us], b, b, P, T)
    for step in (0, 1, 7, 999, 2000):
        assert int(q[step, 0]) == S + arrivals_until(S, t_us, step) - b * step
        exact = (S * t_us / 1e6 - b) * step + S
        assert abs(int(q[step, 0]) - exact) < 1.0


def test_eqn3_reproduces_table_ii(orc):
    # Eqn 3 (b negligible beside t S): Q = T t S + S; with b = 0 the
    # simulation is exactly that, and at the sample size of Section V-F it
    # gives Table II in GiB
    g = json.load(open(GOLDEN))["table_ii_data_accumulated_GiB"]
    for e in g["entries"]:
        t_us = int(round(e["t_s"] * 1e6))
        q, _, _ = orc.stream_run([e["S"]], [t_us], 0, 0, P, e["T"])
        Q = int(q[-1, 0])
        assert Q == e["T"] * e["S"] * t_us // 1_000_000 + e["S"]
        gib = Q * g["bytes_per_sample"] / 2**30
        assert abs(gib - e["GiB"]) <= 2e-3 * e["GiB"], e


def test_linear_growth_and_truncation_bound(orc):
    rates = [100, 600, 130, 635]
    iter_us = [1_200_000, 1_600_000, 1_200_000, 1_600_000]
    T = 1000
    qp, bp, _ = orc.stream_run(rates, iter_us, 8, 1024, P, T)
    qt, bt, dt = orc.stream_run(rates, iter_us, 8, 1024, TR, T)
    for j, (S, t_us) in enumerate(zip(rates, iter_us)):
        d = np.diff(qp[:, j].astype(np.int64))
        assert np.all(d == d[0]) and d[0] == S * t_us // 1_000_000 - S   # slope t S - b with b = S
        # truncation: the buffer never exceeds S, and with t >= 1 s it is exactly S
        assert np.all(qt[:, j] == S)
        assert np.all(bt[:, j] == S)
    # persistence grows as O(S T); truncation stays O(S)
    assert np.all(qp[-1] > 100 * qt[-1])


def test_conservation(orc):
    rng = np.random.default_rng(3)
    K, T = 8, 300
    rates = [int(x) for x in rng.integers(1, 2000, K)]
    iter_us = [int(x) for x in rng.integers(10_000, 4_000_000, K)]
    for policy in (P, TR):
        q, b, d = orc.stream_run(rates, iter_us, 8, 1024, policy, T)
        for j in range(K):
            arrived = rates[j] + arrivals_until(rates[j], iter_us[j], T)
            assert arrived == int(b[:, j].sum()) + int(q[-1, j]) + int(d[j])
            if policy == P:
                assert int(d[j]) == 0


def test_batch_rule_and_starvation(orc):
    # b = S bounded to [b_min, b_max] (§IV; bounds 8 and 1024 of Section V-D)
    bounds = json.load(open(GOLDEN))["batch_bounds"]
    lo, hi = bounds["b_min"], bounds["b_max"]
    q, b, _ = orc.stream_run([4000, 2, 500], [1_000_000] * 3, lo, hi, P, 5)
    assert b[:, 0].tolist() == [hi] * 5
    assert b[:, 2].tolist() == [500] * 5
    # a stream slower than b_min: the device trains on what it holds
    assert b[:, 1].tolist() == [2] * 5
    assert q[:, 1].tolist() == [2] * 6
    # t S < b drains the buffer, then trains on each iteration's arrivals
    q, b, _ = orc.stream_run([100], [500_000], 100, 100, P, 4)
    assert b[:, 0].tolist() == [100, 50, 50, 50]
    assert q[:, 0].tolist() == [100, 50, 50, 50, 50]


def test_rejects_bad_input(orc):
    with pytest.raises(ValueError):
        orc.stream_run([10], [10], 5, 4, P, 3)          # b_min > b_max
    with pytest.raises(ValueError):
        orc.stream_run([10], [10], 0, 4, 2, 3)          # no such policy
    with pytest.raises(ValueError):
        orc.stream_run([2**32], [10], 0, 4, P, 3)       # rate too large
