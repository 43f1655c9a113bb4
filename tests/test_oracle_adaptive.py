"""Pins of the oracle's adaptive compression with a moving average of the
energies (§IV) and its accounting (CNC ratio and floats sent, §V-G): the
instantaneous rule as the special case without smoothing, the closed form of
the moving average, brute-force counting, and the floats Table V prints."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def _run(orc, energies, beta, delta, k, n, counters=None):
    state = np.zeros(2)
    sends = [orc.adaptive_step(state, counters, ea, ek, beta, delta, k, n) for ea, ek in energies]
    return sends, state


def test_without_smoothing_is_the_instantaneous_rule(orc):
    rng = np.random.default_rng(4)
    ea = rng.uniform(0.5, 2.0, 200)
    ek = ea * rng.uniform(0.5, 1.0, 200)
    sends, _ = _run(orc, list(zip(ea, ek)), 0.0, 0.2, 10, 1000)
    assert sends == [orc.compress_decision(a, b, 0.2)[0] for a, b in zip(ea, ek)]
    assert any(sends) and not all(sends)


def test_first_iteration_takes_its_energies(orc):
    state = np.zeros(2)
    send = orc.adaptive_step(state, None, 4.0, 3.0, 0.9, 0.3, 1, 10)
    assert state.tolist() == [4.0, 3.0]
    assert send == orc.compress_decision(4.0, 3.0, 0.3)[0]


@pytest.mark.parametrize("beta", [0.5, 0.9, 0.99])
def test_step_response_closed_form(orc, beta):
    # energies a for t0 iterations, then b: the average tends to b as
    # b + (a - b) * beta^m after m iterations at b (weights on the history)
    a, b, t0, m = (8.0, 2.0), (4.0, 3.5), 5, 40
    energies = [a] * t0 + [b] * m
    state = np.zeros(2)
    for t, (ea, ek) in enumerate(energies):
        orc.adaptive_step(state, None, ea, ek, beta, 0.5, 1, 10)
        if t >= t0:
            mm = t - t0 + 1
            for i in range(2):
                closed = b[i] + (a[i] - b[i]) * beta ** mm
                assert abs(state[i] - closed) <= 64 * np.spacing(abs(closed)), (t, i)


def test_smoothing_delays_the_switch(orc):
    # the uncompressed-loss ratio drops from 0.5 to 0.05 at t = 10; with delta
    # 0.1 the instantaneous rule switches to Top-k at once, the average later
    energies = [(1.0, 0.5)] * 10 + [(1.0, 0.95)] * 30
    inst, _ = _run(orc, energies, 0.0, 0.1, 1, 10)
    slow, _ = _run(orc, energies, 0.9, 0.1, 1, 10)
    assert inst.index(True) == 10
    first = slow.index(True)
    # 0.45 * 0.9^m + 0.05 <= 0.1  =>  m >= log(1/9)/log(0.9) = 20.85
    assert first == 10 + 21 - 1
    assert all(slow[first:])


def test_counters_by_brute_force(orc):
    rng = np.random.default_rng(5)
    k, n = 37, 1000
    energies = [(1.0, float(x)) for x in rng.uniform(0.6, 1.0, 500)]
    counters = np.zeros(3, dtype=np.uint64)
    sends, _ = _run(orc, energies, 0.0, 0.2, k, n, counters)
    tc = sum(sends)
    assert counters.tolist() == [tc, len(sends), sum(k if s else n for s in sends)]
    assert orc.cnc_ratio(counters) == tc / len(sends)


def test_cnc_extremes(orc):
    g = json.load(open(GOLDEN))["cnc_ratio_extremes"]
    never, always = np.zeros(3, dtype=np.uint64), np.zeros(3, dtype=np.uint64)
    _run(orc, [(1.0, 0.1)] * 20, 0.5, 0.2, 1, 10, never)       # loss 0.9 > delta: always dense
    _run(orc, [(1.0, 1.0)] * 20, 0.5, 0.2, 1, 10, always)      # no loss: always Top-k
    assert orc.cnc_ratio(never) == g["never"] and orc.cnc_ratio(always) == g["always"]
    assert never[2] == 20 * 10 and always[2] == 20 * 1


def test_floats_sent_against_table_v(orc):
    # a run of T iterations with the printed CNC and CR, counted by the oracle,
    # scaled to the uncompressed total of its model, gives the printed floats
    t = json.load(open(GOLDEN))["table_v_floats_sent"]
    T, n = 1000, 10_000
    for row in t["fit_identity"]:
        k = int(round(row["cr"] * n))
        tc = int(round(row["cnc"] * T))
        counters = np.zeros(3, dtype=np.uint64)
        energies = [(1.0, 1.0)] * tc + [(1.0, 0.0)] * (T - tc)   # loss 0 -> Top-k, loss 1 -> dense
        _run(orc, energies, 0.0, 0.5, k, n, counters)
        assert abs(orc.cnc_ratio(counters) - row["cnc"]) < 1e-12
        predicted = t["uncompressed"][row["model"]] * float(counters[2]) / (T * n)
        assert abs(predicted - row["floats"]) <= 0.02 * row["floats"], row
