"""Pins of the oracle's k rule, weights (Eqn 4a), aggregation (Eqn 4b) and SGD
(Eqn 4c) against values the paper prints, exact arithmetic and textbook
special cases."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


# ---- k rule (§V-G compression ratio) ---------------------------------------------------

CONFIG_K = [  # (n, ratio, k) for the five workloads
    (1_048_576, 0.01, 10_485), (11_173_962, 0.01, 111_739), (25_557_032, 0.1, 2_555_703),
    (25_557_032, 0.01, 255_570), (25_557_032, 0.001, 25_557), (60_192_808, 0.001, 60_192),
    (143_667_240, 0.01, 1_436_672)]


@pytest.mark.parametrize("n,ratio,k", CONFIG_K)
def test_k_for_workloads(orc, n, ratio, k):
    assert orc.topk_k(n, ratio) == k


def test_k_rule_edges(orc):
    assert orc.topk_k(1000, 1e-9) == 1           # ratio * n < 1 still keeps one entry
    assert orc.topk_k(1000, 1.0) == 1000
    assert orc.topk_k(1, 0.5) == 1
    assert orc.topk_k(0, 0.5) == 0
    assert orc.topk_k(10, 0.0) == 0
    assert orc.topk_k(10, 1.5) == 0
    assert orc.topk_k(10, float("nan")) == 0
    assert orc.topk_k(2**32, 0.5) == 0
    below = math.nextafter(0.07, 0.0)
    assert orc.topk_k(100, 0.07) == math.floor(0.07 * 100)
    assert orc.topk_k(100, below) == math.floor(below * 100)


def test_update_sizes_printed_in_paper(orc):
    """§V-G: at CR 0.1 the fp32 update of ResNet152 (230 MB) shrinks to 23 MB and that of
    VGG19 (548 MB) to 55 MB. The workload sizes and the k rule reproduce both."""
    g = golden()
    mib = 2**20
    for name, n in (("ResNet152", 60_192_808), ("VGG19", 143_667_240)):
        assert abs(n - g["model_parameters"][name]) / g["model_parameters"][name] < 1e-3
        full = g["update_size_MB"][name]["full"]
        comp = g["update_size_MB"][name]["cr_0.1"]
        k = orc.topk_k(n, g["compression_ratio_definition"]["cr"])
        assert round(n * 4 / mib) == full
        assert round(k * 4 / mib) == comp
        assert k / n == pytest.approx(g["compression_ratio_definition"]["fraction_kept"], rel=1e-6)


# ---- weights and learning-rate scale (Eqn 4a, linear scaling rule) -----------------------

def test_weights_eqn4a(orc):
    rates = [38.0, 300.0, 64.0, 256.0, 0.0, 17.5]
    w, gamma = orc.stream_weights(rates, base_batch=64 * 6)
    exact = [Fraction(r) / Fraction(sum(rates)) for r in rates]
    for wj, ej in zip(w, exact):
        assert wj == np.float32(float(ej))                 # r_j = S_j / sum S, rounded once
    assert abs(math.fsum(float(x) for x in w) - 1.0) <= len(rates) * 2**-24
    assert gamma == pytest.approx(sum(rates) / (64 * 6), rel=1e-15)
    assert w[4] == 0.0


def test_weights_batch_bounds(orc):
    g = golden()["batch_bounds"]
    rates = [2.0, 8.0, 500.0, 4000.0]
    w, gamma = orc.stream_weights(rates, b_min=g["b_min"], b_max=g["b_max"], base_batch=64)
    b = [8.0, 8.0, 500.0, 1024.0]
    assert list(w) == [np.float32(x / sum(b)) for x in b]
    assert gamma == pytest.approx(sum(b) / 64)
    with pytest.raises(ValueError):
        orc.stream_weights([0.0, 0.0])
    with pytest.raises(ValueError):
        orc.stream_weights([1.0, -1.0])
    with pytest.raises(ValueError):
        orc.stream_weights([1.0, float("inf")])


def test_equal_rates_reduce_to_plain_average(orc):
    """Equal streaming rates give r_j = 1/N, the weights of conventional DDL (Eqn 1)."""
    w, _ = orc.stream_weights([64.0] * 16)
    assert np.all(w == np.float32(1 / 16))


# ---- aggregation (Eqn 4b) ----------------------------------------------------------------

def test_dense_equal_weights_is_the_mean(orc):
    """ratio 1 with equal weights: the aggregate is the plain mean of Eqn 1."""
    rng = np.random.default_rng(3)
    K, n = 8, 5000
    G = (rng.standard_normal((K, n)) * 0.01).astype(np.float32)
    w = np.full(K, 1 / K, dtype=np.float32)
    out = orc.aggregate([(None, G[j]) for j in range(K)], w, n)
    mean = G.astype(np.float64).mean(axis=0)
    ulp = np.spacing(np.abs(mean).astype(np.float32))
    assert np.all(np.abs(out.astype(np.float64) - mean) <= ulp)


def test_single_device_is_its_scatter(orc):
    rng = np.random.default_rng(4)
    n = 1000
    g = rng.standard_normal(n).astype(np.float32)
    idx, val, _, _ = orc.topk(g, 37)
    out = orc.aggregate([(idx, val)], np.array([1.0], dtype=np.float32), n)
    ref = np.zeros(n, dtype=np.float32)
    ref[idx] = val
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))   # +0 off the set


def test_identical_devices_equal_weights(orc):
    rng = np.random.default_rng(5)
    n, K = 2048, 4
    g = rng.standard_normal(n).astype(np.float32)
    idx, val, _, _ = orc.topk(g, 100)
    out = orc.aggregate([(idx, val)] * K, np.full(K, 0.25, dtype=np.float32), n)
    ref = np.zeros(n, dtype=np.float32)
    ref[idx] = val
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


def test_zero_weight_device_is_removed(orc):
    rng = np.random.default_rng(6)
    n = 3000
    sets, ws = [], [0.5, 0.0, 0.5]
    for j in range(3):
        g = rng.standard_normal(n).astype(np.float32)
        i, v, _, _ = orc.topk(g, 200)
        sets.append((i, v))
    a = orc.aggregate(sets, np.array(ws, dtype=np.float32), n)
    b = orc.aggregate([sets[0], sets[2]], np.array([0.5, 0.5], dtype=np.float32), n)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_dense_device_equals_full_sparse_set(orc):
    rng = np.random.default_rng(8)
    n = 777
    g = rng.standard_normal(n).astype(np.float32)
    h = rng.standard_normal(n).astype(np.float32)
    i, v, _, _ = orc.topk(h, 50)
    w = np.array([0.3, 0.7], dtype=np.float32)
    a = orc.aggregate([(None, g), (i, v)], w, n)
    b = orc.aggregate([(np.arange(n, dtype=np.uint32), g), (i, v)], w, n)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_aggregate_against_exact_rationals(orc):
    """Each output is within one float ulp of the exactly computed weighted sum."""
    rng = np.random.default_rng(9)
    n, K = 64, 5
    sets, w = [], rng.dirichlet(np.ones(K)).astype(np.float32)
    for j in range(K):
        g = (rng.standard_normal(n) * 10.0 ** rng.integers(-6, 0)).astype(np.float32)
        sets.append(orc.topk(g, 20)[:2])
    out = orc.aggregate(sets, w, n)
    for i in range(n):
        exact = Fraction(0)
        for j, (idx, val) in enumerate(sets):
            hit = np.flatnonzero(idx == i)
            if hit.size:
                exact += Fraction(float(w[j])) * Fraction(float(val[hit[0]]))
        assert abs(Fraction(float(out[i])) - exact) <= Fraction(float(np.spacing(np.float32(abs(float(exact))))))
        if exact == 0:
            assert out[i] == 0 and not np.signbit(out[i])


def test_aggregate_at_matches_aggregate(orc):
    rng = np.random.default_rng(10)
    n, K = 500, 3
    sets, contrib = [], np.zeros((K, n), dtype=np.float32)
    for j in range(K):
        g = rng.standard_normal(n).astype(np.float32)
        i, v, _, _ = orc.topk(g, 60)
        sets.append((i, v))
        contrib[j, i] = v
    w = np.array([0.2, 0.3, 0.5], dtype=np.float32)
    assert np.array_equal(orc.aggregate(sets, w, n).view(np.uint32),
                          orc.aggregate_at(contrib, w).view(np.uint32))


# ---- SGD (Eqn 4c) --------------------------------------------------------------------------

def test_sgd(orc):
    rng = np.random.default_rng(11)
    p = rng.standard_normal(300).astype(np.float32)
    g = rng.standard_normal(300).astype(np.float32)
    assert np.array_equal(orc.sgd(p, g, 0.0).view(np.uint32), p.view(np.uint32))
    assert np.array_equal(orc.sgd(p, np.zeros_like(g), 0.5).view(np.uint32), p.view(np.uint32))
    lr = np.float32(0.0125)
    q = orc.sgd(p, g, float(lr))
    for i in range(50):
        exact = Fraction(float(p[i])) - Fraction(float(lr)) * Fraction(float(g[i]))
        assert abs(Fraction(float(q[i])) - exact) <= Fraction(float(np.spacing(np.float32(abs(float(exact))))))
    assert np.all(q[g > 0] < p[g > 0]) and np.all(q[g < 0] > p[g < 0])


def test_extended_energies_against_exact_sums(orc):
    """The long-double energy references used to bound the kernels' double sums:
    within (m - 1) 2^-64 of the exact rational sum of the squares, including
    denormals and signed zeros, and far inside any double summation's bound."""
    from fractions import Fraction
    rng = np.random.default_rng(21)
    for n in (1, 2, 7, 300, 4097):
        g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-6, 1, n)).astype(np.float32)
        if n > 4:
            g[:3] = np.array([np.float32(1e-40), -0.0, np.float32(-3e-39)], dtype=np.float32)
        idx = np.sort(rng.choice(n, size=max(1, n // 5), replace=False)).astype(np.uint32)
        ea, ek = orc.energies_extended(g, idx)
        exact_a = sum(Fraction(float(x)) ** 2 for x in g)
        exact_k = sum(Fraction(float(g[i])) ** 2 for i in idx)
        for got, exact, m in ((ea, exact_a, n), (ek, exact_k, idx.size)):
            err = abs(Fraction(float(got)) - exact) if exact else abs(Fraction(float(got)))
            # the long double result is rounded once more to double for the comparison
            assert err <= (max(m - 1, 0) * 2.0**-64 + 2.0**-53) * float(exact) + 0.0, (n, m)
        # against a correctly rounded double sum
        sq = np.square(g.astype(np.float64))
        assert abs(float(ea) - math.fsum(sq)) <= (n * 2.0**-64 + 2.0**-52) * math.fsum(sq)


def test_extended_energies_catch_a_dropped_term(orc):
    """A reference that dropped one kept square would fail the bound of the
    comparisons at once (the bound is ~m 2^-53 relative, a term is far larger)."""
    rng = np.random.default_rng(22)
    g = rng.standard_normal(100_000).astype(np.float32)
    k = orc.topk_k(g.size, 0.01)
    idx, _, ea, ek = orc.topk(g, k)
    ra, rk = orc.energies_extended(g, idx)
    bound = 2 * k * 2.0**-53 * float(rk)
    assert abs(ek - float(rk)) <= bound
    _, rk_short = orc.energies_extended(g, idx[1:])
    assert abs(ek - float(rk_short)) > bound
