"""Pins of the oracle's per-layer Top-k (the per-layer reading of the Top-k of
§IV: every layer keeps its own top fraction of its entries).

The per-layer kept set has one correct answer: within every layer, the unique
k_l-subset whose entries dominate the layer's dropped entries (larger
magnitude, or equal magnitude and lower index), with k_l = clamp(floor(ratio *
n_l), 1, n_l). These tests check the oracle against that definition by brute
force and against a stable library sort of each layer, and against invariants
that a lost layer offset, a global instead of per-layer selection, a per-layer
k taken from the whole vector, or a dropped energy term would break.
"""
import itertools
import math

import numpy as np
import pytest

TIE_VALUES = np.array([0.0, -0.0, 0.5, -0.5, 1.0, -1.0, 2.0, -2.0], dtype=np.float32)


def random_layers(rng, n, L):
    cuts = np.sort(rng.choice(np.arange(1, n), size=L - 1, replace=False)) if L > 1 else np.array([], int)
    return np.concatenate([[0], cuts, [n]]).astype(np.uint64)


def dominant_subset(g, k):
    """The subset of the definition, by enumeration (tiny layers only)."""
    n = g.size
    mag = np.abs(g)
    found = []
    for S in itertools.combinations(range(n), k):
        s = set(S)
        if all(mag[i] > mag[j] or (mag[i] == mag[j] and i < j) for i in S for j in range(n) if j not in s):
            found.append(S)
    assert len(found) == 1
    return found[0]


def test_worked_example(orc):
    # g = -5..4 in two layers of 4 and 6 entries at ratio 0.3: each keeps
    # floor(0.3 * n_l) = 1 entry, -5 (index 0) and 4 (index 9); the whole
    # gradient's energies are 85 and 25 + 16 = 41.
    g = (np.arange(10) - 5).astype(np.float32)
    idx, val, e_all, e_kept = orc.topk_layers(g, [0, 4, 10], 0.3)
    assert idx.tolist() == [0, 9]
    assert val.tolist() == [-5.0, 4.0]
    assert (e_all, e_kept) == (85.0, 41.0)
    # the whole-vector Top-k at the same k would keep -5 and -4 instead
    gidx, _, _, _ = orc.topk(g, 2)
    assert gidx.tolist() == [0, 1]


@pytest.mark.parametrize("seed", range(10))
def test_bruteforce_per_layer(orc, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 12))
    L = int(rng.integers(1, min(n, 4) + 1))
    off = random_layers(rng, n, L)
    g = rng.choice(TIE_VALUES, size=n)
    for ratio in (0.05, 0.3, 0.5, 0.8, 1.0):
        want = []
        for l in range(L):
            a, b = int(off[l]), int(off[l + 1])
            k_l = max(1, min(b - a, math.floor(ratio * (b - a))))
            want += [a + i for i in dominant_subset(g[a:b], k_l)]
        idx, val, _, _ = orc.topk_layers(g, off, ratio)
        assert idx.tolist() == want
        assert np.array_equal(val.view(np.uint32), g[idx].view(np.uint32))


@pytest.mark.parametrize("n,L,seed", [(1000, 3, 0), (5000, 17, 1), (20000, 38, 2)])
def test_matches_stable_argsort_per_layer(orc, n, L, seed):
    rng = np.random.default_rng(seed)
    off = random_layers(rng, n, L)
    g = (rng.integers(-6, 7, size=n) * 0.125).astype(np.float32)
    g[rng.random(n) < 0.05] = -0.0
    for ratio in (0.001, 0.01, 0.1, 1.0):
        parts = []
        for l in range(L):
            a, b = int(off[l]), int(off[l + 1])
            k_l = max(1, min(b - a, math.floor(ratio * (b - a))))
            parts.append(np.sort(np.argsort(-np.abs(g[a:b]), kind="stable")[:k_l]) + a)
        ref = np.concatenate(parts).astype(np.uint32)
        idx, _, _, _ = orc.topk_layers(g, off, ratio)
        assert np.array_equal(idx, ref)
        tidx, tval, _, _ = orc.topk_layers_by_threshold(g, off, ratio)
        assert np.array_equal(tidx, ref)
        assert np.array_equal(tval.view(np.uint32), g[ref].view(np.uint32))


def test_one_layer_is_the_whole_vector_topk(orc):
    rng = np.random.default_rng(5)
    g = rng.standard_normal(3000).astype(np.float32)
    for ratio in (0.001, 0.01, 0.3):
        k = orc.topk_k(g.size, ratio)
        a = orc.topk(g, k)
        b = orc.topk_layers(g, [0, g.size], ratio)
        assert np.array_equal(a[0], b[0])
        assert np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32))
        assert a[2] == b[2] and a[3] == b[3]


def test_every_layer_keeps_its_own_share(orc):
    # one layer a thousand times larger than the rest: a whole-vector Top-k
    # would take everything from it; the per-layer one takes k_l from each
    rng = np.random.default_rng(7)
    sizes = [64, 1000, 37, 4000, 1]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    g = rng.standard_normal(int(off[-1])).astype(np.float32)
    g[off[3]:off[4]] *= 1000.0
    ratio = 0.01
    idx, _, _, _ = orc.topk_layers(g, off, ratio)
    assert orc.layers_k(off, ratio) == 1 + 10 + 1 + 40 + 1
    for l, n_l in enumerate(sizes):
        inside = (idx >= off[l]) & (idx < off[l + 1])
        assert int(np.count_nonzero(inside)) == max(1, math.floor(ratio * n_l))
    assert np.all(np.diff(idx.astype(np.int64)) > 0)


def test_ratio_one_keeps_everything(orc):
    rng = np.random.default_rng(8)
    g = rng.standard_normal(777).astype(np.float32)
    idx, val, e_all, e_kept = orc.topk_layers(g, [0, 100, 101, 500, 777], 1.0)
    assert np.array_equal(idx, np.arange(777, dtype=np.uint32))
    assert np.array_equal(val.view(np.uint32), g.view(np.uint32))
    assert e_all == e_kept


def test_energies_of_the_whole_gradient(orc):
    rng = np.random.default_rng(9)
    n = 50000
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-8, 2, n))).astype(np.float32)
    off = random_layers(rng, n, 20)
    idx, _, e_all, e_kept = orc.topk_layers(g, off, 0.02)
    x = g.astype(np.float64)
    exact_all = math.fsum(x * x)
    exact_kept = math.fsum(x[idx] * x[idx])
    tol = n * 2.0**-53
    assert abs(e_all - exact_all) <= tol * exact_all
    assert abs(e_kept - exact_kept) <= tol * exact_kept
    assert 0.0 < e_kept < e_all


@pytest.mark.parametrize("off", [[1, 5], [0, 3, 3, 5], [0, 4], [0, 6], [0]])
def test_rejects_bad_layers(orc, off):
    g = np.ones(5, dtype=np.float32)
    with pytest.raises(ValueError):
        orc.topk_layers(g, off, 0.5)


def test_rejects_bad_ratio(orc):
    g = np.ones(5, dtype=np.float32)
    for ratio in (0.0, -0.1, 1.5, float("nan")):
        with pytest.raises(ValueError):
            orc.topk_layers(g, [0, 2, 5], ratio)
