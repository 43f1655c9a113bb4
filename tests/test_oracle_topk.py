"""Pins of the oracle's Top-k (§III-C, §IV "High communication cost").

Top-k with ties to the lower index has one correct answer: the unique k-subset
S such that every kept entry dominates every dropped one, i.e. for i in S and
j not in S, |g_i| > |g_j| or (|g_i| == |g_j| and i < j). These tests check the
oracle against that definition by brute force, against a textbook stable sort,
and against invariants and special cases that a dropped term, a flipped
comparison or a wrong tie-break would break.
"""
import itertools
import math

import numpy as np
import pytest

pytestmark = pytest.mark.filterwarnings("ignore")

TIE_VALUES = np.array([0.0, -0.0, 0.5, -0.5, 1.0, -1.0, 2.0, -2.0], dtype=np.float32)


def dominant_subsets(g, k):
    n = g.size
    mag = np.abs(g)
    out = []
    for S in itertools.combinations(range(n), k):
        s = set(S)
        ok = all(mag[i] > mag[j] or (mag[i] == mag[j] and i < j)
                 for i in S for j in range(n) if j not in s)
        if ok:
            out.append(S)
    return out


@pytest.mark.parametrize("seed", range(12))
def test_bruteforce_unique_subset(orc, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 10))
    g = rng.choice(TIE_VALUES, size=n)
    for k in range(1, n + 1):
        subsets = dominant_subsets(g, k)
        assert len(subsets) == 1, "the definition must single out one subset"
        idx, val, _, _ = orc.topk(g, k)
        assert tuple(int(i) for i in idx) == subsets[0]
        assert np.array_equal(val.view(np.uint32), g[idx].view(np.uint32))
        tidx, _, _, _ = orc.topk_by_threshold(g, k)
        assert tuple(int(i) for i in tidx) == subsets[0]


@pytest.mark.parametrize("n,levels,seed", [(1000, 7, 0), (4097, 3, 1), (20000, 50, 2),
                                           (65536, 1000, 3)])
def test_matches_stable_argsort(orc, n, levels, seed):
    rng = np.random.default_rng(seed)
    g = (rng.integers(-levels, levels + 1, size=n) * 0.25).astype(np.float32)
    g[rng.random(n) < 0.1] = -0.0
    for ratio in (0.001, 0.01, 0.1, 0.5, 1.0):
        k = orc.topk_k(n, ratio)
        ref = np.sort(np.argsort(-np.abs(g), kind="stable")[:k]).astype(np.uint32)
        idx, val, _, _ = orc.topk(g, k)
        assert np.array_equal(idx, ref)
        tidx, _, _, _ = orc.topk_by_threshold(g, k)
        assert np.array_equal(tidx, ref)


def check_invariants(g, k, idx, val):
    n = g.size
    assert idx.size == k
    assert np.all(np.diff(idx.astype(np.int64)) > 0)
    assert int(idx[-1]) < n
    assert np.array_equal(val.view(np.uint32), g[idx].view(np.uint32))
    mag = np.abs(g)
    kept = np.zeros(n, dtype=bool)
    kept[idx] = True
    if k < n:
        t = mag[kept].min()
        assert mag[~kept].max() <= t
        tie_kept = np.flatnonzero(kept & (mag == t))
        tie_drop = np.flatnonzero(~kept & (mag == t))
        if tie_drop.size:
            assert tie_kept.max() < tie_drop.min()


@pytest.mark.parametrize("ratio", [0.001, 0.01, 0.1])
def test_invariants_on_c1_shape(orc, wl, ratio):
    s = wl.spec(1, n=1 << 16)
    g = wl.gradient(s, 0, 1)
    k = orc.topk_k(s.n, ratio)
    idx, val, e_all, e_kept = orc.topk(g, k)
    check_invariants(g, k, idx, val)


def test_invariants_with_ties_and_zeros(orc, wl):
    s = wl.spec(4, n=200_000, K=2)
    k = orc.topk_k(s.n, s.ratios[0, 1])
    g = wl.gradient(s, 0, 1, k=k)
    idx, val, _, _ = orc.topk(g, k)
    check_invariants(g, k, idx, val)
    mag = np.abs(g)
    t = mag[idx].min()
    assert np.count_nonzero(mag == t) > k // 4, "the workload must put many ties on the boundary"


def test_special_cases(orc):
    rng = np.random.default_rng(7)
    g = rng.standard_normal(333).astype(np.float32)
    idx, _, _, _ = orc.topk(g, g.size)                     # ratio 1 keeps everything
    assert np.array_equal(idx, np.arange(g.size, dtype=np.uint32))
    eq = np.full(100, -3.5, dtype=np.float32)
    eq[::2] = 3.5
    idx, _, _, _ = orc.topk(eq, 17)                        # equal magnitudes: lowest indices
    assert np.array_equal(idx, np.arange(17, dtype=np.uint32))
    z = np.zeros(50, dtype=np.float32)
    z[1::3] = -0.0
    idx, _, _, _ = orc.topk(z, 5)                          # -0 ranks equal to +0
    assert np.array_equal(idx, np.arange(5, dtype=np.uint32))
    h = np.array([1.0, -4.0, 2.0, 4.0, -4.0], dtype=np.float32)
    idx, _, _, _ = orc.topk(h, 1)                          # k = 1: lowest argmax of |g|
    assert list(idx) == [1]
    idx, val, e_all, e_kept = orc.topk(np.array([-2.5], dtype=np.float32), 1)
    assert list(idx) == [0] and val[0] == np.float32(-2.5) and e_all == e_kept == 6.25
    d = np.array([1, 0x80000003, 2, 0], dtype=np.uint32).view(np.float32)  # denormals, no flushing
    idx, _, _, _ = orc.topk(d, 2)
    assert list(idx) == [1, 2]


def test_energies(orc, wl):
    s = wl.spec(3, n=50_000, K=1)
    g = wl.gradient(s, 0, 0)
    for ratio in (0.001, 0.01, 0.1, 1.0):
        k = orc.topk_k(s.n, ratio)
        idx, _, e_all, e_kept = orc.topk(g, k)
        exact_all = math.fsum(float(x) * float(x) for x in g.astype(np.float64))
        exact_kept = math.fsum(float(x) * float(x) for x in g[idx].astype(np.float64))
        assert e_all == pytest.approx(exact_all, rel=1e-12)
        assert e_kept == pytest.approx(exact_kept, rel=1e-12)
        send, rho = orc.compress_decision(e_all, e_kept, 0.3)
        # the kept entries are the largest, so their mean square is at least the mean square
        assert 0.0 <= rho <= 1.0 - k / s.n + 1e-12
        if ratio == 1.0:
            assert rho == 0.0 and send
    assert orc.compress_decision(0.0, 0.0, 0.0) == (True, 0.0)    # zero gradient loses nothing
    assert orc.compress_decision(4.0, 3.0, 0.25) == (True, 0.25)  # boundary is inclusive
    assert orc.compress_decision(4.0, 3.0, 0.2499) == (False, 0.25)


def test_energies_helper(orc, wl):
    s = wl.spec(2, n=40_000, K=1)
    g = wl.gradient(s, 0, 0)
    idx, _, e_all, e_kept = orc.topk(g, 400)
    a, b = orc.energies(g, idx)
    assert a == pytest.approx(math.fsum(float(x) ** 2 for x in g), rel=1e-13)
    assert b == pytest.approx(math.fsum(float(x) ** 2 for x in g[idx]), rel=1e-13)
    assert a == pytest.approx(e_all, rel=1e-13) and b == pytest.approx(e_kept, rel=1e-13)


def test_pins_catch_a_wrong_tie_break(orc):
    """A planted mistake (ties to the higher index) fails the brute-force pin."""
    g = np.array([1.0, -1.0, 1.0, 0.5], dtype=np.float32)

    def wrong(g, k):
        order = sorted(range(g.size), key=lambda i: (-abs(float(g[i])), -i))
        return tuple(sorted(order[:k]))

    assert wrong(g, 2) != dominant_subsets(g, 2)[0]
    assert tuple(int(i) for i in orc.topk(g, 2)[0]) == dominant_subsets(g, 2)[0]
