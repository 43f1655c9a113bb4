"""The seeded workload generator: published known answers, determinism and the
shape of the synthetic gradients."""
import numpy as np
import pytest


def test_philox_known_answers(wl):
    """Known-answer vectors of Philox4x32-10 published with the Random123 library
    (Salmon et al., SC'11)."""
    assert wl.philox4x32_10((0, 0, 0, 0), (0, 0)) == (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)
    assert wl.philox4x32_10((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2) == (
        0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)
    assert wl.philox4x32_10((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344),
                            (0xA4093822, 0x299F31D0)) == (0xD16CFE09, 0x94FDCCEB, 0x5001E420,
                                                          0x24126EA1)


def test_deterministic_across_threads(wl):
    s = wl.spec(2, n=300_001, K=2)
    a = wl.gradient(s, 0, 1, nthreads=1)
    b = wl.gradient(s, 0, 1, nthreads=7)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c = wl.gradient(s, 0, 0, nthreads=3)
    assert not np.array_equal(a, c)


@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
def test_full_shapes(wl, config):
    s = wl.spec(config)
    assert (s.K, s.n) == (wl.FULL[config]["K"], wl.FULL[config]["n"])
    assert int(s.seg_end[-1]) == s.n
    assert np.all(np.diff(np.concatenate([[0], s.seg_end.astype(np.int64)])) >= 1)
    assert s.rates.shape == (s.iterations, s.K)
    assert np.all(s.rates >= 0) and np.all(s.rates.sum(axis=1) > 0)
    if config == 5:
        sizes = np.diff(np.concatenate([[0], s.seg_end.astype(np.int64)]))
        assert sizes[-3:].sum() == int(np.floor(0.85 * s.n))
        assert s.iterations == 10
    if config == 3:
        assert list(s.ratios[:, 0]) == [0.1, 0.01, 0.001]


def test_segment_scales(wl):
    s = wl.spec(1, n=1 << 20)
    g = wl.gradient(s, 0, 2)
    start = 0
    for end, sig in zip(s.seg_end.astype(np.int64), s.seg_sigma):
        seg = g[start:end].astype(np.float64)
        assert seg.std() == pytest.approx(sig, rel=0.02)
        start = end
    s3 = wl.spec(3, n=400_000, K=1)
    g3 = wl.gradient(s3, 0, 0).astype(np.float64)
    sizes = np.diff(np.concatenate([[0], s3.seg_end.astype(np.int64)]))
    big = int(np.argmax(sizes))
    lo = 0 if big == 0 else int(s3.seg_end[big - 1])
    seg = g3[lo:int(s3.seg_end[big])]
    kurt = ((seg - seg.mean()) ** 4).mean() / seg.var() ** 2
    assert kurt == pytest.approx(6.0, rel=0.25)          # Laplace excess kurtosis 3


def test_zeros_and_ties(wl, orc):
    s = wl.spec(4, n=400_000, K=2)
    with pytest.raises(ValueError):
        wl.gradient(s, 0, 0)                 # the tied workload needs the caller's k
    g = wl.gradient(s, 0, 0, k=orc.topk_k(s.n, s.ratios[0, 0]))
    zeros = g == 0
    assert zeros.mean() == pytest.approx(0.05, abs=0.005)
    assert 0.3 < np.signbit(g[zeros]).mean() < 0.7
    mag = np.abs(g)
    vals, counts = np.unique(mag[~zeros], return_counts=True)
    assert counts.max() == pytest.approx(0.01 * s.n, rel=0.1)
