"""Edge cases of the HIP path against the oracle: tiny and ragged sizes, the
fast-path size boundary, k = 1 and k = n, all-equal and all-zero vectors,
signed zeros, denormals, ties straddling the threshold, K = 1 and K = 64,
zero weights, user-provided sets (sparse and dense), validation, determinism."""
import math

import numpy as np
import pytest

import oracle
from _gpu_common import check_energies, log, same_bits, torch_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


def topk_vs_oracle(sc, g: np.ndarray, ratio: float, label: str):
    torch, dev = torch_dev()
    k = oracle.topk_k(g.size, ratio)
    idx_o, val_o, ea, ek = oracle.topk(g, k)
    ref = oracle.energies_extended(g, idx_o)
    check_energies(f"{label} (oracle)", ea, ek, ref, g.size, k)
    for mode in ("default", "force_exact", "force_fallback"):
        if mode != "default":
            sc.set_option(mode, 1)
        try:
            idx, val, en = sc.topk_select(torch.from_numpy(g).to(dev), ratio, energies=True)
            torch.cuda.synchronize()
        finally:
            if mode != "default":
                sc.set_option(mode, 0)
        assert np.array_equal(idx.cpu().numpy(), idx_o), f"{label} [{mode}]: indices"
        assert same_bits(val.cpu().numpy(), val_o), f"{label} [{mode}]: values"
        e = en.cpu().numpy()
        check_energies(f"{label} [{mode}]", e[0], e[1], ref, g.size, k)


SIZES = [1, 2, 3, 4, 5, 255, 1023, 1024, 1025, 16383, 16384, 16385, 65535, 65536, 65537, 131072 + 77,
         1_000_000]


@pytest.mark.parametrize("n", SIZES)
def test_sizes(sc, n):
    log(f"edge sizes n={n}")
    rng = np.random.default_rng(n)
    g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-4, 0, n)).astype(np.float32)
    for ratio in (1e-9, 0.001, 0.01, 0.1, 0.3, 1.0):
        topk_vs_oracle(sc, g, ratio, f"n={n} ratio={ratio}")


def test_all_equal_zero_and_signed_zero(sc):
    log("edge equal/zero")
    n = 200_000
    eq = np.where(np.arange(n) % 3 == 0, -1.5, 1.5).astype(np.float32)
    topk_vs_oracle(sc, eq, 0.01, "all equal magnitude")
    z = np.zeros(n, dtype=np.float32)
    z[1::2] = -0.0
    topk_vs_oracle(sc, z, 0.01, "all zero with -0")
    topk_vs_oracle(sc, z, 1.0, "all zero ratio 1")


def test_denormals(sc):
    log("edge denormals")
    rng = np.random.default_rng(5)
    n = 300_000
    bits = rng.integers(1, 1 << 23, n, dtype=np.uint32) | (rng.integers(0, 2, n, dtype=np.uint32) << 31)
    g = bits.view(np.float32).copy()
    g[::1000] = np.float32(1e-30)
    topk_vs_oracle(sc, g, 0.01, "denormals")
    topk_vs_oracle(sc, g, 0.2, "denormals 0.2")


def test_ties_at_threshold(sc):
    log("edge ties")
    rng = np.random.default_rng(6)
    n = 1_000_000
    g = (rng.standard_normal(n) * 0.01).astype(np.float32)
    k = oracle.topk_k(n, 0.01)
    mag = np.sort(np.abs(g))[::-1]
    m = mag[k // 2]
    pos = rng.choice(n, size=50_000, replace=False)
    g[pos] = np.where(rng.random(pos.size) < 0.5, -m, m)
    topk_vs_oracle(sc, g, 0.01, "50k ties at the threshold")
    few = (rng.integers(-3, 4, n) * 0.5).astype(np.float32)
    topk_vs_oracle(sc, few, 0.01, "7 distinct values")
    topk_vs_oracle(sc, few, 0.45, "7 distinct values, ratio 0.45")


def test_adversarial_sample(sc):
    """Inputs built against the systematic sample (one 256-element chunk every
    65536 elements). (a) The sampled chunks hold large values, so the bracket
    from the sample sits above the true k-th largest magnitude: fewer than k
    candidates, and the device must take the exact path. (b) The largest values
    hide where the sample never looks, with a wide band of ties below them."""
    log("edge adversarial sample")
    n = 1 << 22
    pos = np.arange(n)
    g = np.full(n, 1e-6, dtype=np.float32)
    g[(pos % 65536) < 256] = 1.0
    g[(pos % 65536) == 40000] = -5.0
    g[(pos % 65536) == 50000] = 3e-3
    topk_vs_oracle(sc, g, 0.01, "bracket above the threshold")
    h = np.full(n, 1e-3, dtype=np.float32)
    h[(pos % 65536) >= 4096] = 1.0e-6
    h[(pos % 65536) == 40000] = 5.0
    h[(pos % 65536) == 40001] = -5.0
    topk_vs_oracle(sc, h, 0.001, "top values outside the sample, ties below")


def test_dense_candidate_chunks(sc):
    """A narrow high-variance band holds about half of its elements as
    candidates, far more than a 4096-element chunk can stage (512): those
    chunks take the overflow path of the single-read pass."""
    log("edge dense candidate chunks")
    rng = np.random.default_rng(11)
    n = 2_000_003
    g = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    g[300_001:500_001] = (rng.standard_normal(200_000) * 1.0).astype(np.float32)
    topk_vs_oracle(sc, g, 0.05, "dense band, ratio 0.05")
    g[1_000_000:1_004_096] = 7.0           # one fully dense chunk of ties
    topk_vs_oracle(sc, g, 0.05, "dense band + tied chunk")


def test_k1_and_kn_in_fused_step(sc):
    log("edge fused k=1/k=n")
    torch, dev = torch_dev()
    rng = np.random.default_rng(7)
    K, n = 3, 70_001
    G = (rng.standard_normal((K, n)) * 0.1).astype(np.float32)
    ratios = [1e-9, 1.0, 0.5]
    w = np.array([0.25, 0.5, 0.25], dtype=np.float32)
    out = sc.FusedStep(torch.from_numpy(G).to(dev), ratios).run(w)
    torch.cuda.synchronize()
    sets = []
    for j in range(K):
        k = oracle.topk_k(n, ratios[j])
        idx, val, _, _ = oracle.topk(G[j], k)
        assert np.array_equal(out.idx[j].cpu().numpy(), idx)
        sets.append((idx, val))
    assert same_bits(out.dense.cpu().numpy(), oracle.aggregate(sets, w, n))


def test_k1_device_and_64_devices(sc):
    log("edge K=1 / K=64")
    torch, dev = torch_dev()
    rng = np.random.default_rng(8)
    for K, n in ((1, 100_003), (64, 70_000)):
        G = (rng.standard_normal((K, n)) * 10.0 ** rng.uniform(-5, -1, (K, 1))).astype(np.float32)
        rates = rng.uniform(1, 100, K)
        if K > 1:
            rates[0] = 0.0             # a device that streamed nothing: weight 0
        w, _ = sc.stream_weights(rates)
        params = (rng.standard_normal(n) * 0.05).astype(np.float32)
        p_dev = torch.from_numpy(params).to(dev)
        out = sc.FusedStep(torch.from_numpy(G).to(dev), [0.01] * K, params=p_dev).run(w, 0.05)
        torch.cuda.synchronize()
        sets = []
        for j in range(K):
            idx, val, _, _ = oracle.topk(G[j], oracle.topk_k(n, 0.01))
            assert np.array_equal(out.idx[j].cpu().numpy(), idx), f"K={K} device {j}"
            sets.append((idx, val))
        dense = oracle.aggregate(sets, w, n)
        assert same_bits(out.dense.cpu().numpy(), dense)
        assert same_bits(p_dev.cpu().numpy(), oracle.sgd(params, dense, 0.05))


def test_weighted_aggregate_user_sets(sc):
    """The standalone aggregation call on sets it did not produce, sparse and dense."""
    log("edge user sets")
    torch, dev = torch_dev()
    rng = np.random.default_rng(9)
    n = 123_457
    sets, dsets = [], []
    for j, kind in enumerate(["sparse", "dense", "sparse", "empty", "sparse"]):
        if kind == "dense":
            v = rng.standard_normal(n).astype(np.float32)
            sets.append((None, v))
            dsets.append((None, torch.from_numpy(v).to(dev)))
        else:
            k = 0 if kind == "empty" else int(rng.integers(1, n // 3))
            idx = np.sort(rng.choice(n, size=k, replace=False)).astype(np.uint32)
            v = rng.standard_normal(k).astype(np.float32)
            sets.append((idx, v))
            dsets.append((torch.from_numpy(idx).to(dev), torch.from_numpy(v).to(dev)))
    w = np.array([0.1, 0.2, 0.3, 0.15, 0.25], dtype=np.float32)
    got = sc.weighted_aggregate(dsets, w, n)
    torch.cuda.synchronize()
    assert same_bits(got.cpu().numpy(), oracle.aggregate(sets, w, n))


def test_validation_mode(sc):
    log("edge validation")
    torch, dev = torch_dev()
    n = 10_000
    idx = torch.tensor([5, 3, 9], dtype=torch.uint32, device=dev)
    val = torch.ones(3, dtype=torch.float32, device=dev)
    sc.set_option("validate", 1)
    try:
        with pytest.raises(sc.ScadlesError) as e:
            sc.weighted_aggregate([(idx, val)], [1.0], n)
        assert e.value.code == 4
        big = torch.tensor([5, 9, n + 3], dtype=torch.uint32, device=dev)
        with pytest.raises(sc.ScadlesError):
            sc.weighted_aggregate([(big, val)], [1.0], n)
        ok = torch.tensor([3, 5, 9], dtype=torch.uint32, device=dev)
        got = sc.weighted_aggregate([(ok, val)], [1.0], n).cpu().numpy()
        assert got[3] == 1.0 and got[5] == 1.0 and got[9] == 1.0 and got.sum() == 3.0
    finally:
        sc.set_option("validate", 0)


def test_apply_sgd(sc):
    log("edge sgd")
    torch, dev = torch_dev()
    rng = np.random.default_rng(10)
    for n in (1, 3, 4, 1_000_003):
        p = (rng.standard_normal(n) * 0.05).astype(np.float32)
        g = (rng.standard_normal(n) * 0.01).astype(np.float32)
        pd = torch.from_numpy(p).to(dev)
        sc.apply_sgd(pd, torch.from_numpy(g).to(dev), 0.0125)
        torch.cuda.synchronize()
        assert same_bits(pd.cpu().numpy(), oracle.sgd(p, g, 0.0125))


def test_determinism(sc):
    """Re-running gives bit-identical outputs, whatever the scheduling."""
    log("edge determinism")
    torch, dev = torch_dev()
    import workloads
    s = workloads.spec(4, n=2_000_003, K=16)
    G = torch.from_numpy(np.stack([workloads.gradient(s, 0, j, k=oracle.topk_k(s.n, s.ratios[0, j]))
                                   for j in range(s.K)])).to(dev)
    w, _ = sc.stream_weights(s.rates[0])
    step = sc.FusedStep(G, s.ratios[0], delta=0.5)
    ref = None
    for rep in range(3):
        out = step.run(w)
        torch.cuda.synchronize()
        snap = ([t.cpu().numpy().copy() for t in out.idx], [t.cpu().numpy().copy() for t in out.val],
                out.dense.cpu().numpy().copy(), out.energies.cpu().numpy().copy(),
                out.compressed.cpu().numpy().copy())
        if ref is None:
            ref = snap
        else:
            for a, b in zip(ref[0], snap[0]):
                assert np.array_equal(a, b)
            for a, b in zip(ref[1], snap[1]):
                assert same_bits(a, b)
            assert same_bits(ref[2], snap[2])
            assert np.array_equal(ref[3].view(np.uint64), snap[3].view(np.uint64))
            assert np.array_equal(ref[4], snap[4])


def test_validation_reports_internal_errors(sc):
    """In validation mode the selection calls read every device's state back:
    a clean call returns OK, a count check forced to fail (from the host, for
    device 0) returns SCADLES_EINTERNAL naming the device; without validation
    the same call returns OK (nothing is read back)."""
    log("edge validation of the selection state")
    torch, dev = torch_dev()
    rng = np.random.default_rng(31)
    g = torch.from_numpy(rng.standard_normal(300_001).astype(np.float32)).to(dev)
    G = torch.from_numpy(rng.standard_normal((3, 200_003)).astype(np.float32)).to(dev)
    w, _ = sc.stream_weights([1.0, 2.0, 3.0])
    try:
        sc.set_option("validate", 1)
        sc.topk_select(g, 0.01)
        sc.FusedStep(G, [0.01] * 3).run(w)
        sc.set_option("inject_count_error", 1)
        with pytest.raises(sc.ScadlesError) as e1:
            sc.topk_select(g, 0.01)
        assert e1.value.code == 5 and "device 0" in str(e1.value)
        with pytest.raises(sc.ScadlesError) as e2:
            sc.FusedStep(G, [0.01] * 3).run(w)
        assert e2.value.code == 5
        sc.set_option("validate", 0)
        sc.topk_select(g, 0.01)
        torch.cuda.synchronize()
    finally:
        sc.set_option("inject_count_error", 0)
        sc.set_option("validate", 0)


@pytest.mark.parametrize("offset", [0, 1, 3])
def test_overflowed_interior_and_edge_tiles(sc, offset):
    """Tiles whose candidates overflow the main pass's staging are re-scanned
    after it: dense magnitudes in the first, a middle and the last tile make
    all three overflow, at a 4-byte offset into the buffer (offset 1 and 3:
    the first tile is an edge tile holding pads) and with a ragged end."""
    torch, dev = torch_dev()
    n = 9 * 16384 + 777
    rng = np.random.default_rng(41 + offset)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    g[:20000] = (rng.standard_normal(20000) * 10.0).astype(np.float32)
    g[4 * 16384:5 * 16384] = (rng.standard_normal(16384) * 10.0).astype(np.float32)
    g[-3000:] = (rng.standard_normal(3000) * 10.0).astype(np.float32)
    buf = torch.zeros(n + 4, dtype=torch.float32, device=dev)
    buf[offset:offset + n].copy_(torch.from_numpy(g))
    view = buf[offset:offset + n]
    log(f"edge overflowed tiles, offset {offset}")
    for ratio in (0.05, 0.1):
        k = oracle.topk_k(n, ratio)
        idx_o, val_o, ea, ek = oracle.topk(g, k)
        idx, val, en = sc.topk_select(view, ratio, energies=True)
        torch.cuda.synchronize()
        assert np.array_equal(idx.cpu().numpy(), idx_o), f"offset {offset} ratio {ratio}: indices"
        assert same_bits(val.cpu().numpy(), val_o), f"offset {offset} ratio {ratio}: values"
        e = en.cpu().numpy()
        check_energies(f"offset {offset} ratio {ratio}", e[0], e[1], oracle.energies_extended(g, idx_o), n, k)
