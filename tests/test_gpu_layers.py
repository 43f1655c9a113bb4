"""Per-layer Top-k on the HIP path against the oracle (every layer keeps its
own top fraction, the per-layer reading of the Top-k of §IV): the workloads'
own layer layouts, tiny and ragged layers, ties across layer bounds, every
selection path, and the layered sets fed to the Eqn 4b aggregation. Indices
and values bit for bit; energies within the bound of a double sum of their
terms in any order, against extended-precision references."""

import numpy as np
import pytest

import oracle
import workloads
from _gpu_common import check_energies, decision_window, log, same_bits, torch_dev

pytestmark = pytest.mark.gpu

MODES = ("default", "force_exact", "force_fallback")
# Layers of at most row_max elements are selected by one workgroup per
# (device, layer) row; longer ones by the multi-launch selection. 0 sends every
# layer to the multi-launch selection, 2^32 - 1 every layer to the rows.
ROW_MAX_DEFAULT = 1 << 21
ROW_MAXES = (ROW_MAX_DEFAULT, 0, 2**32 - 1)
# Rows of more than row_split elements (at least 65536) are split into parts
# read by workgroups of their own: the default splits every row above 65536
# elements, 2^18 only the longer ones, 2^32 - 1 none. These runs take the
# test's largest row_max (with the default list, every layer a row).
ROW_SPLIT_DEFAULT = 65536
ROW_SPLITS = (1 << 18, 2**32 - 1)
LAYER_ORDER_DEFAULT = 1


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


def layers_vs_oracle(sc, G: np.ndarray, seg_off, ratios, label, modes=("default",), topk=None,
                     check_aggregate=False, row_maxes=ROW_MAXES, row_splits=ROW_SPLITS):
    """Run the per-layer selection of every device of G (K x n) and compare it
    with the oracle; returns the oracle's per-device results."""
    torch, dev = torch_dev()
    K = G.shape[0]
    fn = topk or oracle.topk_layers
    ref = [fn(G[j], seg_off, ratios[j]) for j in range(K)]
    refs = [oracle.energies_extended(G[j], ref[j][0]) for j in range(K)]
    for j in range(K):
        check_energies(f"{label} device {j} (oracle)", ref[j][2], ref[j][3], refs[j], G.shape[1], ref[j][0].size)
    g_dev = torch.from_numpy(G).to(dev)
    runs = ([(m, ROW_MAX_DEFAULT, ROW_SPLIT_DEFAULT) for m in modes]
            + [("default", r, ROW_SPLIT_DEFAULT) for r in row_maxes if r != ROW_MAX_DEFAULT or not modes]
            + [("default", max(row_maxes), r) for r in row_splits])
    for mode, row_max, row_split in runs:
        if mode != "default":
            sc.set_option(mode, 1)
        sc.set_option("row_max", row_max)
        sc.set_option("row_split", row_split)
        try:
            sel = sc.LayerSelect(g_dev, seg_off, ratios)
            idx, val, en = sel.run()
            torch.cuda.synchronize()
        finally:
            if mode != "default":
                sc.set_option(mode, 0)
            sc.set_option("row_max", ROW_MAX_DEFAULT)
            sc.set_option("row_split", ROW_SPLIT_DEFAULT)
        mode = f"{mode}, row_max {row_max}, row_split {row_split}"
        e = en.cpu().numpy()
        for j in range(K):
            idx_o, val_o, ea, ek = ref[j]
            got = idx[j].cpu().numpy()
            if not np.array_equal(got, idx_o):
                bad = np.flatnonzero(got != idx_o) if got.shape == idx_o.shape else "length"
                raise AssertionError(f"{label} [{mode}] device {j}: indices (first mismatch {bad[:5]})")
            assert same_bits(val[j].cpu().numpy(), val_o), f"{label} [{mode}] device {j}: values"
            check_energies(f"{label} [{mode}] device {j}", e[2 * j], e[2 * j + 1], refs[j], G.shape[1],
                           idx_o.size)
        if check_aggregate:
            w, _ = sc.stream_weights(np.arange(1.0, K + 1.0))
            dense = sc.weighted_aggregate(list(zip(idx, val)), w, G.shape[1])
            torch.cuda.synchronize()
            dense_o = oracle.aggregate([(r[0], r[1]) for r in ref], w, G.shape[1])
            assert same_bits(dense.cpu().numpy(), dense_o), f"{label} [{mode}]: aggregate of the layered sets"
        del sel
    return ref


@pytest.mark.parametrize("config,n,K", [(1, None, None), (2, 700_001, 3), (3, 400_000, 4), (4, 900_000, 2),
                                        (5, 1_200_000, 3)])
def test_workload_layers(sc, config, n, K):
    s = workloads.spec(config, n=n, K=K, iterations=1)
    seg_off = [0] + [int(x) for x in s.seg_end]
    log(f"layers C{config} n={s.n} K={s.K} L={len(seg_off) - 1}")
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j], k=oracle.topk_k(s.n, s.ratios[0, j]))
    layers_vs_oracle(sc, G, seg_off, list(s.ratios[0]), f"C{config} layers", modes=MODES,
                     check_aggregate=True)


def test_tiny_and_ragged_layers(sc):
    rng = np.random.default_rng(11)
    sizes = [1, 2, 3, 4, 5, 63, 64, 65, 255, 1023, 1024, 1025, 16385, 65537, 131072 + 77, 7]
    seg_off = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    n = seg_off[-1]
    K = 3
    G = (rng.standard_normal((K, n)) * 10.0 ** rng.uniform(-4, 0, (K, n))).astype(np.float32)
    for ratios in ([1e-9, 0.01, 0.3], [1.0, 0.5, 0.001]):
        log(f"layers tiny/ragged ratios={ratios}")
        layers_vs_oracle(sc, G, seg_off, ratios, f"ragged {ratios}", modes=MODES)


def test_ties_across_layer_bounds(sc):
    # few magnitude levels, signed zeros: every layer's threshold is tied, and
    # equal values sit on both sides of each layer bound
    rng = np.random.default_rng(12)
    n = 300_000
    seg_off = [0, 1000, 1001, 70_000, 70_001, 150_000, n]
    G = (rng.integers(-3, 4, size=(2, n)) * 0.5).astype(np.float32)
    G[rng.random((2, n)) < 0.2] = -0.0
    for ratios in ([0.01, 0.1], [0.5, 0.9]):
        log(f"layers ties ratios={ratios}")
        layers_vs_oracle(sc, G, seg_off, ratios, f"ties {ratios}", modes=MODES)


def test_layers_at_the_row_limit(sc):
    # one layer just at the row limit (selected by a workgroup, its threshold
    # bin too large for LDS), one just above it (multi-launch selection), and
    # a short tail
    rng = np.random.default_rng(15)
    sizes = [ROW_MAX_DEFAULT, ROW_MAX_DEFAULT + 1, 3]
    seg_off = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    G = rng.standard_normal((2, seg_off[-1])).astype(np.float32)
    log("layers at the row limit")
    layers_vs_oracle(sc, G, seg_off, [0.01, 0.3], "row limit", topk=oracle.topk_layers_by_threshold,
                     row_maxes=(ROW_MAX_DEFAULT,))


def test_rows_with_equal_keys(sc):
    # whole layers of one magnitude (every key tied), of zeros and signed
    # zeros, and a layer whose keys differ only in the lowest bits
    n_l = 40_000
    parts = [np.full(n_l, -1.25, dtype=np.float32), np.zeros(n_l, dtype=np.float32),
             np.where(np.arange(n_l) % 2 == 0, 0.0, -0.0).astype(np.float32),
             (np.float32(1.0) + np.arange(n_l, dtype=np.float32) % 7 * np.float32(2.0**-23)).astype(np.float32)]
    g = np.concatenate(parts)
    seg_off = [0, n_l, 2 * n_l, 3 * n_l, 4 * n_l]
    log("layers with equal keys")
    layers_vs_oracle(sc, np.stack([g, -g]), seg_off, [0.01, 0.5], "equal keys")


def test_split_rows(sc):
    # rows split into parts: lengths around the part size (65536) and its
    # multiples, unaligned layer starts, a row whose keys are all equal and
    # one with few magnitude levels (their selection intervals overflow, so
    # the select kernel writes them on its own), dense large magnitudes in one
    # part only
    rng = np.random.default_rng(18)
    sizes = [65_537, 3, 131_071, 131_073, 1, 200_000, 100_000, 90_001, 70_000]
    seg_off = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    n = seg_off[-1]
    G = rng.standard_normal((2, n)).astype(np.float32)
    a, b = seg_off[6], seg_off[7]
    G[:, a:b] = -2.5                                       # all keys equal
    a, b = seg_off[7], seg_off[8]
    G[:, a:b] = (rng.integers(-3, 4, size=(2, b - a)) * 0.25).astype(np.float32)
    a = seg_off[5]
    G[:, a + 70_000:a + 75_000] *= 1e3                     # large values in one part
    for ratios in ([0.01, 0.2], [0.001, 0.6]):
        log(f"layers split rows ratios={ratios}")
        layers_vs_oracle(sc, G, seg_off, ratios, f"split rows {ratios}", row_maxes=(ROW_MAX_DEFAULT,),
                         row_splits=(0,))


def test_one_layer_matches_whole_vector(sc):
    torch, dev = torch_dev()
    rng = np.random.default_rng(13)
    n = 500_000
    g = rng.standard_normal(n).astype(np.float32)
    log("layers L=1 vs the whole-vector selection")
    idx, val, en = sc.LayerSelect(torch.from_numpy(g[None, :]).to(dev), [0, n], [0.01]).run()
    idx1, val1, en1 = sc.topk_select(torch.from_numpy(g).to(dev), 0.01, energies=True)
    torch.cuda.synchronize()
    assert np.array_equal(idx[0].cpu().numpy(), idx1.cpu().numpy())
    assert same_bits(val[0].cpu().numpy(), val1.cpu().numpy())
    e, e1 = en.cpu().numpy(), en1.cpu().numpy()
    k = idx1.numel()
    ref = oracle.energies_extended(g, idx1.cpu().numpy())
    check_energies("one layer", e[0], e[1], ref, n, k)
    check_energies("whole vector", e1[0], e1[1], ref, n, k)


def test_repeated_runs_reuse_workspace(sc):
    torch, dev = torch_dev()
    rng = np.random.default_rng(14)
    n = 250_000
    seg_off = [0, 100, 60_000, 60_100, n]
    G = rng.standard_normal((2, n)).astype(np.float32)
    ref = [oracle.topk_layers(G[j], seg_off, 0.02) for j in range(2)]
    g_dev = torch.from_numpy(G).to(dev)
    sel = sc.LayerSelect(g_dev, seg_off, [0.02, 0.02])
    log("layers repeated runs")
    for _ in range(3):
        idx, val, en = sel.run()
        torch.cuda.synchronize()
        for j in range(2):
            assert np.array_equal(idx[j].cpu().numpy(), ref[j][0])
            assert same_bits(val[j].cpu().numpy(), ref[j][1])


def test_layers_validation(sc):
    torch, dev = torch_dev()
    g = torch.zeros(10, dtype=torch.float32, device=dev)
    with pytest.raises(sc.ScadlesError):
        sc.LayerSelect([g], [0, 5, 5, 10], [0.5])
    with pytest.raises(ValueError):
        sc.LayerSelect([g], [0, 5, 11], [0.5])
    with pytest.raises(sc.ScadlesError):
        sc.LayerSelect([g], [0, 5, 10], [0.0])


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_full_size_vgg19_layers_fused(sc):
    """The largest workload (32 devices x 143,667,240, its 38 layers) at ratio
    0.01 in the launch configuration the benchmark times: the fused per-layer
    step (selection, the rule of §IV at delta = +inf, Eqn 4b, Eqn 4c) over two
    consecutive iterations, every device's kept set against the O(n) oracle,
    the aggregate and the update bit for bit."""
    from concurrent.futures import ThreadPoolExecutor
    torch, dev = torch_dev()
    s = workloads.spec(5, iterations=2)
    seg_off = [0] + [int(x) for x in s.seg_end]
    log(f"full-size fused layers C5 n={s.n} K={s.K} L={len(seg_off) - 1}")
    G = torch.empty((s.K, s.n), dtype=torch.float32, device=dev)
    params = workloads.params0(s)
    p_dev = torch.from_numpy(params).to(dev)
    p_ref = params
    host = np.empty(s.n, dtype=np.float32)
    step = None
    for it in range(s.iterations):
        for j in range(s.K):
            workloads.gradient(s, it, j, out=host)
            G[j].copy_(torch.from_numpy(host))
        if step is None:
            step = sc.FusedStep(G, s.ratios[0], params=p_dev, seg_off=seg_off)
        w, gam = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
        lr = float(np.float32(s.eta * gam))
        out = step.run(w, lr)
        torch.cuda.synchronize()
        log(f"  iteration {it}: step done, oracle on every device")

        def one(j):
            g = workloads.gradient(s, it, j, nthreads=2)
            idx, val, ea, ek = oracle.topk_layers_by_threshold(g, seg_off, s.ratios[it, j])
            return idx, val, ea, ek, oracle.energies_extended(g, idx)

        with ThreadPoolExecutor(8) as ex:
            res = list(ex.map(one, range(s.K)))
        e = out.energies.cpu().numpy()
        assert np.all(out.compressed.cpu().numpy() == 1), "delta = +inf always sends Top-k"
        sets = []
        for j, (idx, val, ea, ek, ref) in enumerate(res):
            assert np.array_equal(out.idx[j].cpu().numpy(), idx), f"iteration {it} device {j}: indices"
            assert same_bits(out.val[j].cpu().numpy(), val), f"iteration {it} device {j}: values"
            check_energies(f"iteration {it} device {j} (oracle)", ea, ek, ref, s.n, idx.size)
            check_energies(f"iteration {it} device {j}", e[2 * j], e[2 * j + 1], ref, s.n, idx.size)
            sets.append((idx, val))
        dense_o = oracle.aggregate(sets, w, s.n)
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"iteration {it}: aggregate"
        p_ref = oracle.sgd(p_ref, dense_o, lr)
        assert same_bits(p_dev.cpu().numpy(), p_ref), f"iteration {it}: update"
        del res, sets, dense_o


@pytest.mark.parametrize("config,n,K,iters,beta,optimizer", [(5, 1_500_001, 6, 3, 0.5, "sgd"),
                                                              (2, 700_001, 8, 2, None, "momentum"),
                                                              (4, 900_000, 4, 2, 0.9, "momentum")])
def test_fused_layers_step(sc, config, n, K, iters, beta, optimizer):
    """Per-layer selection, the adaptive rule on the whole-gradient energies
    (moving average when beta is set), Eqn 4b and the update in one call,
    over several iterations with fresh gradients, against the oracle."""
    torch, dev = torch_dev()
    s = workloads.spec(config, n=n, K=K, iterations=iters)
    seg_off = [0] + [int(x) for x in s.seg_end]
    log(f"fused layers C{config} n={s.n} K={s.K} L={len(seg_off) - 1} beta={beta} {optimizer}")
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j], k=oracle.topk_k(s.n, s.ratios[0, j]))
    sets0 = [oracle.topk_layers(G[j], seg_off, s.ratios[0, j]) for j in range(s.K)]
    rho = sorted(oracle.compress_decision(r[2], r[3], 0.0)[1] for r in sets0)
    delta = 0.5 * (rho[len(rho) // 2 - 1] + rho[len(rho) // 2])
    g_dev = torch.from_numpy(G).to(dev)
    params = workloads.params0(s)
    p_dev = torch.from_numpy(params).to(dev)
    mom = (0.9, 5e-4) if optimizer == "momentum" else None
    v_dev = torch.zeros(s.n, dtype=torch.float32, device=dev) if mom else None
    step = sc.FusedStep(g_dev, s.ratios[0], delta=delta, params=p_dev, seg_off=seg_off, ewma_beta=beta, track=True,
                        momentum_buf=v_dev, momentum=mom[0] if mom else 0.0, weight_decay=mom[1] if mom else 0.0)
    p_ref = params.copy()
    v_ref = np.zeros(s.n, dtype=np.float32)
    state = np.zeros((s.K, 2))
    counters = np.zeros((s.K, 3), dtype=np.uint64)
    for it in range(s.iterations):
        if it:
            for j in range(s.K):
                workloads.gradient(s, it, j, out=G[j], k=oracle.topk_k(s.n, s.ratios[it, j]))
            g_dev.copy_(torch.from_numpy(G))
        res = sets0 if it == 0 else [oracle.topk_layers(G[j], seg_off, s.ratios[it, j]) for j in range(s.K)]
        w, gamma = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
        lr = float(np.float32(s.eta * gamma))
        out = step.run(w, lr)
        torch.cuda.synchronize()
        got = out.compressed.cpu().numpy()
        e = out.energies.cpu().numpy()
        sets = []
        for j, (idx, val, e_all, e_kept) in enumerate(res):
            assert np.array_equal(out.idx[j].cpu().numpy(), idx), f"iteration {it} device {j}: indices"
            assert same_bits(out.val[j].cpu().numpy(), val), f"iteration {it} device {j}: values"
            check_energies(f"iteration {it} device {j}", e[2 * j], e[2 * j + 1],
                           oracle.energies_extended(G[j], idx), s.n, idx.size)
            if beta is None:
                send, r = oracle.compress_decision(e_all, e_kept, delta)
            else:
                send = oracle.adaptive_step(state[j], counters[j], e_all, e_kept, beta, delta,
                                            oracle.layers_k(seg_off, s.ratios[it, j]), s.n)
                r = oracle.compress_decision(state[j][0], state[j][1], 0.0)[1]
            if abs(r - delta) <= decision_window(s.n, idx.size, updates=0 if beta is None else it + 1):
                send = bool(got[j])               # within rounding of delta either answer is correct
            assert bool(got[j]) == send, f"iteration {it} device {j}: decision"
            sets.append((idx, val) if send else (None, G[j]))
        dense_o = oracle.aggregate(sets, w, s.n)
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"iteration {it}: aggregate"
        if mom:
            p_ref, v_ref = oracle.momentum_sgd(p_ref, v_ref, dense_o, lr, mom[0], mom[1])
            assert same_bits(v_dev.cpu().numpy(), v_ref), f"iteration {it}: momentum buffer"
        else:
            p_ref = oracle.sgd(p_ref, dense_o, lr)
        assert same_bits(p_dev.cpu().numpy(), p_ref), f"iteration {it}: update"
    acc = step.accounting()
    assert np.all(acc[:, 1] == s.iterations)
    sent = acc[:, 0]
    assert np.all(acc[:, 2] == sent * np.array(step.k) + (s.iterations - sent) * s.n)


def test_fused_layers_sparse_sets(sc):
    """Fused per-layer step with kept sets so sparse that consecutive kept
    indices lie many aggregation ranges apart (down to one entry per layer),
    beside denser devices and one that keeps everything: each range's first
    entry is found for every device, so the aggregate and the update match the
    oracle bit for bit."""
    torch, dev = torch_dev()
    ratios = [1e-6, 2e-5, 3e-4, 0.02, 1.0]
    s = workloads.spec(5, n=3_000_001, K=len(ratios), iterations=1)
    seg_off = [0] + [int(x) for x in s.seg_end]
    log(f"fused layers, sparse sets n={s.n} K={s.K} L={len(seg_off) - 1} ratios={ratios}")
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j], k=oracle.topk_k(s.n, ratios[j]))
    g_dev = torch.from_numpy(G).to(dev)
    params = workloads.params0(s)
    p_dev = torch.from_numpy(params).to(dev)
    step = sc.FusedStep(g_dev, ratios, params=p_dev, seg_off=seg_off)
    w, gamma = sc.stream_weights(s.rates[0], base_batch=s.base_batch)
    lr = float(np.float32(s.eta * gamma))
    for rep in range(2):          # the second call reuses the first call's markers' memory
        out = step.run(w, lr)
        torch.cuda.synchronize()
        sets = []
        for j in range(s.K):
            idx, val, _, _ = oracle.topk_layers(G[j], seg_off, ratios[j])
            assert np.array_equal(out.idx[j].cpu().numpy(), idx), f"call {rep} device {j}: indices"
            assert same_bits(out.val[j].cpu().numpy(), val), f"call {rep} device {j}: values"
            sets.append((idx, val))
        gaps = np.diff(sets[0][0].astype(np.int64)) // 2048
        assert gaps.max() > 64, "the sparsest device spans many ranges between kept entries"
        dense_o = oracle.aggregate(sets, w, s.n)
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"call {rep}: aggregate"
        params = oracle.sgd(params, dense_o, lr)
        assert same_bits(p_dev.cpu().numpy(), params), f"call {rep}: update"


def test_layer_order(sc):
    """The long layers run in index order, by ascending or by descending
    length: each writes its own part of the outputs and of the per-layer
    energies, summed in layer order, so the kept sets, the energies (bit for
    bit) and the fused step's aggregate and update do not change, and match
    the oracle."""
    torch, dev = torch_dev()
    s = workloads.spec(5, n=2_000_003, K=3, iterations=1)
    seg_off = [0] + [int(x) for x in s.seg_end]
    row_max = 1 << 15
    nlong = int(np.sum(np.diff(seg_off) > row_max))
    log(f"layer order n={s.n} K={s.K} L={len(seg_off) - 1}, {nlong} long layers")
    assert nlong >= 4
    ratios = [0.01, 0.003, 0.05]
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j], k=oracle.topk_k(s.n, ratios[j]))
    ref = [oracle.topk_layers(G[j], seg_off, ratios[j]) for j in range(s.K)]
    g_dev = torch.from_numpy(G).to(dev)
    params = workloads.params0(s)
    w, gamma = sc.stream_weights(s.rates[0], base_batch=s.base_batch)
    lr = float(np.float32(s.eta * gamma))
    dense_o = oracle.aggregate([(r[0], r[1]) for r in ref], w, s.n)
    p_ref = oracle.sgd(params, dense_o, lr)
    energies = []
    for order in (0, 1, 2):
        sc.set_option("layer_order", order)
        sc.set_option("row_max", row_max)
        try:
            sel = sc.LayerSelect(g_dev, seg_off, ratios)
            idx, val, en = sel.run()
            p_dev = torch.from_numpy(params).to(dev)
            step = sc.FusedStep(g_dev, ratios, params=p_dev, seg_off=seg_off)
            out = step.run(w, lr)
            torch.cuda.synchronize()
        finally:
            sc.set_option("layer_order", LAYER_ORDER_DEFAULT)
            sc.set_option("row_max", ROW_MAX_DEFAULT)
        e = en.cpu().numpy()
        for j in range(s.K):
            idx_o, val_o, _, _ = ref[j]
            assert np.array_equal(idx[j].cpu().numpy(), idx_o), f"order {order} device {j}: indices"
            assert same_bits(val[j].cpu().numpy(), val_o), f"order {order} device {j}: values"
            assert np.array_equal(out.idx[j].cpu().numpy(), idx_o), f"order {order} device {j}: fused indices"
            check_energies(f"order {order} device {j}", e[2 * j], e[2 * j + 1],
                           oracle.energies_extended(G[j], idx_o), s.n, idx_o.size)
        assert same_bits(out.energies.cpu().numpy(), e), f"order {order}: fused step's energies"
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"order {order}: aggregate"
        assert same_bits(p_dev.cpu().numpy(), p_ref), f"order {order}: update"
        energies.append(e)
        del sel, step
    for order in (1, 2):
        assert same_bits(energies[order], energies[0]), f"order {order}: energies differ from index order"


def test_layers_validation_of_long_layers(sc):
    """With the validate option the per-layer calls read the long layers'
    selection checks back: OK on good input, SCADLES_EINTERNAL (code 5) for
    device 0 when the count check is made to fail; without the option the
    same calls return OK."""
    torch, dev = torch_dev()
    rng = np.random.default_rng(37)
    n = 2_600_001
    seg_off = [0, 120_000, 120_000 + (1 << 21) + 5_000, n]       # the middle layer is long
    G = torch.from_numpy(rng.standard_normal((3, n)).astype(np.float32)).to(dev)
    w, _ = sc.stream_weights([1.0, 2.0, 3.0])
    log("per-layer validation of the long layers' selection state")
    try:
        sc.set_option("validate", 1)
        sc.LayerSelect(G, seg_off, [0.01] * 3).run()
        sc.FusedStep(G, [0.01] * 3, seg_off=seg_off).run(w)
        sc.set_option("inject_count_error", 1)
        with pytest.raises(sc.ScadlesError) as e1:
            sc.LayerSelect(G, seg_off, [0.01] * 3).run()
        assert e1.value.code == 5 and "device 0" in str(e1.value)
        with pytest.raises(sc.ScadlesError) as e2:
            sc.FusedStep(G, [0.01] * 3, seg_off=seg_off).run(w)
        assert e2.value.code == 5
        sc.set_option("validate", 0)
        sc.LayerSelect(G, seg_off, [0.01] * 3).run()
        torch.cuda.synchronize()
    finally:
        sc.set_option("inject_count_error", 0)
        sc.set_option("validate", 0)


def test_long_row_without_chunk_tallies(sc):
    # with every layer short, a 3M-element layer is one workgroup's row, too
    # long for the per-chunk tallies: its output takes the scanned path
    rng = np.random.default_rng(16)
    sizes = [3_000_000, 1000]
    seg_off = np.concatenate([[0], np.cumsum(sizes)]).tolist()
    G = (rng.standard_normal((2, seg_off[-1])) * rng.uniform(0.1, 2.0, (2, 1))).astype(np.float32)
    log("layers: one long row without chunk tallies")
    layers_vs_oracle(sc, G, seg_off, [0.01, 0.2], "long row", topk=oracle.topk_layers_by_threshold,
                     row_maxes=(2**32 - 1,), modes=())


def test_select_layers_without_energies(sc):
    import ctypes
    torch, dev = torch_dev()
    rng = np.random.default_rng(17)
    seg_off = [0, 5000, 3_000_000, 3_000_100]
    G = rng.standard_normal((2, seg_off[-1])).astype(np.float32)
    ref = [oracle.topk_layers(G[j], seg_off, 0.01) for j in range(2)]
    g_dev = torch.from_numpy(G).to(dev)
    sel = sc.LayerSelect(g_dev, seg_off, [0.01, 0.01])
    log("layers without energies")
    rc = sc._topk_select_layers(sel._grad_ptrs, sel.K, sel._seg, sel._L, sel._ratios, sel._idx_ptrs, sel._val_ptrs,
                                None, sel.ws.data_ptr(), sel.ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    for j in range(2):
        assert np.array_equal(sel.idx[j].cpu().numpy(), ref[j][0])
        assert same_bits(sel.val[j].cpu().numpy(), ref[j][1])


@pytest.mark.parametrize("K", [1, 64])
def test_device_count_extremes(sc, K):
    # one device, and the most devices a call takes, over short and long layers
    rng = np.random.default_rng(18 + K)
    seg_off = [0, 3000, 40_000, 2_300_000] if K == 1 else [0, 700, 20_000, 90_000]
    G = (rng.standard_normal((K, seg_off[-1])) * rng.uniform(0.01, 3.0, (K, 1))).astype(np.float32)
    ratios = list(rng.choice([0.001, 0.01, 0.1, 0.5], size=K))
    log(f"layers with K={K}")
    ref = layers_vs_oracle(sc, G, seg_off, ratios, f"K={K}", topk=oracle.topk_layers_by_threshold,
                           check_aggregate=True)
    # the fused per-layer step (its own range markers, Eqn 4b, Eqn 4c) at this K
    torch, dev = torch_dev()
    n = seg_off[-1]
    params = rng.standard_normal(n).astype(np.float32)
    p_dev = torch.from_numpy(params).to(dev)
    w, _ = sc.stream_weights(np.arange(1.0, K + 1.0))
    lr = float(np.float32(0.05))
    out = sc.FusedStep(torch.from_numpy(G).to(dev), ratios, params=p_dev, seg_off=seg_off).run(w, lr)
    torch.cuda.synchronize()
    dense_o = oracle.aggregate([(r[0], r[1]) for r in ref], w, n)
    assert same_bits(out.dense.cpu().numpy(), dense_o), f"K={K}: fused per-layer aggregate"
    assert same_bits(p_dev.cpu().numpy(), oracle.sgd(params, dense_o, lr)), f"K={K}: fused per-layer update"


def test_concurrent_callers(sc):
    """Two host threads, each with its own stream, buffers and workspace, run
    per-layer selections at once: the library's shared streams and events are
    used by one call's launch sequence at a time, so both stay exact."""
    import threading
    torch, dev = torch_dev()
    rng = np.random.default_rng(19)
    seg_off = [0, 4000, 2_500_000, 2_600_000]
    data = [rng.standard_normal((2, seg_off[-1])).astype(np.float32) for _ in range(2)]
    refs = [[oracle.topk_layers(G[j], seg_off, 0.01) for j in range(2)] for G in data]
    sels = [sc.LayerSelect(torch.from_numpy(G).to(dev), seg_off, [0.01, 0.01]) for G in data]
    torch.cuda.synchronize()
    errors = []

    def work(t):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for _ in range(5):
                    idx, val, _ = sels[t].run(stream=stream)
                stream.synchronize()
            for j in range(2):
                assert np.array_equal(idx[j].cpu().numpy(), refs[t][j][0]), f"thread {t} device {j}"
                assert same_bits(val[j].cpu().numpy(), refs[t][j][1]), f"thread {t} device {j}"
        except Exception as exc:      # reported from the main thread
            errors.append(exc)

    log("layers from two threads at once")
    threads = [threading.Thread(target=work, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
