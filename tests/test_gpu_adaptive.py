"""Parity of the adaptive rule on moving averages of the energies (§IV) and of
the CNC / floats-sent accounting (§V-G) with the oracle, over several
iterations with fresh gradients. The energies are sums in double whose order
differs between the kernels and the oracle, so the averages agree within the
bound of such sums (plus the rounding of every moving-average update), and a
decision is compared wherever the oracle's loss ratio is farther from delta
than the two sides' ratios can differ. A device's counters are compared
whenever none of its decisions was that close to delta."""
import numpy as np
import pytest

import oracle
import workloads
from _gpu_common import check_energies, decision_window, gamma, log, same_bits, torch_dev, U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


def _energies(s, it, G):
    out = []
    for j in range(s.K):
        k = oracle.topk_k(s.n, s.ratios[it, j])
        idx, val, e_all, e_kept = oracle.topk(G[j], k)
        out.append((k, idx, val, e_all, e_kept))
    return out


@pytest.mark.parametrize("config,n,K,iters,beta", [(1, 300_007, 4, 6, 0.9), (3, 400_001, 16, 3, 0.5),
                                                   (2, 200_003, 8, 4, 0.0)])
def test_moving_average_rule_and_accounting(sc, config, n, K, iters, beta):
    torch, dev = torch_dev()
    s = workloads.spec(config, n=n, K=K, iterations=iters)
    log(f"adaptive C{config} n={n} K={K} beta={beta}")
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j])
    # delta between the middle two loss ratios of the first iteration: both kinds of decision occur
    first = _energies(s, 0, G)
    rho = sorted(oracle.compress_decision(e[3], e[4], 0.0)[1] for e in first)
    delta = 0.5 * (rho[len(rho) // 2 - 1] + rho[len(rho) // 2])
    g_dev = torch.from_numpy(G).to(dev)
    step = sc.FusedStep(g_dev, s.ratios[0], delta=delta, ewma_beta=beta, track=True)
    state = np.zeros((s.K, 2))
    counters = np.zeros((s.K, 3), dtype=np.uint64)
    near = np.zeros(s.K, dtype=bool)        # a device with a decision within rounding of delta
    for it in range(s.iterations):
        if it:
            for j in range(s.K):
                workloads.gradient(s, it, j, out=G[j])
            g_dev.copy_(torch.from_numpy(G))
        if any(s.ratios[it] != step.ratios):
            step.set_ratios(s.ratios[it])
        res = first if it == 0 else _energies(s, it, G)
        w, _ = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
        out = step.run(w, 0.0)
        torch.cuda.synchronize()
        got = out.compressed.cpu().numpy()
        en = out.energies.cpu().numpy()
        sets = []
        for j, (k, idx, val, e_all, e_kept) in enumerate(res):
            check_energies(f"iteration {it} device {j}", en[2 * j], en[2 * j + 1],
                           oracle.energies_extended(G[j], idx), s.n, k)
            send = oracle.adaptive_step(state[j], counters[j], e_all, e_kept, beta, delta, k, s.n)
            r = oracle.compress_decision(state[j][0], state[j][1], 0.0)[1]
            if abs(r - delta) <= decision_window(s.n, k, updates=it + 1):
                near[j] = True                    # several answers are correct here
                send = bool(got[j])
            assert bool(got[j]) == send, f"iteration {it} device {j}: decision"
            sets.append((idx, val) if send else (None, G[j]))
        dense_o = oracle.aggregate(sets, w, s.n)
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"iteration {it}: aggregate"
        # each average is a convex combination of its device's energies (relative
        # error of a double sum of n terms, both sides) plus 4u per update
        ewma = step.ewma.cpu().numpy().reshape(s.K, 2)
        rel = 2 * (gamma(s.n) + 4 * (it + 1) * U)
        assert np.all(np.abs(ewma - state) <= rel * np.abs(state)), f"iteration {it}: averages"
    acc = step.accounting()
    for j in range(s.K):
        if not near[j]:
            assert np.array_equal(acc[j], counters[j]), f"device {j}: counters"
            assert oracle.cnc_ratio(acc[j]) == oracle.cnc_ratio(counters[j])
    assert np.all(acc[:, 1] == s.iterations)
    assert 0 < sum(acc[:, 0]) < s.K * s.iterations     # both decisions occurred
    assert not near.all(), "every device had a decision within rounding of delta"


def test_zero_beta_is_the_instantaneous_rule(sc):
    """beta = 0 with accounting against the oracle's instantaneous rule and
    counters (and against the call without options, bit for bit)."""
    torch, dev = torch_dev()
    s = workloads.spec(1, n=250_001, K=4, iterations=1)
    G = np.stack([workloads.gradient(s, 0, j) for j in range(s.K)])
    g_dev = torch.from_numpy(G).to(dev)
    e = _energies(s, 0, G)
    rho = sorted(oracle.compress_decision(x[3], x[4], 0.0)[1] for x in e)
    delta = 0.5 * (rho[1] + rho[2])
    w, _ = sc.stream_weights(s.rates[0], base_batch=s.base_batch)
    a = sc.FusedStep(g_dev, s.ratios[0], delta=delta)
    b = sc.FusedStep(g_dev, s.ratios[0], delta=delta, ewma_beta=0.0, track=True)
    oa = a.run(w, 0.0)
    ca, da = oa.compressed.cpu().numpy().copy(), oa.dense.cpu().numpy().copy()
    ob = b.run(w, 0.0)
    torch.cuda.synchronize()
    assert np.array_equal(ca, ob.compressed.cpu().numpy())
    assert same_bits(da, ob.dense.cpu().numpy())
    acc = b.accounting()
    for j, (k, idx, val, e_all, e_kept) in enumerate(e):
        want = np.zeros(3, dtype=np.uint64)
        send_o = oracle.adaptive_step(np.zeros(2), want, e_all, e_kept, 0.0, delta, k, s.n)
        _, r = oracle.compress_decision(e_all, e_kept, delta)
        if abs(r - delta) > decision_window(s.n, k):
            assert bool(ca[j]) == send_o, f"device {j}: decision"
            assert np.array_equal(acc[j], want), f"device {j}: counters"
        assert acc[j, 2] == (k if ca[j] else s.n)
    sets = [(x[1], x[2]) if c else (None, G[j]) for j, (x, c) in enumerate(zip(e, ca))]
    assert same_bits(ob.dense.cpu().numpy(), oracle.aggregate(sets, w, s.n))
