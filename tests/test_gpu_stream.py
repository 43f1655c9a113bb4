"""The whole loop of a streaming iteration on the HIP path: stream buffers ->
batch sizes -> Eqn 4a weights and scaled learning rate (host) -> fused Top-k,
aggregation and SGD step (GPU), against the oracle's buffer simulation, Eqn 4a,
Top-k, aggregation and SGD over several iterations under both policies."""
import numpy as np
import pytest

import oracle
import workloads
from _gpu_common import log, same_bits, torch_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


@pytest.mark.parametrize("policy", ["persistence", "truncation"])
def test_stream_driven_steps(sc, policy):
    torch, dev = torch_dev()
    s = workloads.spec(2, n=300_000, K=6, iterations=1)
    rates = np.array([0, 3, 40, 700, 2000, 64], dtype=np.uint64)   # one silent stream, one below b_min
    iter_us = [1_600_000, 900_000, 1_200_000, 1_600_000, 200_000, 1_000_000]
    T = 4
    q_o, b_o, _ = oracle.stream_run(rates, iter_us, 8, 1024, 0 if policy == "persistence" else 1, T)
    G = np.empty((s.K, s.n), dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=G[j])
    params = workloads.params0(s)
    p_dev = torch.from_numpy(params).to(dev)
    step = sc.FusedStep(torch.from_numpy(G).to(dev), s.ratios[0], params=p_dev)
    buf = sc.StreamBuffers(rates, b_min=8, b_max=1024, policy=policy, base_batch=s.base_batch)
    ks = [oracle.topk_k(s.n, s.ratios[0, j]) for j in range(s.K)]
    sets = [oracle.topk(G[j], ks[j])[:2] for j in range(s.K)]
    p_ref = params.copy()
    for t in range(T):
        log(f"stream {policy} iteration {t}")
        batch, w, gamma = buf.iteration(iter_us)
        assert np.array_equal(batch, b_o[t])
        w_o, g_o = oracle.stream_weights(b_o[t].astype(np.float64), base_batch=s.base_batch)
        assert same_bits(w, w_o) and gamma == g_o
        lr = float(np.float32(s.eta * gamma))
        out = step.run(w, lr)
        torch.cuda.synchronize()
        dense_o = oracle.aggregate(sets, w_o, s.n)
        assert same_bits(out.dense.cpu().numpy(), dense_o), f"iteration {t}: aggregate"
        p_ref = oracle.sgd(p_ref, dense_o, lr)
        assert same_bits(p_dev.cpu().numpy(), p_ref), f"iteration {t}: SGD"
    assert np.array_equal(buf.field("queued"), q_o[T])
