"""Parity of the HIP path with the oracle on the five workloads, shrunk to sizes
the full-sort oracle finishes in seconds (many main tiles, many candidate
blocks, ragged tails). Top-k indices and values must be bit-identical; the
aggregate and the SGD update must be within 1e-6 relative / 1e-7 absolute,
and are in fact checked bit for bit (the kernels accumulate in double in device
order, as the oracle does)."""
import math

import numpy as np
import pytest

from _gpu_common import log, run_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


@pytest.fixture
def exact_mode(sc):
    sc.set_option("force_exact", 1)
    yield
    sc.set_option("force_exact", 0)


@pytest.fixture
def fallback_mode(sc):
    sc.set_option("force_fallback", 1)
    yield
    sc.set_option("force_fallback", 0)


CASES = [  # config, n, K, iterations
    (1, 300_007, 4, 1),
    (2, 400_003, 8, 1),
    (3, 500_001, 16, 3),
    (4, 1_000_003, 16, 1),
    (5, 600_001, 32, 3),
]


@pytest.mark.parametrize("config,n,K,iters", CASES)
def test_workload_fast_path(sc, config, n, K, iters):
    log(f"parity fast path C{config} n={n} K={K}")
    run_config(sc, config, n=n, K=K, iterations=iters)


@pytest.mark.parametrize("config,n,K,iters", [CASES[0], CASES[3]])
def test_workload_exact_path(sc, exact_mode, config, n, K, iters):
    log(f"parity exact path C{config} n={n} K={K}")
    run_config(sc, config, n=n, K=K, iterations=iters)


@pytest.mark.parametrize("config,n,K,iters", [CASES[1], CASES[3]])
def test_workload_runtime_fallback(sc, fallback_mode, config, n, K, iters):
    log(f"parity runtime fallback C{config} n={n} K={K}")
    run_config(sc, config, n=n, K=K, iterations=iters)


@pytest.mark.parametrize("parts", [2, 3, 4])
@pytest.mark.parametrize("config,n,K,iters", [CASES[3], CASES[4]])
def test_pipelined_device_groups(sc, parts, config, n, K, iters):
    # devices split into groups whose selections overlap on two streams
    log(f"parity with {parts} device groups C{config} n={n} K={K}")
    sc.set_option("parts", parts)
    try:
        run_config(sc, config, n=n, K=K, iterations=iters)
    finally:
        sc.set_option("parts", 1)


@pytest.mark.parametrize("mode", ["force_exact", "force_fallback"])
def test_pipelined_groups_on_the_exact_path(sc, mode):
    config, n, K, iters = CASES[3]
    log(f"parity with 2 device groups, {mode}, C{config} n={n} K={K}")
    sc.set_option("parts", 2)
    sc.set_option(mode, 1)
    try:
        run_config(sc, config, n=n, K=K, iterations=iters)
    finally:
        sc.set_option(mode, 0)
        sc.set_option("parts", 1)


def test_per_device_ratios(sc):
    log("parity per-device ratios")
    K = 16
    ratios = np.array([[0.1, 0.01, 0.001, 0.05, 0.2, 0.003, 0.3, 1.0] * 2])
    run_config(sc, 3, n=300_000, K=K, iterations=1, ratio_override=ratios)


@pytest.mark.parametrize("delta", [0.0, 0.5, 0.9])
def test_adaptive_rule_mixes_dense_and_sparse(sc, delta):
    """Finite delta: devices whose energy loss exceeds delta send their dense
    gradient (§IV); the aggregate mixes both kinds."""
    log(f"parity adaptive delta={delta}")
    run_config(sc, 3, n=200_003, K=16, iterations=3, delta=delta)


def test_full_size_c1(sc):
    """C1 at its full size with the full-sort oracle."""
    log("parity C1 full size")
    run_config(sc, 1)


def test_concurrent_fused_steps_with_groups(sc):
    """Two host threads run fused steps at once on their own streams with two
    device groups each (the library's second stream is shared between them)."""
    import threading
    import numpy as np
    import oracle
    import workloads
    from _gpu_common import same_bits, torch_dev
    torch, dev = torch_dev()
    s = workloads.spec(2, n=300_001, K=4, iterations=1)
    G = np.stack([workloads.gradient(s, 0, j) for j in range(s.K)])
    w, _ = sc.stream_weights(s.rates[0], base_batch=s.base_batch)
    sets = [oracle.topk(G[j], oracle.topk_k(s.n, s.ratios[0, j]))[:2] for j in range(s.K)]
    dense_o = oracle.aggregate(sets, w, s.n)
    steps = [sc.FusedStep(torch.from_numpy(G).to(dev), s.ratios[0]) for _ in range(2)]
    torch.cuda.synchronize()
    errors = []

    def work(t):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for _ in range(5):
                    out = steps[t].run(w, 0.0, stream=stream)
                stream.synchronize()
            assert same_bits(out.dense.cpu().numpy(), dense_o), f"thread {t}: aggregate"
        except Exception as exc:
            errors.append(exc)

    log("fused steps from two threads, two device groups")
    sc.set_option("parts", 2)
    try:
        threads = [threading.Thread(target=work, args=(t,)) for t in range(2)]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
    finally:
        sc.set_option("parts", 1)
    assert not errors, errors
