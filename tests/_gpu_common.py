"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare it with the oracle on the same seeded inputs."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
import workloads


# pytest's capture manager (set by a fixture in conftest.py): progress lines of
# long tests reach the terminal even while the test's output is captured.
CAPTURE = None


def log(msg: str):
    if CAPTURE is not None:
        with CAPTURE.global_and_fixture_disabled():
            print(msg, flush=True)
    else:
        print(msg, flush=True)
        sys.stdout.flush()


def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch, torch.device("cuda:0")


def same_bits(a: np.ndarray, b: np.ndarray) -> bool:
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    if a.shape != b.shape:
        return False
    return np.array_equal(a.view(np.uint32), b.view(np.uint32))


U = 2.0**-53          # unit roundoff of double
UX = 2.0**-64         # unit roundoff of the x86-64 long double of the energy references


def gamma(m: int, u: float = U) -> float:
    """gamma_m = m u / (1 - m u). Any order of additions of m + 1 non-negative
    terms, each exact, rounds every term at most m times, so the computed sum
    is within gamma_m of the exact one, relative to it."""
    m = max(int(m), 0)
    return m * u / (1.0 - m * u)


def energy_bound(m: int, ref) -> float:
    """Largest |kernel sum - reference| for an energy of m exact squares: the
    kernels add them in an order of their own (gamma_{m-1}; one more rounding
    is allowed for a product folded into a sum, hence gamma_m), the reference
    (oracle.energies_extended) is within gamma_{m-1} of exact in long double."""
    return (gamma(m) + gamma(m, UX)) * float(ref)


def check_energies(label: str, got_all: float, got_kept: float, ref, n: int, k: int):
    """Both energies of one device against the extended-precision references
    ref = (E_all, E_kept) of n and k terms."""
    ra, rk = ref
    assert abs(float(got_all) - float(ra)) <= energy_bound(n, ra), \
        f"{label}: E_all {got_all!r} vs {float(ra)!r} (bound {energy_bound(n, ra):.3g})"
    assert abs(float(got_kept) - float(rk)) <= energy_bound(k, rk), \
        f"{label}: E_kept {got_kept!r} vs {float(rk)!r} (bound {energy_bound(k, rk):.3g})"


def decision_window(n: int, k: int, updates: int = 0) -> float:
    """How far apart two computations of the §IV loss ratio rho = (E_all -
    E_kept) / E_all may be. With relative errors a and b in E_all and E_kept,
    rho~ = (rho + alpha - (E_kept / E_all) beta) / (1 + alpha), rounded twice,
    so |rho~ - rho| <= (1 + rho) a + b + 2u <= 2a + b + 2u to first order. Each
    side (kernels, oracle) sums n and k exact squares (a = gamma_n, b = gamma_k);
    every moving-average update m <- beta m + (1 - beta) E keeps the relative
    error of a convex combination of the energies and adds at most 4u. The two
    sides together, with a margin for second-order terms: twice one side."""
    a = gamma(n) + 4 * updates * U
    b = gamma(k) + 4 * updates * U
    return 2.0 * (2 * a + b + 2 * U) * (1 + 1e-6) + 8 * U


def energy_tol(n: int) -> float:
    """Relative bound of one double sum of n exact non-negative terms in any order
    (gamma_n), for comparisons of two such sums: twice that."""
    return 2.0 * gamma(n)


def within_aggregate_tolerance(x: np.ndarray, ref: np.ndarray) -> bool:
    """|x - ref| <= 1e-7 + 1e-6 |ref| elementwise (the float tolerance of the aggregate)."""
    x = x.astype(np.float64)
    r = ref.astype(np.float64)
    return bool(np.all(np.abs(x - r) <= 1e-7 + 1e-6 * np.abs(r)))


def threshold_topk(g, k):
    """Oracle Top-k in O(n) for full-size vectors: (idx, val, e_all, e_kept)."""
    idx, _, _, _ = oracle.topk_by_threshold(g, k)
    e_all, e_kept = oracle.energies(g, idx)
    return idx, g[idx], e_all, e_kept


def oracle_topk_all(s, it, G, topk=None, threads=1):
    """The oracle's Top-k of every device with the extended-precision energy
    references: a list of (idx, val, e_all, e_kept, ref). Optionally on a thread
    pool (the oracle and numpy release the GIL)."""
    fn = topk or oracle.topk
    ks = [oracle.topk_k(s.n, s.ratios[it, j]) for j in range(s.K)]

    def one(j):
        idx, val, e_all, e_kept = fn(G[j], ks[j])
        return idx, val, e_all, e_kept, oracle.energies_extended(G[j], idx)

    if threads <= 1:
        return [one(j) for j in range(s.K)]
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(threads) as ex:
        return list(ex.map(one, range(s.K)))


def check_step(sc, s, it, G, out, w, lr, params_before, params_after, delta=math.inf, topk=None,
               label="", threads=1, mom=None):
    """Compare one fused step against the oracle. `topk(g, k)` returns the oracle's
    (idx, val, e_all, e_kept); defaults to the full-sort oracle. With `mom` =
    (momentum, weight_decay, buf_before, buf_after) the update is momentum SGD
    and (params, buf) of the oracle are returned."""
    n, K = s.n, s.K
    results = oracle_topk_all(s, it, G, topk, threads)
    w_o, gamma_o = oracle.stream_weights(s.rates[it], base_batch=s.base_batch)
    assert same_bits(w_o, w), f"{label}: weights differ"
    lr_o = float(np.float32(s.eta * gamma_o))
    assert lr_o == lr
    energies = out.energies.cpu().numpy()
    compressed = out.compressed.cpu().numpy()
    sets = []
    for j in range(K):
        k = oracle.topk_k(n, s.ratios[it, j])
        idx, val, e_all, e_kept, ref = results[j]
        got_idx = out.idx[j].cpu().numpy()
        got_val = out.val[j].cpu().numpy()
        if not np.array_equal(got_idx, idx):
            bad = np.flatnonzero(got_idx != idx) if got_idx.shape == idx.shape else []
            raise AssertionError(f"{label} device {j}: Top-k indices differ (k={k}, first mismatch "
                                 f"{bad[:5] if len(bad) else 'length'})")
        assert same_bits(got_val, val), f"{label} device {j}: values differ"
        check_energies(f"{label} device {j} (oracle)", e_all, e_kept, ref, n, k)
        check_energies(f"{label} device {j}", energies[2 * j], energies[2 * j + 1], ref, n, k)
        send, rho = oracle.compress_decision(e_all, e_kept, delta)
        if abs(rho - delta) > decision_window(n, k):
            assert bool(compressed[j]) == send, f"{label} device {j}: adaptive decision"
        else:
            send = bool(compressed[j])     # rho within rounding of delta: either decision is correct
        sets.append((idx, val) if send else (None, G[j]))
    dense_o = oracle.aggregate(sets, w_o, n)
    dense = out.dense.cpu().numpy()
    assert within_aggregate_tolerance(dense, dense_o), f"{label}: aggregate outside tolerance"
    assert same_bits(dense, dense_o), f"{label}: aggregate not bit-identical to the oracle"
    if params_before is not None and mom is not None:
        mu, wd, v_before, v_after = mom
        p_o, v_o = oracle.momentum_sgd(params_before, v_before, dense_o, lr_o, mu, wd)
        assert same_bits(v_after, v_o), f"{label}: momentum buffer differs"
        assert same_bits(params_after, p_o), f"{label}: momentum SGD update differs"
        return p_o, v_o
    if params_before is not None:
        p_o = oracle.sgd(params_before, dense_o, lr_o)
        assert same_bits(params_after, p_o), f"{label}: SGD update differs"
        return p_o
    return None


def run_config(sc, config, n=None, K=None, iterations=None, delta=math.inf, with_params=True, topk=None,
               ratio_override=None, threads=1, momentum=None):
    """Run `iterations` fused steps of a workload and check each against the oracle.
    `momentum` = (momentum, weight_decay) runs the momentum-SGD fused step from a
    zero buffer."""
    torch, dev = torch_dev()
    s = workloads.spec(config, n=n, K=K, iterations=iterations)
    if ratio_override is not None:
        s.ratios[:] = np.asarray(ratio_override, dtype=np.float64)
    label = f"C{config} n={s.n} K={s.K}"
    params = workloads.params0(s) if with_params else None
    p_dev = torch.from_numpy(params).to(dev) if with_params else None
    p_ref = params.copy() if with_params else None
    if momentum is not None:
        v_ref = np.zeros(s.n, dtype=np.float32)
        v_dev = torch.zeros(s.n, dtype=torch.float32, device=dev)
    for it in range(s.iterations):
        log(f"  {label} iteration {it}: ratio {s.ratios[it, 0]}")
        G = np.empty((s.K, s.n), dtype=np.float32)
        for j in range(s.K):
            workloads.gradient(s, it, j, out=G[j], k=oracle.topk_k(s.n, s.ratios[it, j]))
        g_dev = torch.from_numpy(G).to(dev)
        w, gamma = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
        lr = float(np.float32(s.eta * gamma))
        if momentum is not None:
            step = sc.FusedStep(g_dev, s.ratios[it], delta=delta, params=p_dev, momentum_buf=v_dev,
                                momentum=momentum[0], weight_decay=momentum[1])
        else:
            step = sc.FusedStep(g_dev, s.ratios[it], delta=delta, params=p_dev)
        out = step.run(w, lr)
        torch.cuda.synchronize()
        p_after = p_dev.cpu().numpy() if with_params else None
        if momentum is not None:
            p_ref, v_ref = check_step(sc, s, it, G, out, w, lr, p_ref, p_after, delta=delta, topk=topk,
                                      label=f"{label} it={it}", threads=threads,
                                      mom=(momentum[0], momentum[1], v_ref, v_dev.cpu().numpy()))
        else:
            p_ref = check_step(sc, s, it, G, out, w, lr, p_ref, p_after, delta=delta, topk=topk,
                               label=f"{label} it={it}", threads=threads)
        del g_dev, step, out, G
    return s
