"""Pins of the oracle's momentum SGD with weight decay (the optimizer of the
paper's evaluation, §V training setup, applied after the aggregation of Eqn
4b): reductions to Eqn 4c, a library implementation of the same algorithm,
and closed forms."""
from fractions import Fraction

import numpy as np
import pytest


def _ulp(x):
    return np.spacing(np.abs(np.asarray(x, dtype=np.float32))).astype(np.float64)


def test_no_momentum_no_decay_is_eqn4c(orc):
    rng = np.random.default_rng(1)
    p = rng.standard_normal(257).astype(np.float32)
    v = rng.standard_normal(257).astype(np.float32)      # ignored when momentum is 0
    g = rng.standard_normal(257).astype(np.float32)
    q, w = orc.momentum_sgd(p, v, g, 0.03, 0.0, 0.0)
    assert np.array_equal(q.view(np.uint32), orc.sgd(p, g, 0.03).view(np.uint32))
    assert np.array_equal(w.view(np.uint32), g.view(np.uint32))


def test_first_step_from_zero_buffer(orc):
    # zero buffer: v = g + wd * w, then the plain step with v (Eqn 4c, pinned on its own)
    rng = np.random.default_rng(2)
    p = rng.standard_normal(200).astype(np.float32)
    g = rng.standard_normal(200).astype(np.float32)
    wd, lr = np.float32(5e-4), np.float32(0.01)
    q, v = orc.momentum_sgd(p, np.zeros_like(p), g, float(lr), 0.9, float(wd))
    for i in range(200):
        exact = Fraction(float(g[i])) + Fraction(float(wd)) * Fraction(float(p[i]))
        assert abs(Fraction(float(v[i])) - exact) <= Fraction(float(np.spacing(np.float32(abs(float(exact))))))
    assert np.array_equal(q.view(np.uint32), orc.sgd(p, v, float(lr)).view(np.uint32))


@pytest.mark.parametrize("mu,wd", [(0.9, 1e-4), (0.9, 5e-4), (0.5, 0.0), (0.0, 1e-2)])
def test_matches_library_sgd(orc, mu, wd):
    # torch.optim.SGD (no dampening, no Nesterov) in float64 on the CPU: the same
    # published algorithm from an independent implementation; the oracle stores
    # float32, so the two agree to a few float32 rounding steps per iteration.
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    n, steps, lr = 1000, 6, 0.05
    p0 = rng.standard_normal(n).astype(np.float32)
    w = torch.tensor(p0.astype(np.float64), requires_grad=True)
    # the hyperparameters as the float32 values the oracle receives
    f32 = lambda x: float(np.float32(x))
    opt = torch.optim.SGD([w], lr=f32(lr), momentum=f32(mu), weight_decay=f32(wd), dampening=0.0, nesterov=False)
    p, v = p0.copy(), np.zeros(n, dtype=np.float32)
    # each step rounds v and w to float once: the errors stay within a few
    # float ulps of the largest magnitudes each element has taken so far
    pmax, vmax = np.abs(p0).astype(np.float64), np.zeros(n)
    for t in range(steps):
        g = rng.standard_normal(n).astype(np.float32)
        w.grad = torch.tensor(g.astype(np.float64))
        opt.step()
        p, v = orc.momentum_sgd(p, v, g, np.float32(lr), np.float32(mu), np.float32(wd))
        ref = w.detach().numpy()
        pmax, vmax = np.maximum(pmax, np.abs(ref)), np.maximum(vmax, np.abs(v))
        tol_v = 2.0 * (t + 1) * _ulp(vmax)
        tol_p = 2.0 * (t + 1) * (_ulp(pmax) + lr * _ulp(vmax))
        assert np.all(np.abs(p.astype(np.float64) - ref) <= tol_p), t
        if mu > 0:
            buf = opt.state[w]["momentum_buffer"].numpy()
            assert np.all(np.abs(v.astype(np.float64) - buf) <= tol_v), t
        # a misplaced term (decay after the momentum, lr inside the buffer) is far outside
        assert np.max(np.abs(p.astype(np.float64) - ref)) < 1e-5


def test_constant_gradient_geometric_series(orc):
    # wd = 0, constant g from a zero buffer: v_T = g (1 - mu^T) / (1 - mu),
    # w_T = w_0 - lr * sum_{t=1..T} v_t
    mu, lr, T = 0.9, 0.01, 20
    g = np.array([1.0, -0.75, 3.0e-3, 2.5], dtype=np.float32)
    p0 = np.array([0.5, -1.0, 2.0, 0.0], dtype=np.float32)
    p, v = p0.copy(), np.zeros(4, dtype=np.float32)
    vs = []
    for _ in range(T):
        p, v = orc.momentum_sgd(p, v, g, lr, mu, 0.0)
        vs.append(v.astype(np.float64))
    m = np.float64(np.float32(mu))
    for t, vt in enumerate(vs, start=1):
        closed = g.astype(np.float64) * (1 - m ** t) / (1 - m)
        assert np.all(np.abs(vt - closed) <= 2 * t * _ulp(closed))
    closed_p = p0.astype(np.float64) - np.float64(np.float32(lr)) * np.sum(vs, axis=0)
    assert np.all(np.abs(p.astype(np.float64) - closed_p) <= 4 * T * (_ulp(closed_p) + _ulp(p0)))


def test_weight_decay_alone_shrinks_geometrically(orc):
    # mu = 0, g = 0: w_T = w_0 (1 - lr wd)^T
    lr, wd, T = 0.1, 0.05, 30
    p0 = np.array([1.0, -3.0, 1e-3, 7.5], dtype=np.float32)
    p, v = p0.copy(), np.zeros(4, dtype=np.float32)
    for _ in range(T):
        p, v = orc.momentum_sgd(p, v, np.zeros(4, dtype=np.float32), lr, 0.0, wd)
    f = 1.0 - np.float64(np.float32(lr)) * np.float64(np.float32(wd))
    closed = p0.astype(np.float64) * f ** T
    assert np.all(np.abs(p.astype(np.float64) - closed) <= 2 * T * _ulp(closed))
