"""Seeded synthetic workloads for the ScaDLES hot path.

Shared by the tests, the benchmark and the oracle side. It draws random
numbers and nothing else: no ranking, selection, weighting or update of the
method happens here. Streaming rates (batch sizes) are returned raw; turning
them into aggregation weights (Eqn 4a) is the method's job.

The five workloads stand in for the gradients of the paper's models (Table
III: ResNet152 with 60.2M and VGG19 with 143.7M parameters, trained on
CIFAR10/100, which are not used): flat fp32 vectors with the models' sizes and
a per-layer scale structure (segments with log-uniform standard deviations).

Bulk values come from ``gen.c`` (Philox4x32-10, Box-Muller, inverse-CDF
Laplace), compiled with gcc and OpenMP.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB_PATH = os.path.join(_HERE, "libgen.so")
_lib = None
_lock = threading.Lock()

SEED_BASE = 230108897
# Philox key tags separating independent draws of one config.
TAG_GRAD, TAG_MARK, TAG_PARAMS, TAG_SEG, TAG_SIGMA, TAG_RATES, TAG_SPLIT = 1, 2, 3, 4, 5, 6, 7


def build() -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
           _SRC, "-o", _LIB_PATH, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        u64p = ctypes.POINTER(ctypes.c_uint64)
        f64p = ctypes.POINTER(ctypes.c_double)
        f32p = ctypes.POINTER(ctypes.c_float)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        lib.gen_philox4x32_10.argtypes = [u32p, u32p, u32p]
        lib.gen_philox4x32_10.restype = None
        lib.gen_uniforms.argtypes = [f64p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                     ctypes.c_uint32, ctypes.c_uint64]
        lib.gen_uniforms.restype = None
        lib.gen_fill.argtypes = [f32p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                 ctypes.c_uint32, ctypes.c_uint32, u64p, f64p, ctypes.c_uint32,
                                 ctypes.c_int, ctypes.c_int]
        lib.gen_fill.restype = None
        lib.gen_mark.argtypes = [f32p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                 ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int, ctypes.c_double,
                                 ctypes.c_double, ctypes.c_float, ctypes.c_int]
        lib.gen_mark.restype = None
        _lib = lib
        return lib


def threads() -> int:
    """Worker threads for bulk generation: OMP_NUM_THREADS if set, else the CPUs
    this process may use, at most 16."""
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit() and int(env) > 0:
        return int(env)
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(16, os.cpu_count() or 1))


def philox4x32_10(ctr, key):
    """Raw Philox4x32-10 block (for the generator's known-answer test)."""
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    _load().gen_philox4x32_10(c, k, o)
    return tuple(int(x) for x in o)


class UniformStream:
    """Sequential (0, 1) uniforms from Philox, for small host-side draws."""

    def __init__(self, seed: int, tag: int, stream: int = 0, block: int = 4096):
        self.seed, self.tag, self.stream, self.block = seed, tag, stream, block
        self.offset = 0
        self.buf = np.empty(0)
        self.pos = 0

    def next(self) -> float:
        if self.pos >= self.buf.size:
            self.buf = np.empty(self.block, dtype=np.float64)
            _load().gen_uniforms(self.buf.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                 self.block, self.seed, self.tag, self.stream, self.offset)
            self.offset += self.block
            self.pos = 0
        u = float(self.buf[self.pos])
        self.pos += 1
        return u

    def normal(self) -> float:
        a, b = self.next(), self.next()
        return math.sqrt(-2.0 * math.log(a)) * math.cos(2.0 * math.pi * b)

    def exponential(self) -> float:
        return -math.log(self.next())

    def poisson(self, mu: float) -> int:
        """Count of rate-mu exponential arrivals in [0, 1]."""
        t, count = 0.0, 0
        while True:
            t += self.exponential() / mu
            if t > 1.0:
                return count
            count += 1

    def gamma(self, a: float) -> float:
        """Marsaglia & Tsang (2000); shape < 1 via Gamma(a+1) * U^(1/a)."""
        if a < 1.0:
            return self.gamma(a + 1.0) * self.next() ** (1.0 / a)
        d = a - 1.0 / 3.0
        c = 1.0 / math.sqrt(9.0 * d)
        while True:
            x = self.normal()
            v = (1.0 + c * x) ** 3
            if v <= 0.0:
                continue
            if math.log(self.next()) < 0.5 * x * x + d - d * v + d * math.log(v):
                return d * v


def _largest_remainder(weights: np.ndarray, total: int) -> np.ndarray:
    """Integer sizes proportional to weights summing to total, each >= 1."""
    w = np.asarray(weights, dtype=np.float64)
    exact = w / w.sum() * total
    sizes = np.floor(exact).astype(np.int64)
    rem = total - int(sizes.sum())
    order = np.lexsort((np.arange(w.size), -(exact - sizes)))
    sizes[order[:rem]] += 1
    for i in np.flatnonzero(sizes == 0):
        j = int(np.argmax(sizes))
        sizes[j] -= 1
        sizes[i] += 1
    return sizes


@dataclass
class Spec:
    """One workload: K devices of n fp32 gradient elements over `iterations`."""
    config: int
    name: str
    K: int
    n: int
    iterations: int
    dist: int                       # 0 normal, 1 Laplace
    seg_end: np.ndarray             # uint64[L], cumulative segment ends
    seg_sigma: np.ndarray           # float64[L]
    ratios: np.ndarray              # float64[iterations, K]
    rates: np.ndarray               # float64[iterations, K]: batch sizes / stream rates
    eta: float                      # base learning rate
    base_batch: float               # B of the linear scaling rule
    p_zero: float = 0.0
    p_tie: float = 0.0
    params_sigma: float = 0.05
    seed: int = 0
    notes: dict = field(default_factory=dict)



# Full-size shapes of the five workloads.
FULL = {
    1: dict(K=4, n=1_048_576),
    2: dict(K=8, n=11_173_962),
    3: dict(K=16, n=25_557_032),
    4: dict(K=16, n=60_192_808),
    5: dict(K=32, n=143_667_240),
}
NAMES = {
    1: "C1: K=4 x n=1,048,576, N(0,s_l) 8 segments, ratio 0.01",
    2: "C2: K=8 x n=11,173,962 (ResNet-18-sized), 62 segments, ratio 0.01",
    3: "C3: K=16 x n=25,557,032 (ResNet-50-sized), Laplace, ratios 0.1/0.01/0.001",
    4: "C4: K=16 x n=60,192,808 (ResNet-152-sized), 5% zeros + 1% ties, ratio 0.001",
    5: "C5: K=32 x n=143,667,240 (VGG-19-sized), ratio 0.01, 10 iterations",
}


def spec(config: int, n: int | None = None, K: int | None = None,
         iterations: int | None = None) -> Spec:
    """The workload of `config` (1..5), optionally shrunk to n elements and K devices
    with the same recipe (segment structure rescaled to n)."""
    full = FULL[config]
    n = int(n or full["n"])
    K = int(K or full["K"])
    seed = SEED_BASE + config
    seg_u = UniformStream(seed, TAG_SEG)
    sig_u = UniformStream(seed, TAG_SIGMA)

    if config == 1:
        L, lo, hi, dist = 8, -4.0, -1.0, 0
        sizes = _largest_remainder(np.ones(L), n)
    elif config in (2, 3, 4):
        L = {2: 62, 3: 161, 4: 467}[config]
        lo, hi = (-5.0, -1.0)
        dist = 1 if config == 3 else 0
        raw = np.array([math.exp(math.log(64.0) + seg_u.next() * (math.log(2.4e6) - math.log(64.0)))
                        for _ in range(L)])
        sizes = _largest_remainder(raw, n)
    else:
        L, lo, hi, dist = 38, -6.0, -1.0, 0
        big = int(math.floor(0.85 * n))
        su = UniformStream(seed, TAG_SPLIT)     # Dirichlet(1,1,1) split of 85% of n
        split = np.array([su.exponential() for _ in range(3)])
        raw = np.array([math.exp(math.log(64.0) + seg_u.next() * (math.log(2.4e6) - math.log(64.0)))
                        for _ in range(L - 3)])
        sizes = np.concatenate([_largest_remainder(raw, n - big),
                                _largest_remainder(split, big)])
    if n < L:
        raise ValueError(f"n={n} is smaller than the {L} segments of config {config}")
    sigma = np.array([10.0 ** (lo + sig_u.next() * (hi - lo)) for _ in range(L)])
    seg_end = np.cumsum(sizes).astype(np.uint64)

    iters = {1: 1, 2: 1, 3: 3, 4: 1, 5: 10}[config]
    if iterations is not None:
        iters = int(iterations)
    ratio_of_iter = {3: [0.1, 0.01, 0.001]}.get(config)
    base_ratio = {1: 0.01, 2: 0.01, 4: 0.001, 5: 0.01}.get(config, 0.01)
    ratios = np.empty((iters, K))
    for t in range(iters):
        ratios[t, :] = ratio_of_iter[t % 3] if ratio_of_iter else base_ratio

    rates = np.empty((iters, K))
    for t in range(iters):
        ru = UniformStream(seed, TAG_RATES, stream=t)
        for j in range(K):
            if config == 1:
                rates[t, j] = [16, 32, 48, 64][j % 4]
            elif config == 2:
                rates[t, j] = min(128, max(1, ru.poisson(32.0)))
            elif config == 3:
                rates[t, j] = ru.gamma(0.5)          # Dirichlet(0.5) after normalisation
            elif config == 4:
                rates[t, j] = 8 + min(248, int(ru.next() * 249))
            else:
                mu = 4.0 * 128.0 ** (j / 31.0) if K > 1 else 4.0
                rates[t, j] = ru.poisson(mu)
        if rates[t].sum() == 0:
            rates[t, 0] = 1.0

    eta = {1: 0.01, 2: 0.1, 3: 0.1, 4: 0.1, 5: 0.01}[config]
    s = Spec(config=config, name=NAMES[config], K=K, n=n, iterations=iters, dist=dist,
             seg_end=seg_end, seg_sigma=sigma, ratios=ratios, rates=rates, eta=eta,
             base_batch=64.0 * K, seed=seed)
    if config == 4:
        s.p_zero, s.p_tie = 0.05, 0.01
    return s


def gradient(s: Spec, it: int, j: int, out: np.ndarray | None = None,
             nthreads: int | None = None, k: int | None = None) -> np.ndarray:
    """Device j's gradient at iteration `it` (float32[n]). A workload with tied
    magnitudes (s.p_tie > 0) places them at the ceil(k/2)-th largest magnitude,
    so that they straddle the Top-k boundary: its caller passes k, the number
    of entries kept at this device's ratio (this module holds no k rule)."""
    if s.p_tie > 0.0 and k is None:
        raise ValueError(f"{s.name}: pass k (the kept count at ratio {s.ratios[it, j]}) to place the ties")
    lib = _load()
    if out is None:
        out = np.empty(s.n, dtype=np.float32)
    nt = nthreads or threads()
    seg_end = np.ascontiguousarray(s.seg_end, dtype=np.uint64)
    sig = np.ascontiguousarray(s.seg_sigma, dtype=np.float64)
    f32p = ctypes.POINTER(ctypes.c_float)
    ptr = out.ctypes.data_as(f32p)
    lib.gen_fill(ptr, s.n, s.seed, TAG_GRAD, j, it,
                 seg_end.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                 sig.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), sig.size, s.dist, nt)
    if s.p_zero > 0.0 or s.p_tie > 0.0:
        lib.gen_mark(ptr, s.n, s.seed, TAG_MARK, j, it, 0, s.p_zero, s.p_tie, 0.0, nt)
        if s.p_tie > 0.0:
            # Tie magnitude m*: the ceil(k/2)-th largest |g| before the ties go in,
            # so that the tied block straddles the Top-k boundary.
            r = (int(k) + 1) // 2
            mag = np.abs(out)
            m_star = float(np.partition(mag, s.n - r)[s.n - r])
            del mag
            lib.gen_mark(ptr, s.n, s.seed, TAG_MARK, j, it, 1, s.p_zero, s.p_tie, m_star, nt)
    return out


def params0(s: Spec, out: np.ndarray | None = None, nthreads: int | None = None) -> np.ndarray:
    """Initial parameters ~ N(0, 0.05^2) (float32[n])."""
    lib = _load()
    if out is None:
        out = np.empty(s.n, dtype=np.float32)
    seg_end = np.array([s.n], dtype=np.uint64)
    sig = np.array([s.params_sigma], dtype=np.float64)
    lib.gen_fill(out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), s.n, s.seed, TAG_PARAMS,
                 0, 0, seg_end.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                 sig.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), 1, 0,
                 nthreads or threads())
    return out
