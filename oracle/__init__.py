"""CPU oracle of the ScaDLES hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path
(``paper_2301_08897_amd``) never imports it, and the two share no code.

The arithmetic lives in ``scadles_oracle.c`` (plain C, double precision,
full sort, serial sums); this module compiles it with gcc and wraps it for
numpy arrays. ``topk_by_threshold`` is a second, O(n) statement of the same
Top-k definition for vectors too long to sort in a test: the k-th largest
magnitude from a library selection routine (``numpy.partition``), then the
definition of the kept set written out.

Paper: Tyagi & Swany, "ScaDLES: Scalable Deep Learning over Streaming data at
the Edge", arXiv 2301.08897. Section, equation and table numbers below refer
to it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "scadles_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()

_u32p = ctypes.POINTER(ctypes.c_uint32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u64p = ctypes.POINTER(ctypes.c_uint64)


def build() -> str:
    """Compile the oracle with gcc (no -ffast-math: IEEE semantics, denormals kept)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", _SRC, "-o", _LIB_PATH, "-lm"]
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
        lib.oracle_topk_k.restype = ctypes.c_uint64
        lib.oracle_topk_k.argtypes = [ctypes.c_uint64, ctypes.c_double]
        lib.oracle_topk.restype = ctypes.c_int
        lib.oracle_topk.argtypes = [_f32p, ctypes.c_uint64, ctypes.c_uint64, _u32p, _f32p,
                                    _f64p, _f64p]
        lib.oracle_topk_layers.restype = ctypes.c_int
        lib.oracle_topk_layers.argtypes = [_f32p, _u64p, ctypes.c_uint32, ctypes.c_double, _u32p, _f32p,
                                           _f64p, _f64p, _u64p]
        lib.oracle_stream_run.restype = ctypes.c_int
        lib.oracle_stream_run.argtypes = [ctypes.c_uint32, _u64p, _u64p, ctypes.c_uint64, ctypes.c_uint64,
                                          ctypes.c_int, ctypes.c_uint64, _u64p, _u64p, _u64p]
        lib.oracle_compress_decision.restype = ctypes.c_int
        lib.oracle_compress_decision.argtypes = [ctypes.c_double, ctypes.c_double,
                                                 ctypes.c_double, _f64p]
        lib.oracle_aggregate.restype = ctypes.c_int
        lib.oracle_aggregate.argtypes = [ctypes.c_uint32, ctypes.c_uint64,
                                         ctypes.POINTER(_u32p), ctypes.POINTER(_f32p),
                                         _u64p, _f32p, _f32p]
        lib.oracle_sgd.restype = None
        lib.oracle_sgd.argtypes = [_f32p, _f32p, ctypes.c_uint64, ctypes.c_float]
        lib.oracle_adaptive_step.restype = ctypes.c_int
        lib.oracle_adaptive_step.argtypes = [_f64p, ctypes.POINTER(ctypes.c_uint64), ctypes.c_double,
                                             ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                             ctypes.c_uint64, ctypes.c_uint64]
        lib.oracle_momentum_sgd.restype = None
        lib.oracle_momentum_sgd.argtypes = [_f32p, _f32p, _f32p, ctypes.c_uint64, ctypes.c_float,
                                            ctypes.c_float, ctypes.c_float]
        lib.oracle_stream_weights.restype = ctypes.c_int
        lib.oracle_stream_weights.argtypes = [_f64p, ctypes.c_uint32, ctypes.c_double,
                                              ctypes.c_double, ctypes.c_double, _f32p, _f64p]
        _lib = lib
        return lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def topk_k(n: int, ratio: float) -> int:
    """k = clamp(floor(ratio * n), 1, n) in double (§V-G); 0 for invalid input."""
    return int(_load().oracle_topk_k(int(n), float(ratio)))


def topk(g: np.ndarray, k: int):
    """Top-k of one gradient by full sort (§III-C, §IV).

    Returns (idx uint32 ascending, val float32, e_all, e_kept)."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    n = g.size
    idx = np.empty(k, dtype=np.uint32)
    val = np.empty(k, dtype=np.float32)
    e_all = ctypes.c_double()
    e_kept = ctypes.c_double()
    rc = _load().oracle_topk(_ptr(g, ctypes.c_float), n, int(k), _ptr(idx, ctypes.c_uint32),
                             _ptr(val, ctypes.c_float), ctypes.byref(e_all),
                             ctypes.byref(e_kept))
    if rc != 0:
        raise ValueError(f"oracle_topk rejected n={n} k={k}")
    return idx, val, e_all.value, e_kept.value


def topk_by_threshold(g: np.ndarray, k: int):
    """Top-k of one gradient in O(n), for full-size vectors (§III-C, §IV).

    The k-th largest magnitude T comes from ``numpy.partition``. Kept set, by
    definition: every entry with |g| > T, plus the lowest-indexed entries with
    |g| == T until k are kept. Returns (idx uint32 ascending, T as float32
    magnitude, count above T, number of ties kept)."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    n = g.size
    if not 1 <= k <= n:
        raise ValueError("k out of range")
    mag = np.abs(g)
    t = np.partition(mag, n - k)[n - k]
    above = mag > t
    c_gt = int(np.count_nonzero(above))
    need = k - c_gt
    ties = np.flatnonzero(mag == t)[:need]
    keep = above
    keep[ties] = True
    idx = np.flatnonzero(keep).astype(np.uint32)
    return idx, np.float32(t), c_gt, need


def layers_k(seg_off, ratio: float) -> int:
    """Entries kept by the per-layer Top-k: the sum over layers of topk_k(layer size, ratio)."""
    off = np.asarray(seg_off, dtype=np.uint64)
    return sum(topk_k(int(off[l + 1] - off[l]), ratio) for l in range(off.size - 1))


def topk_layers(g: np.ndarray, seg_off, ratio: float):
    """Per-layer Top-k (each layer keeps its own top fraction; the per-layer
    reading of §IV) by a full sort of every layer. ``seg_off`` = [0, ..., n],
    layer l being g[seg_off[l]:seg_off[l+1]]. Returns (idx uint32 ascending,
    val float32, e_all, e_kept) of the whole gradient."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    off = np.ascontiguousarray(seg_off, dtype=np.uint64)
    L = off.size - 1
    if L < 1 or int(off[-1]) != g.size:
        raise ValueError("seg_off must run from 0 to g.size")
    k = layers_k(off, ratio)
    idx = np.empty(max(k, 1), dtype=np.uint32)
    val = np.empty(max(k, 1), dtype=np.float32)
    e_all = ctypes.c_double()
    e_kept = ctypes.c_double()
    k_out = ctypes.c_uint64()
    rc = _load().oracle_topk_layers(_ptr(g, ctypes.c_float), _ptr(off, ctypes.c_uint64), L, float(ratio),
                                    _ptr(idx, ctypes.c_uint32), _ptr(val, ctypes.c_float), ctypes.byref(e_all),
                                    ctypes.byref(e_kept), ctypes.byref(k_out))
    if rc != 0 or int(k_out.value) != k:
        raise ValueError(f"oracle_topk_layers rejected L={L} ratio={ratio}")
    return idx[:k], val[:k], e_all.value, e_kept.value


def topk_layers_by_threshold(g: np.ndarray, seg_off, ratio: float):
    """Per-layer Top-k in O(n) for full-size vectors: ``topk_by_threshold`` on
    every layer, indices shifted by the layer's start. Returns (idx, val,
    e_all, e_kept) like ``topk_layers``."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    off = np.asarray(seg_off, dtype=np.uint64)
    parts = []
    for l in range(off.size - 1):
        a, b = int(off[l]), int(off[l + 1])
        i, _, _, _ = topk_by_threshold(g[a:b], topk_k(b - a, ratio))
        parts.append(i.astype(np.uint64) + a)
    idx = np.concatenate(parts).astype(np.uint32)
    e_all, e_kept = energies(g, idx)
    return idx, g[idx], e_all, e_kept


def energies(g: np.ndarray, idx: np.ndarray):
    """The two energies of the adaptive rule (§IV) for a kept set ``idx``:
    (sum over all i of g_i^2, sum over kept i of g_i^2), squares and sums in double."""
    g64 = np.asarray(g, dtype=np.float32).astype(np.float64)
    return float(np.sum(g64 * g64)), float(np.sum(g64[idx] * g64[idx]))


def energies_extended(g: np.ndarray, idx: np.ndarray):
    """The same two energies (§IV) as references for comparing double sums taken
    in other orders: every square of a float is exact in double, and both sums
    run in numpy's long double (64-bit significand on x86-64), so a sum of m
    terms is within (m - 1) * 2^-64 of its exact value relative to it, far below
    the error any order of double additions may have. Returns np.longdouble."""
    if np.finfo(np.longdouble).nmant < 63:
        raise RuntimeError("long double has no 64-bit significand on this host")
    sq = np.square(np.asarray(g, dtype=np.float32), dtype=np.float64)
    return np.sum(sq, dtype=np.longdouble), np.sum(sq[np.asarray(idx, dtype=np.int64)], dtype=np.longdouble)


def compress_decision(e_all: float, e_kept: float, delta: float):
    """Adaptive rule of §IV. Returns (send_topk: bool, energy-loss ratio)."""
    rho = ctypes.c_double()
    r = _load().oracle_compress_decision(float(e_all), float(e_kept), float(delta),
                                         ctypes.byref(rho))
    return bool(r), rho.value


def adaptive_step(state: np.ndarray, counters, e_all: float, e_kept: float, beta: float, delta: float,
                  k: int, n: int) -> bool:
    """Adaptive rule of §IV on the moving average of the energies, with the
    accounting of §V-G. ``state`` (float64[2]) and ``counters`` (uint64[3] or
    None) of one device are updated in place. Returns whether Top-k is sent."""
    if state.dtype != np.float64 or state.size != 2 or not state.flags.c_contiguous:
        raise ValueError("state must be a contiguous float64[2]")
    cp = None
    if counters is not None:
        if counters.dtype != np.uint64 or counters.size != 3 or not counters.flags.c_contiguous:
            raise ValueError("counters must be a contiguous uint64[3]")
        cp = counters.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))
    return bool(_load().oracle_adaptive_step(_ptr(state, ctypes.c_double), cp, float(e_all), float(e_kept),
                                             float(beta), float(delta), int(k), int(n)))


def cnc_ratio(counters) -> float:
    """CNC ratio of §V-G: iterations that sent Top-k over all iterations."""
    return float(counters[0]) / float(counters[1]) if counters[1] else 0.0


def aggregate(sets, weights, n: int) -> np.ndarray:
    """Eqn 4b. ``sets`` is a list of (idx uint32 or None for dense, val float32)."""
    K = len(sets)
    w = np.ascontiguousarray(weights, dtype=np.float32)
    idx_arrs, val_arrs = [], []
    idx_ptrs = (_u32p * K)()
    val_ptrs = (_f32p * K)()
    ks = np.empty(K, dtype=np.uint64)
    for j, (idx, val) in enumerate(sets):
        v = np.ascontiguousarray(val, dtype=np.float32)
        val_arrs.append(v)
        val_ptrs[j] = _ptr(v, ctypes.c_float)
        if idx is None:
            idx_ptrs[j] = _u32p()
            ks[j] = n
        else:
            i = np.ascontiguousarray(idx, dtype=np.uint32)
            idx_arrs.append(i)
            idx_ptrs[j] = _ptr(i, ctypes.c_uint32)
            ks[j] = i.size
    out = np.empty(n, dtype=np.float32)
    rc = _load().oracle_aggregate(K, n, idx_ptrs, val_ptrs, _ptr(ks, ctypes.c_uint64),
                                  _ptr(w, ctypes.c_float), _ptr(out, ctypes.c_float))
    if rc != 0:
        raise ValueError("oracle_aggregate rejected its input")
    return out


def aggregate_at(contrib: np.ndarray, weights) -> np.ndarray:
    """Eqn 4b at selected positions only: ``contrib`` is float32[K, m], device
    j's value at each position (0 where it keeps nothing). Sums in double in
    device order, one rounding to float -- the same arithmetic as
    ``aggregate`` restricted to m positions."""
    contrib = np.asarray(contrib, dtype=np.float32)
    w = np.asarray(weights, dtype=np.float32)
    acc = np.zeros(contrib.shape[1], dtype=np.float64)
    for j in range(contrib.shape[0]):
        acc += np.float64(w[j]) * contrib[j].astype(np.float64)
    return acc.astype(np.float32)


def sgd(params: np.ndarray, grad: np.ndarray, lr: float) -> np.ndarray:
    """Eqn 4c on a copy of ``params``."""
    p = np.array(params, dtype=np.float32, copy=True)
    g = np.ascontiguousarray(grad, dtype=np.float32)
    _load().oracle_sgd(_ptr(p, ctypes.c_float), _ptr(g, ctypes.c_float), p.size,
                       ctypes.c_float(lr))
    return p


def momentum_sgd(params: np.ndarray, buf: np.ndarray, grad: np.ndarray, lr: float, momentum: float,
                 weight_decay: float):
    """Momentum SGD with weight decay (§V training setup) on copies of ``params``
    and the momentum buffer ``buf``; returns (params, buf)."""
    p = np.array(params, dtype=np.float32, copy=True)
    v = np.array(buf, dtype=np.float32, copy=True)
    g = np.ascontiguousarray(grad, dtype=np.float32)
    if not (p.size == v.size == g.size):
        raise ValueError("params, buf and grad must have the same size")
    _load().oracle_momentum_sgd(_ptr(p, ctypes.c_float), _ptr(v, ctypes.c_float), _ptr(g, ctypes.c_float),
                                p.size, ctypes.c_float(lr), ctypes.c_float(momentum),
                                ctypes.c_float(weight_decay))
    return p, v


def stream_weights(rates, b_min: float = 0.0, b_max: float = float("inf"),
                   base_batch: float = 1.0):
    """Eqn 4a weights and the linear-scaling factor gamma (§IV)."""
    r = np.ascontiguousarray(rates, dtype=np.float64)
    K = r.size
    w = np.empty(K, dtype=np.float32)
    gamma = ctypes.c_double()
    rc = _load().oracle_stream_weights(_ptr(r, ctypes.c_double), K, float(b_min), float(b_max),
                                       float(base_batch), _ptr(w, ctypes.c_float),
                                       ctypes.byref(gamma))
    if rc != 0:
        raise ValueError("oracle_stream_weights rejected its input")
    return w, gamma.value


PERSISTENCE, TRUNCATION = 0, 1


def stream_run(rates, iter_us, b_min: int, b_max: int, policy: int, T: int):
    """Streaming buffers of K devices over T iterations (§II-C Eqn 2, §IV buffer
    policies and batch rule). ``rates``: samples/s per device, ``iter_us``:
    iteration time per device in microseconds (integers). Returns (queued
    uint64[T+1, K], batch uint64[T, K], dropped uint64[K])."""
    r = np.ascontiguousarray(rates, dtype=np.uint64)
    t = np.ascontiguousarray(iter_us, dtype=np.uint64)
    K = r.size
    if t.size != K:
        raise ValueError("one iteration time per device")
    queued = np.empty((T + 1, K), dtype=np.uint64)
    batch = np.empty((max(T, 1), K), dtype=np.uint64)
    dropped = np.empty(K, dtype=np.uint64)
    rc = _load().oracle_stream_run(K, _ptr(r, ctypes.c_uint64), _ptr(t, ctypes.c_uint64), int(b_min), int(b_max),
                                   int(policy), int(T), _ptr(queued, ctypes.c_uint64), _ptr(batch, ctypes.c_uint64),
                                   _ptr(dropped, ctypes.c_uint64))
    if rc != 0:
        raise ValueError("oracle_stream_run rejected its input")
    return queued, batch[:T], dropped
