"""The C-ABI library: it loads, exports every declared symbol, and validates
arguments on the host (no GPU needed for any of these)."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scadles.h")


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    return sc


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(scadles_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_hot_path():
    names = declared_functions()
    for required in ("scadles_topk_select", "scadles_weighted_aggregate", "scadles_apply_sgd",
                     "scadles_step_fused", "scadles_stream_weights", "scadles_topk_k"):
        assert required in names


def test_every_declared_symbol_is_exported(sc):
    lib = ctypes.CDLL(sc.library_path())
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} is declared in scadles.h but not exported"


def test_k_rule_matches_oracle(sc, orc):
    rng = np.random.default_rng(0)
    cases = [(1_048_576, 0.01), (11_173_962, 0.01), (25_557_032, 0.1), (25_557_032, 0.001),
             (60_192_808, 0.001), (143_667_240, 0.01), (1, 1.0), (100, 0.07),
             (100, math.nextafter(0.07, 0)), (2**32 - 1, 0.5), (2**32, 0.5), (0, 0.5), (10, 0.0),
             (10, float("nan")), (10, 1.0000001)]
    cases += [(int(rng.integers(1, 10**9)), float(rng.random())) for _ in range(200)]
    for n, r in cases:
        assert sc.topk_k(n, r) == orc.topk_k(n, r), (n, r)


def test_stream_weights_match_oracle_bitwise(sc, orc, wl):
    for c in (1, 2, 3, 4, 5):
        s = wl.spec(c)
        for it in range(s.iterations):
            w, g = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
            wo, go = orc.stream_weights(s.rates[it], base_batch=s.base_batch)
            assert np.array_equal(w.view(np.uint32), wo.view(np.uint32))
            assert g == go
    w, g = sc.stream_weights([2.0, 8.0, 500.0, 4000.0], b_min=8, b_max=1024, base_batch=64)
    wo, go = orc.stream_weights([2.0, 8.0, 500.0, 4000.0], b_min=8, b_max=1024, base_batch=64)
    assert np.array_equal(w, wo) and g == go


def test_stream_weights_rejects(sc):
    for rates in ([0.0, 0.0], [1.0, -1.0], [1.0, float("nan")], [float("inf")]):
        with pytest.raises(sc.ScadlesError) as e:
            sc.stream_weights(rates)
        assert e.value.code == 1
    with pytest.raises(sc.ScadlesError):
        sc.stream_weights([1.0], b_min=5, b_max=2)


def test_host_validation_before_any_launch(sc):
    """Invalid calls return a status and launch nothing (no GPU is touched)."""
    E = {"inval": 1, "ws": 2}
    assert sc._topk_select(None, 10, 0.5, 16, 16, None, None, 0, None) == E["inval"]
    assert sc._topk_select(16, 0, 0.5, 16, 16, None, None, 0, None) == E["inval"]
    assert sc._topk_select(16, 2**32, 0.5, 16, 16, None, None, 0, None) == E["inval"]
    assert sc._topk_select(16, 10, 0.0, 16, 16, None, None, 0, None) == E["inval"]
    assert sc._topk_select(18, 10, 0.5, 16, 16, None, None, 0, None) == E["inval"]   # misaligned grad
    assert sc._topk_select(16, 10, 0.5, 16, 16, None, None, 0, None) == E["ws"]
    assert sc._topk_select(16, 10, 0.5, 16, 16, None, 4096 + 8, 1 << 20, None) == E["ws"]  # misaligned ws
    assert sc._topk_select(16, 10, 0.5, 16, 16, None, 4096, 16, None) == E["ws"]       # too small
    assert sc._apply_sgd(None, 16, 10, 0.1, None) == E["inval"]
    assert sc._apply_sgd(16, 16, 10, 0.1, None) == E["inval"]                          # aliasing
    assert sc._apply_sgd(16, 4096, 10, float("nan"), None) == E["inval"]
    sets = (sc.Sparse * 2)(sc.Sparse(16, 16, 3), sc.Sparse(16, 16, 3))
    w = (ctypes.c_float * 2)(0.5, 0.5)
    assert sc._weighted_aggregate(sets, w, 0, 10, 16, 4096, 1 << 20, None) == E["inval"]   # K = 0
    assert sc._weighted_aggregate(sets, w, 65, 10, 16, 4096, 1 << 20, None) == E["inval"]  # K > 64
    bad = (ctypes.c_float * 2)(0.6, 0.6)
    assert sc._weighted_aggregate(sets, bad, 2, 10, 16, 4096, 1 << 20, None) == E["inval"]  # sum != 1
    neg = (ctypes.c_float * 2)(1.5, -0.5)
    assert sc._weighted_aggregate(sets, neg, 2, 10, 16, 4096, 1 << 20, None) == E["inval"]
    dense_bad = (sc.Sparse * 2)(sc.Sparse(None, 16, 3), sc.Sparse(16, 16, 3))
    assert sc._weighted_aggregate(dense_bad, w, 2, 10, 16, 4096, 1 << 20, None) == E["inval"]
    over = (sc.Sparse * 2)(sc.Sparse(16, 16, 11), sc.Sparse(16, 16, 3))
    assert sc._weighted_aggregate(over, w, 2, 10, 16, 4096, 1 << 20, None) == E["inval"]
    assert sc._weighted_aggregate(sets, w, 2, 10, 16, 4096, 8, None) == E["ws"]
    grads = (ctypes.c_void_p * 2)(16, 32)
    ratios = (ctypes.c_double * 2)(0.1, 0.1)
    outs = (ctypes.c_void_p * 2)(16, 32)
    assert sc._step_fused(grads, 2, 1000, ratios, -1.0, w, outs, outs, 16, None, None, None, 0.0,
                          4096, 1 << 30, None) == E["inval"]                              # delta < 0
    assert sc._step_fused(grads, 2, 1000, ratios, float("nan"), w, outs, outs, 16, None, None, None,
                          0.0, 4096, 1 << 30, None) == E["inval"]
    bad_r = (ctypes.c_double * 2)(0.1, 1.5)
    assert sc._step_fused(grads, 2, 1000, bad_r, math.inf, w, outs, outs, 16, None, None, None, 0.0,
                          4096, 1 << 30, None) == E["inval"]
    assert sc._step_fused(grads, 2, 1000, ratios, math.inf, w, outs, outs, 16, None, None, None, 0.0,
                          4096, 64, None) == E["ws"]
    assert sc._set_option(b"no_such_option", 1) == E["inval"]
    assert b"no_such_option" in sc._last_error()
    # the per-layer order of the long layers: 0, 1 (default) or 2
    assert sc._set_option(b"layer_order", 3) == E["inval"]
    assert sc._set_option(b"layer_order", -1) == E["inval"]
    for v in (0, 2, 1):
        assert sc._set_option(b"layer_order", v) == 0


def test_momentum_validation_before_any_launch(sc):
    """Invalid momentum-SGD calls return EINVAL and launch nothing."""
    inval = 1
    f = sc._apply_momentum_sgd
    assert f(None, 4096, 8192, 10, 0.1, 0.9, 0.0, None) == inval                 # NULL params
    assert f(16, None, 8192, 10, 0.1, 0.9, 0.0, None) == inval                   # NULL buffer
    assert f(16, 4096, 8192, 0, 0.1, 0.9, 0.0, None) == inval                    # n = 0
    assert f(20, 4096, 8192, 10, 0.1, 0.9, 0.0, None) == inval                   # misaligned
    assert f(16, 16, 8192, 10, 0.1, 0.9, 0.0, None) == inval                     # params is the buffer
    assert f(16, 4096, 16, 10, 0.1, 0.9, 0.0, None) == inval                     # grad aliases params
    assert f(16, 4096, 8192, 10, 0.1, float("inf"), 0.0, None) == inval          # momentum not finite
    assert f(16, 4096, 8192, 10, 0.1, 0.9, float("nan"), None) == inval          # decay not finite
    grads = (ctypes.c_void_p * 2)(16, 32)
    ratios = (ctypes.c_double * 2)(0.1, 0.1)
    outs = (ctypes.c_void_p * 2)(16, 32)
    w = (ctypes.c_float * 2)(0.5, 0.5)

    def ex(params, opts):
        return sc._step_fused_ex(grads, 2, 1000, ratios, math.inf, w, outs, outs, 16, None, None, params, 0.1,
                                 ctypes.byref(opts) if opts is not None else None, 4096, 1 << 30, None)

    O = sc.StepOptions
    assert ex(8192, None) == inval                                            # no options
    assert ex(None, O(4096, 0.9, 0.0, None, 0.0, None)) == inval              # momentum without params
    assert ex(8192, O(8192, 0.9, 0.0, None, 0.0, None)) == inval              # buffer is params
    assert ex(8192, O(16, 0.9, 0.0, None, 0.0, None)) == inval                # buffer is dense
    assert ex(8192, O(65536, float("nan"), 0.0, None, 0.0, None)) == inval    # momentum not finite
    assert ex(8192, O(None, 0.0, 0.0, 65536, 1.0, None)) == inval             # beta outside [0, 1)
    assert ex(8192, O(None, 0.0, 0.0, 65536, -0.5, None)) == inval
    assert ex(8192, O(None, 0.0, 0.0, 65537, 0.5, None)) == inval             # misaligned ewma
    assert ex(8192, O(None, 0.0, 0.0, None, 0.0, 65539)) == inval             # misaligned counters


def test_workspace_queries(sc):
    assert sc.workspace_bytes(1, 0, [0.5]) == 0
    assert sc.workspace_bytes(65, 100, [0.5] * 65) == 0
    assert sc.workspace_bytes(2, 100, [0.5, 2.0]) == 0
    K, n = 32, 143_667_240
    big = sc.workspace_bytes(K, n, [0.01] * K)
    # per-wave candidate slots take one byte per gradient element; the candidate
    # lists and the rest are a few k per device
    assert 0 < big < K * n + 2 * 1024**3
    assert sc.aggregate_workspace_bytes(0, 10) == 0
    assert sc.aggregate_workspace_bytes(4, 1 << 20) > 0


def test_layers_validation_before_any_launch(sc):
    """Invalid per-layer selections return a status and launch nothing."""
    inval, ws = 1, 2
    grads = (ctypes.c_void_p * 2)(16, 32)
    idx = (ctypes.c_void_p * 2)(4096, 8192)
    val = (ctypes.c_void_p * 2)(12288, 16384)
    ratios = (ctypes.c_double * 2)(0.1, 0.1)

    def call(off, r=ratios, K=2, g=grads, ws_bytes=1 << 30):
        arr = (ctypes.c_uint64 * len(off))(*off)
        return sc._topk_select_layers(g, K, arr, len(off) - 1, r, idx, val, None, 65536, ws_bytes, None)

    assert call([1, 10]) == inval                                   # does not start at 0
    assert call([0, 5, 5, 10]) == inval                             # empty layer
    assert call([0, 6, 5, 10]) == inval                             # out of order
    assert call([0, 2**32]) == inval                                # n too large
    assert call([0]) == inval                                       # no layer
    assert call([0, 10], r=(ctypes.c_double * 2)(0.1, 0.0)) == inval
    assert call([0, 10], K=0) == inval
    assert call([0, 10], g=(ctypes.c_void_p * 2)(18, 32)) == inval  # misaligned gradient
    assert call([0, 5, 10], ws_bytes=64) == ws
    assert sc._topk_select_layers(grads, 2, None, 1, ratios, idx, val, None, 65536, 1 << 30, None) == inval
    few = (ctypes.c_uint64 * 2)(0, 10)       # more than 2^24 layers is rejected before seg_off is read
    assert sc._topk_select_layers(grads, 2, few, (1 << 24) + 1, ratios, idx, val, None, 65536, 1 << 30,
                                  None) == inval
    assert sc._layers_k(few, (1 << 24) + 1, 0.5) == 0


def test_layers_queries(sc, orc):
    for off, r in (([0, 4, 10], 0.3), ([0, 64, 1064, 1101, 5101, 5102], 0.01), ([0, 10], 1.0),
                   ([0, 1, 2, 3], 0.5), ([0, 100, 10**6, 143_667_240], 0.01)):
        assert sc.layers_k(off, r) == orc.layers_k(off, r)
    assert sc.layers_k([0, 5, 5, 10], 0.5) == 0
    assert sc.layers_k([1, 10], 0.5) == 0
    assert sc.layers_k([0, 10], 0.0) == 0
    off = [0, 1000, 2_000_000, 2_000_100]
    need = sc.layers_workspace_bytes(3, off, [0.01] * 3)
    assert need >= sc.workspace_bytes(3, 1_999_000, [0.01] * 3) > 0
    assert sc.layers_workspace_bytes(3, [0, 5, 5], [0.01] * 3) == 0


def test_fused_layers_validation_before_any_launch(sc):
    """Invalid per-layer fused steps return EINVAL / EWORKSPACE and launch nothing."""
    inval, ws = 1, 2
    grads = (ctypes.c_void_p * 2)(16, 32)
    outs = (ctypes.c_void_p * 2)(4096, 8192)
    ratios = (ctypes.c_double * 2)(0.1, 0.1)
    w = (ctypes.c_float * 2)(0.5, 0.5)

    def call(off, delta=math.inf, weights=w, dense=1 << 20, ws_bytes=1 << 30, params=None):
        arr = (ctypes.c_uint64 * len(off))(*off)
        return sc._step_fused_layers(grads, 2, arr, len(off) - 1, ratios, delta, weights, outs, outs, dense, None,
                                     None, params, 0.1, None, 65536, ws_bytes, None)

    assert call([0, 5, 5, 10]) == inval                                   # empty layer
    assert call([0, 10], delta=-1.0) == inval
    assert call([0, 10], weights=(ctypes.c_float * 2)(0.7, 0.7)) == inval  # weights do not sum to 1
    assert call([0, 10], dense=(1 << 20) + 4) == inval                    # misaligned dense
    assert call([0, 10], params=(1 << 21) + 8) == inval                   # misaligned params
    assert call([0, 4, 10], ws_bytes=64) == ws
    O = sc.StepOptions
    arr = (ctypes.c_uint64 * 2)(0, 10)
    bad = O(None, 0.0, 0.0, 65536, 1.5, None)                             # beta outside [0, 1)
    assert sc._step_fused_layers(grads, 2, arr, 1, ratios, math.inf, w, outs, outs, 1 << 20, None, None, None,
                                 0.1, ctypes.byref(bad), 65536, 1 << 30, None) == inval
    need = sc._step_layers_ws_bytes(2, arr, 1, ratios)
    assert need >= sc.layers_workspace_bytes(2, [0, 10], [0.1, 0.1]) > 0


def test_layer_workspace_sizes(sc):
    import numpy as np
    rng = np.random.default_rng(3)
    for _ in range(20):
        L = int(rng.integers(1, 50))
        sizes = rng.integers(1, 3_000_000, L)
        off = [0] + np.cumsum(sizes).tolist()
        K = int(rng.integers(1, 65))
        ratios = [float(r) for r in rng.choice([0.001, 0.01, 0.1, 1.0], K)]
        sel = sc.layers_workspace_bytes(K, off, ratios)
        arr = (ctypes.c_uint64 * len(off))(*off)
        rr = (ctypes.c_double * K)(*ratios)
        step = int(sc._step_layers_ws_bytes(K, arr, L, rr))
        assert sel > 0 and step > sel
        # at least two selection regions of the longest layer
        assert sel >= 2 * sc.workspace_bytes(K, int(max(sizes)), ratios)
        # more devices never need less
        if K < 64:
            assert sc.layers_workspace_bytes(K + 1, off, ratios + [0.01]) >= sel


def test_noalloc_select_rejects_oversize_on_the_host(sc):
    """The allocation-free selection refuses, before touching the GPU, a size
    whose workspace exceeds the static scratch (the pointers are never used)."""
    lib = ctypes.CDLL(sc.library_path())
    f = lib.scadles_topk_select_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p]
    fake = 1 << 20                                  # aligned, never dereferenced on the host
    n = 143_667_240
    assert sc.workspace_bytes(1, n, [0.1]) > sc.NOALLOC_SCRATCH_BYTES
    assert f(fake, n, 0.1, fake, fake, None, None) == 2          # SCADLES_EWORKSPACE
    err = lib.scadles_last_error
    err.restype = ctypes.c_char_p
    assert b"scratch" in err()
    assert f(None, n, 0.01, fake, fake, None, None) == 1          # SCADLES_EINVAL
    assert f(fake, n, 0.0, fake, fake, None, None) == 1
    assert sc.workspace_bytes(1, n, [0.01]) <= sc.NOALLOC_SCRATCH_BYTES
