"""ScaDLES hot path on MI355X: Top-k sparsification, streaming-rate-weighted
aggregation and SGD in hand-written HIP kernels for gfx950.

This package is a thin ctypes binding over ``libscadles.so`` (C ABI in
``include/scadles.h``). It only marshals arguments: every step runs in the HIP
kernels. PyTorch supplies device memory and the stream. Importing fails
loudly when the library has not been built (``__graft_entry__.build()``).
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libscadles.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first "
                      "(there is no fallback implementation)")

# torch bundles its own HIP runtime under the same soname as the system one.
# Loading torch first makes libscadles bind to that runtime, so the process has
# exactly one HIP/HSA runtime (two would each try to own the GPU).
import torch as _torch_for_runtime  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

MAX_DEVICES = 64
NOALLOC_SCRATCH_BYTES = 128 << 20      # SCADLES_NOALLOC_SCRATCH_BYTES
PROFILE_STAGES = 5
STAGE_NAMES = ("bracket", "main_select", "post_select", "aggregate", "total")

_vp = ctypes.c_void_p
_u64 = ctypes.c_uint64
_u32 = ctypes.c_uint32


class Sparse(ctypes.Structure):
    _fields_ = [("idx", _vp), ("val", _vp), ("k", _u64)]


class StepOptions(ctypes.Structure):
    """scadles_step_options (momentum SGD, moving-average adaptive rule, accounting)."""
    _fields_ = [("momentum_buf", _vp), ("momentum", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("ewma", _vp), ("ewma_beta", ctypes.c_double), ("counters", _vp)]


class Stream(ctypes.Structure):
    """scadles_stream: one device's stream buffer."""
    _fields_ = [("rate", _u64), ("elapsed_us", _u64), ("queued", _u64), ("trained", _u64), ("dropped", _u64)]


def _sig(name, restype, *argtypes):
    f = getattr(_lib, name)
    f.restype = restype
    f.argtypes = list(argtypes)
    return f


_topk_k = _sig("scadles_topk_k", _u64, _u64, ctypes.c_double)
_ws_bytes = _sig("scadles_workspace_bytes", ctypes.c_size_t, _u32, _u64, ctypes.POINTER(ctypes.c_double))
_agg_ws_bytes = _sig("scadles_aggregate_workspace_bytes", ctypes.c_size_t, _u32, _u64)
_topk_select = _sig("scadles_topk_select", ctypes.c_int, _vp, _u64, ctypes.c_double, _vp, _vp, _vp, _vp,
                    ctypes.c_size_t, _vp)
_topk_select_noalloc = _sig("scadles_topk_select_noalloc", ctypes.c_int, _vp, _u64, ctypes.c_double, _vp, _vp,
                            _vp, _vp)
_layers_k = _sig("scadles_layers_k", _u64, ctypes.POINTER(_u64), _u32, ctypes.c_double)
_layers_ws_bytes = _sig("scadles_layers_workspace_bytes", ctypes.c_size_t, _u32, ctypes.POINTER(_u64), _u32,
                        ctypes.POINTER(ctypes.c_double))
_topk_select_layers = _sig("scadles_topk_select_layers", ctypes.c_int, ctypes.POINTER(_vp), _u32,
                           ctypes.POINTER(_u64), _u32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_vp),
                           ctypes.POINTER(_vp), _vp, _vp, ctypes.c_size_t, _vp)
_weighted_aggregate = _sig("scadles_weighted_aggregate", ctypes.c_int, ctypes.POINTER(Sparse),
                           ctypes.POINTER(ctypes.c_float), _u32, _u64, _vp, _vp, ctypes.c_size_t, _vp)
_apply_sgd = _sig("scadles_apply_sgd", ctypes.c_int, _vp, _vp, _u64, ctypes.c_float, _vp)
_apply_momentum_sgd = _sig("scadles_apply_momentum_sgd", ctypes.c_int, _vp, _vp, _vp, _u64, ctypes.c_float,
                           ctypes.c_float, ctypes.c_float, _vp)
_step_fused = _sig("scadles_step_fused", ctypes.c_int, ctypes.POINTER(_vp), _u32, _u64,
                   ctypes.POINTER(ctypes.c_double), ctypes.c_double, ctypes.POINTER(ctypes.c_float),
                   ctypes.POINTER(_vp), ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, ctypes.c_float, _vp,
                   ctypes.c_size_t, _vp)
_step_fused_ex = _sig("scadles_step_fused_ex", ctypes.c_int, ctypes.POINTER(_vp), _u32, _u64,
                      ctypes.POINTER(ctypes.c_double), ctypes.c_double, ctypes.POINTER(ctypes.c_float),
                      ctypes.POINTER(_vp), ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, ctypes.c_float,
                      ctypes.POINTER(StepOptions), _vp, ctypes.c_size_t, _vp)
_stream_weights = _sig("scadles_stream_weights", ctypes.c_int, ctypes.POINTER(ctypes.c_double), _u32,
                       ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_float),
                       ctypes.POINTER(ctypes.c_double))
_step_layers_ws_bytes = _sig("scadles_step_layers_workspace_bytes", ctypes.c_size_t, _u32, ctypes.POINTER(_u64),
                             _u32, ctypes.POINTER(ctypes.c_double))
_step_fused_layers = _sig("scadles_step_fused_layers", ctypes.c_int, ctypes.POINTER(_vp), _u32, ctypes.POINTER(_u64),
                          _u32, ctypes.POINTER(ctypes.c_double), ctypes.c_double, ctypes.POINTER(ctypes.c_float),
                          ctypes.POINTER(_vp), ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, ctypes.c_float,
                          ctypes.POINTER(StepOptions), _vp, ctypes.c_size_t, _vp)
_stream_init = _sig("scadles_stream_init", ctypes.c_int, _u32, ctypes.POINTER(_u64), ctypes.POINTER(Stream))
_stream_iteration = _sig("scadles_stream_iteration", ctypes.c_int, _u32, ctypes.POINTER(Stream), ctypes.POINTER(_u64),
                         _u64, _u64, ctypes.c_int, ctypes.c_double, ctypes.POINTER(_u64),
                         ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double))
_stream_simulate = _sig("scadles_stream_simulate", ctypes.c_int, _u32, ctypes.POINTER(_u64), ctypes.POINTER(_u64), _u64,
                        _u64, ctypes.c_int, _u64, ctypes.POINTER(_u64), ctypes.POINTER(_u64), ctypes.POINTER(_u64))
_last_error = _sig("scadles_last_error", ctypes.c_char_p)
_set_option = _sig("scadles_set_option", ctypes.c_int, ctypes.c_char_p, ctypes.c_int64)
_profile_enable = _sig("scadles_profile_enable", ctypes.c_int, ctypes.c_int)
_profile_read = _sig("scadles_profile_read", ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                     ctypes.POINTER(_u32))

STATUS = {0: "SCADLES_OK", 1: "SCADLES_EINVAL", 2: "SCADLES_EWORKSPACE", 3: "SCADLES_EHIP",
          4: "SCADLES_EUNSORTED", 5: "SCADLES_EINTERNAL"}


class ScadlesError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


def _check(code: int):
    if code != 0:
        raise ScadlesError(code, _last_error().decode(errors="replace"))


def _torch():
    import torch
    return torch


def _stream_ptr(stream) -> Optional[int]:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dev_f32(t, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous float32 tensor")
    return t.data_ptr()


def library_path() -> str:
    return LIB_PATH


# ---- host-side rules ----------------------------------------------------------------------

def topk_k(n: int, ratio: float) -> int:
    """k = clamp(floor(ratio * n), 1, n) (0 for invalid input)."""
    return int(_topk_k(int(n), float(ratio)))


def workspace_bytes(K: int, n: int, ratios: Sequence[float]) -> int:
    r = (ctypes.c_double * K)(*[float(x) for x in ratios])
    return int(_ws_bytes(K, int(n), r))


def _seg_array(seg_off):
    off = [int(x) for x in seg_off]
    return (_u64 * len(off))(*off), len(off) - 1


def layers_k(seg_off: Sequence[int], ratio: float) -> int:
    """Entries kept by the per-layer Top-k over layers [seg_off[l], seg_off[l+1])
    (0 for invalid input)."""
    arr, L = _seg_array(seg_off)
    return int(_layers_k(arr, max(L, 0), float(ratio))) if L >= 1 else 0


def layers_workspace_bytes(K: int, seg_off: Sequence[int], ratios: Sequence[float]) -> int:
    arr, L = _seg_array(seg_off)
    r = (ctypes.c_double * K)(*[float(x) for x in ratios])
    return int(_layers_ws_bytes(K, arr, L, r)) if L >= 1 else 0


def aggregate_workspace_bytes(K: int, n: int) -> int:
    return int(_agg_ws_bytes(K, int(n)))


def stream_weights(rates, b_min: float = 0.0, b_max: float = math.inf, base_batch: Optional[float] = None):
    """Eqn 4a weights (float32[K]) and, if base_batch is given, the linear-scaling gamma."""
    r = np.ascontiguousarray(rates, dtype=np.float64)
    K = r.size
    w = np.empty(K, dtype=np.float32)
    g = ctypes.c_double()
    _check(_stream_weights(r.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), K, float(b_min), float(b_max),
                           float(base_batch) if base_batch is not None else 0.0,
                           w.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                           ctypes.byref(g) if base_batch is not None else None))
    return (w, g.value) if base_batch is not None else (w, None)


PERSISTENCE, TRUNCATION = 0, 1
NO_BOUND = 2**64 - 1
_POLICIES = {"persistence": PERSISTENCE, "truncation": TRUNCATION, PERSISTENCE: PERSISTENCE,
             TRUNCATION: TRUNCATION}


def _u64_array(x, n=None):
    a = np.ascontiguousarray(x, dtype=np.uint64)
    if n is not None and a.size != n:
        raise ValueError(f"expected {n} values")
    return a


def _p64(a):
    return a.ctypes.data_as(ctypes.POINTER(_u64))


class StreamBuffers:
    """The stream buffers of K devices (persistence or truncation) and, per
    training iteration, the batch each device trains on with the Eqn 4a
    weights and learning-rate scale that follow from them. Host only."""

    def __init__(self, rates, *, b_min: int = 0, b_max: int = NO_BOUND, policy="persistence",
                 base_batch: Optional[float] = None):
        r = _u64_array(rates)
        self.K = r.size
        self.b_min, self.b_max = int(b_min), int(b_max)
        self.policy = _POLICIES[policy]
        self.base_batch = base_batch
        self.state = (Stream * self.K)()
        _check(_stream_init(self.K, _p64(r), self.state))

    def iteration(self, iter_us):
        """One iteration of iter_us microseconds per device (scalar or per device).
        Returns (batch uint64[K], weights float32[K], gamma or None)."""
        t = _u64_array(np.broadcast_to(np.asarray(iter_us, dtype=np.uint64), (self.K,)), self.K)
        batch = np.empty(self.K, dtype=np.uint64)
        w = np.empty(self.K, dtype=np.float32)
        g = ctypes.c_double()
        _check(_stream_iteration(self.K, self.state, _p64(t), self.b_min, self.b_max, self.policy,
                                 float(self.base_batch) if self.base_batch is not None else 0.0, _p64(batch),
                                 w.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                 ctypes.byref(g) if self.base_batch is not None else None))
        return batch, w, (g.value if self.base_batch is not None else None)

    def field(self, name: str) -> np.ndarray:
        return np.array([getattr(s, name) for s in self.state], dtype=np.uint64)


def stream_simulate(rates, iter_us, b_min: int, b_max: int, policy, T: int):
    """T iterations from fresh buffers: (queued uint64[T+1, K], batch uint64[T, K], dropped uint64[K])."""
    r = _u64_array(rates)
    K = r.size
    t = _u64_array(iter_us, K)
    queued = np.empty((T + 1, K), dtype=np.uint64)
    batch = np.empty((max(T, 1), K), dtype=np.uint64)
    dropped = np.empty(K, dtype=np.uint64)
    _check(_stream_simulate(K, _p64(r), _p64(t), int(b_min), int(b_max), _POLICIES[policy], int(T), _p64(queued),
                            _p64(batch), _p64(dropped)))
    return queued, batch[:T], dropped


def set_option(name: str, value: int):
    _check(_set_option(name.encode(), int(value)))


def profile_enable(on: bool = True):
    _check(_profile_enable(1 if on else 0))


def profile_read():
    """(dict stage -> summed ms, number of calls) since the last read; syncs the events."""
    ms = (ctypes.c_double * PROFILE_STAGES)()
    calls = _u32()
    _check(_profile_read(ms, ctypes.byref(calls)))
    return dict(zip(STAGE_NAMES, list(ms))), int(calls.value)


def _workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---- the three calls of the hot path -----------------------------------------------------------

def topk_select(grad, ratio: float, *, workspace=None, energies: bool = False, stream=None):
    """Top-k of one gradient. Returns (idx uint32[k], val float32[k]) or, with
    energies=True, (idx, val, float64[2] = (sum g^2, sum kept g^2))."""
    torch = _torch()
    gp = _dev_f32(grad, "grad")
    n = grad.numel()
    k = topk_k(n, ratio)
    if k == 0:
        raise ScadlesError(1, f"invalid n={n} or ratio={ratio}")
    dev = grad.device
    idx = torch.empty(k, dtype=torch.uint32, device=dev)
    val = torch.empty(k, dtype=torch.float32, device=dev)
    en = torch.empty(2, dtype=torch.float64, device=dev) if energies else None
    need = workspace_bytes(1, n, [ratio])
    ws = workspace if workspace is not None else _workspace(need, dev)
    _check(_topk_select(gp, n, float(ratio), idx.data_ptr(), val.data_ptr(),
                        en.data_ptr() if en is not None else None, ws.data_ptr(), ws.numel(),
                        _stream_ptr(stream)))
    return (idx, val, en) if energies else (idx, val)


def topk_select_noalloc(grad, ratio: float, idx, val, energies=None, *, stream=None):
    """Top-k of one gradient into caller-given outputs (idx uint32[k], val
    float32[k], energies float64[2] or None) using the library's static
    scratch: the call allocates nothing (scadles_topk_select_noalloc)."""
    torch = _torch()
    gp = _dev_f32(grad, "grad")
    n = grad.numel()
    k = topk_k(n, ratio)
    if k == 0:
        raise ScadlesError(1, f"invalid n={n} or ratio={ratio}")
    if idx.numel() < k or val.numel() < k or not idx.is_cuda or not idx.is_contiguous():
        raise ValueError(f"idx and val must be contiguous GPU tensors of at least k={k} entries")
    if idx.dtype not in (torch.uint32, torch.int32):
        raise TypeError("idx must be uint32")
    if energies is not None and (energies.dtype != torch.float64 or energies.numel() < 2 or not energies.is_cuda):
        raise TypeError("energies must be a float64 GPU tensor of 2 entries")
    _check(_topk_select_noalloc(gp, n, float(ratio), idx.data_ptr(), _dev_f32(val, "val"),
                                energies.data_ptr() if energies is not None else None, _stream_ptr(stream)))
    return idx, val, energies


def weighted_aggregate(sets, weights, n: int, *, out=None, workspace=None, stream=None):
    """Eqn 4b. ``sets``: list of (idx uint32 tensor or None for dense, val float32 tensor)."""
    torch = _torch()
    K = len(sets)
    w = np.ascontiguousarray(weights, dtype=np.float32)
    if w.size != K:
        raise ValueError("one weight per set")
    arr = (Sparse * K)()
    dev = None
    for j, (idx, val) in enumerate(sets):
        vp = _dev_f32(val, f"sets[{j}].val")
        dev = val.device
        if idx is None:
            arr[j] = Sparse(None, vp, val.numel())
        else:
            if idx.dtype not in (torch.uint32, torch.int32) or not idx.is_cuda or not idx.is_contiguous():
                raise TypeError(f"sets[{j}].idx must be a contiguous uint32 GPU tensor")
            if idx.numel() != val.numel():
                raise ValueError(f"sets[{j}]: idx and val differ in length")
            arr[j] = Sparse(idx.data_ptr(), vp, idx.numel())
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else _workspace(aggregate_workspace_bytes(K, n), dev)
    _check(_weighted_aggregate(arr, w.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), K, int(n),
                               _dev_f32(out, "out"), ws.data_ptr(), ws.numel(), _stream_ptr(stream)))
    return out


def apply_sgd(params, grad, lr: float, *, stream=None):
    """Eqn 4c in place on ``params``."""
    _check(_apply_sgd(_dev_f32(params, "params"), _dev_f32(grad, "grad"), params.numel(), float(lr),
                      _stream_ptr(stream)))
    return params


def apply_momentum_sgd(params, momentum_buf, grad, lr: float, momentum: float, weight_decay: float, *,
                       stream=None):
    """Momentum SGD with weight decay (§V training setup) in place on ``params``
    and ``momentum_buf``."""
    if not (params.numel() == momentum_buf.numel() == grad.numel()):
        raise ValueError("params, momentum_buf and grad must have the same size")
    _check(_apply_momentum_sgd(_dev_f32(params, "params"), _dev_f32(momentum_buf, "momentum_buf"),
                               _dev_f32(grad, "grad"), params.numel(), float(lr), float(momentum),
                               float(weight_decay), _stream_ptr(stream)))
    return params, momentum_buf


class LayerSelect:
    """Per-layer Top-k of K gradients that share one layer layout (every layer
    keeps its own top fraction): outputs and workspace allocated once, ``run``
    only marshals pointers. ``seg_off`` = [0, ..., n] are the layer bounds."""

    def __init__(self, grads, seg_off: Sequence[int], ratios: Sequence[float]):
        torch = _torch()
        if isinstance(grads, torch.Tensor) and grads.dim() == 2:
            grads = [grads[j] for j in range(grads.shape[0])]
        self.grads = list(grads)
        self.K = len(self.grads)
        if not 1 <= self.K <= MAX_DEVICES:
            raise ValueError(f"K must be in [1, {MAX_DEVICES}]")
        self.seg_off = [int(x) for x in seg_off]
        self.n = self.seg_off[-1] if self.seg_off else 0
        for j, g in enumerate(self.grads):
            _dev_f32(g, f"grads[{j}]")
            if g.numel() != self.n:
                raise ValueError("every gradient must have seg_off[-1] elements")
        self.ratios = [float(r) for r in ratios]
        if len(self.ratios) != self.K:
            raise ValueError("one ratio per device")
        self.k = [layers_k(self.seg_off, r) for r in self.ratios]
        if min(self.k) == 0:
            raise ScadlesError(1, "invalid layer bounds or ratio")
        dev = self.grads[0].device
        self.idx = [torch.empty(k, dtype=torch.uint32, device=dev) for k in self.k]
        self.val = [torch.empty(k, dtype=torch.float32, device=dev) for k in self.k]
        self.energies = torch.empty(2 * self.K, dtype=torch.float64, device=dev)
        self.ws = _workspace(layers_workspace_bytes(self.K, self.seg_off, self.ratios), dev)
        self._seg, self._L = _seg_array(self.seg_off)
        self._ratios = (ctypes.c_double * self.K)(*self.ratios)
        self._grad_ptrs = (_vp * self.K)(*[g.data_ptr() for g in self.grads])
        self._idx_ptrs = (_vp * self.K)(*[t.data_ptr() for t in self.idx])
        self._val_ptrs = (_vp * self.K)(*[t.data_ptr() for t in self.val])

    def run(self, *, stream=None):
        """Select every device's kept set; returns (idx list, val list, energies float64[2K])."""
        _check(_topk_select_layers(self._grad_ptrs, self.K, self._seg, self._L, self._ratios, self._idx_ptrs,
                                   self._val_ptrs, self.energies.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                   _stream_ptr(stream)))
        return self.idx, self.val, self.energies


# ---- the fused step -----------------------------------------------------------------------------

@dataclass
class StepOutputs:
    idx: list
    val: list
    dense: object
    energies: object
    compressed: object


class FusedStep:
    """One hot-path step for K devices of n elements (Top-k + energies + adaptive
    rule + Eqn 4b aggregation + optional Eqn 4c update), with every output and
    the workspace allocated once so that ``run`` only marshals pointers."""

    def __init__(self, grads, ratios: Sequence[float], *, delta: float = math.inf, params=None,
                 momentum_buf=None, momentum: float = 0.0, weight_decay: float = 0.0,
                 ewma_beta: Optional[float] = None, track: bool = False, seg_off: Optional[Sequence[int]] = None):
        torch = _torch()
        if isinstance(grads, torch.Tensor) and grads.dim() == 2:
            grads = [grads[j] for j in range(grads.shape[0])]
        self.K = len(grads)
        if not 1 <= self.K <= MAX_DEVICES:
            raise ValueError(f"K must be in [1, {MAX_DEVICES}]")
        self.n = grads[0].numel()
        # per-layer Top-k over layers [seg_off[l], seg_off[l+1]) when given
        self.seg_off = None if seg_off is None else [int(x) for x in seg_off]
        if self.seg_off is not None:
            if len(self.seg_off) < 2 or self.seg_off[-1] != self.n:
                raise ValueError("seg_off must run from 0 to the gradients' size")
            self._seg, self._L = _seg_array(self.seg_off)
        self.grads = list(grads)
        for j, g in enumerate(self.grads):
            _dev_f32(g, f"grads[{j}]")
            if g.numel() != self.n:
                raise ValueError("all gradients must have n elements")
        dev = self.grads[0].device
        self.device = dev
        self.params = params
        # momentum SGD with weight decay in place of Eqn 4c when a buffer is given
        self.momentum_buf = momentum_buf
        self.momentum = float(momentum)
        self.weight_decay = float(weight_decay)
        if momentum_buf is not None:
            if params is None:
                raise ValueError("momentum_buf needs params")
            _dev_f32(momentum_buf, "momentum_buf")
            if momentum_buf.numel() != self.n or params.numel() != self.n:
                raise ValueError("params and momentum_buf must have n elements")
        self.delta = float(delta)
        self.set_ratios(ratios)
        # §IV moving average of the energies (state zero-filled: no history) and
        # §V-G accounting, both kept on the device across run() calls
        self.ewma_beta = None if ewma_beta is None else float(ewma_beta)
        self.ewma = (torch.zeros(2 * self.K, dtype=torch.float64, device=dev)
                     if ewma_beta is not None else None)
        self.counters = torch.zeros(3 * self.K, dtype=torch.int64, device=dev) if track else None
        self._opts = StepOptions(
            momentum_buf.data_ptr() if momentum_buf is not None else None, self.momentum, self.weight_decay,
            self.ewma.data_ptr() if self.ewma is not None else None,
            self.ewma_beta if self.ewma_beta is not None else 0.0,
            self.counters.data_ptr() if self.counters is not None else None)
        self.dense = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.energies = torch.empty(2 * self.K, dtype=torch.float64, device=dev)
        self.compressed = torch.empty(self.K, dtype=torch.uint8, device=dev)
        self._grad_ptrs = (_vp * self.K)(*[g.data_ptr() for g in self.grads])
        self._w = (ctypes.c_float * self.K)()

    def set_grads(self, grads):
        """Point the step at other gradients of the same shape (marshalling only)."""
        torch = _torch()
        if isinstance(grads, torch.Tensor) and grads.dim() == 2:
            grads = [grads[j] for j in range(grads.shape[0])]
        if len(grads) != self.K:
            raise ValueError("one gradient per device")
        for j, g in enumerate(grads):
            _dev_f32(g, f"grads[{j}]")
            if g.numel() != self.n:
                raise ValueError("all gradients must have n elements")
        self.grads = list(grads)
        self._grad_ptrs = (_vp * self.K)(*[g.data_ptr() for g in self.grads])

    def set_ratios(self, ratios):
        torch = _torch()
        ratios = [float(r) for r in ratios]
        if len(ratios) != self.K:
            raise ValueError("one ratio per device")
        self.ratios = ratios
        if self.seg_off is not None:
            self.k = [layers_k(self.seg_off, r) for r in ratios]
        else:
            self.k = [topk_k(self.n, r) for r in ratios]
        if min(self.k) == 0:
            raise ScadlesError(1, "ratio outside (0, 1]")
        self.idx = [torch.empty(k, dtype=torch.uint32, device=self.device) for k in self.k]
        self.val = [torch.empty(k, dtype=torch.float32, device=self.device) for k in self.k]
        self._ratios = (ctypes.c_double * self.K)(*ratios)
        self._idx_ptrs = (_vp * self.K)(*[t.data_ptr() for t in self.idx])
        self._val_ptrs = (_vp * self.K)(*[t.data_ptr() for t in self.val])
        if self.seg_off is not None:
            need = int(_step_layers_ws_bytes(self.K, self._seg, self._L, self._ratios))
        else:
            need = workspace_bytes(self.K, self.n, ratios)
        if need == 0:
            raise ScadlesError(1, "workspace query rejected the arguments")
        if getattr(self, "ws", None) is None or self.ws.numel() < need:
            self.ws = _workspace(need, self.device)

    def run(self, weights, lr: float = 0.0, *, stream=None) -> StepOutputs:
        w = np.ascontiguousarray(weights, dtype=np.float32)
        for j in range(self.K):
            self._w[j] = float(w[j])
        pp = _dev_f32(self.params, "params") if self.params is not None else None
        opts = self.momentum_buf is not None or self.ewma is not None or self.counters is not None
        if self.seg_off is not None:
            _check(_step_fused_layers(self._grad_ptrs, self.K, self._seg, self._L, self._ratios, self.delta, self._w,
                                      self._idx_ptrs, self._val_ptrs, self.dense.data_ptr(),
                                      self.energies.data_ptr(), self.compressed.data_ptr(), pp, float(lr),
                                      ctypes.byref(self._opts) if opts else None, self.ws.data_ptr(),
                                      self.ws.numel(), _stream_ptr(stream)))
        elif opts:
            _check(_step_fused_ex(self._grad_ptrs, self.K, self.n, self._ratios, self.delta, self._w,
                                  self._idx_ptrs, self._val_ptrs, self.dense.data_ptr(), self.energies.data_ptr(),
                                  self.compressed.data_ptr(), pp, float(lr), ctypes.byref(self._opts),
                                  self.ws.data_ptr(), self.ws.numel(), _stream_ptr(stream)))
        else:
            _check(_step_fused(self._grad_ptrs, self.K, self.n, self._ratios, self.delta, self._w,
                               self._idx_ptrs, self._val_ptrs, self.dense.data_ptr(), self.energies.data_ptr(),
                               self.compressed.data_ptr(), pp, float(lr), self.ws.data_ptr(), self.ws.numel(),
                               _stream_ptr(stream)))
        return StepOutputs(self.idx, self.val, self.dense, self.energies, self.compressed)

    def accounting(self):
        """The counters of ``track=True`` as uint64[K, 3]: per device the iterations
        that sent Top-k, the iterations, and the floats sent (§V-G)."""
        if self.counters is None:
            raise ValueError("construct with track=True")
        return self.counters.cpu().numpy().reshape(self.K, 3).astype(np.uint64)


def step_fused(grads, ratios, weights, *, delta: float = math.inf, params=None, lr: float = 0.0,
               stream=None) -> StepOutputs:
    """One-shot convenience wrapper around FusedStep."""
    return FusedStep(grads, ratios, delta=delta, params=params).run(weights, lr, stream=stream)
