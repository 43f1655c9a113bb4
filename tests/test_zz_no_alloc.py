"""The allocation-free Top-k entry point (scadles_topk_select_noalloc, its
workspace in the library's static per-GPU scratch) against the entry point
with a caller workspace (scadles_topk_select), both called through the C ABI:
indices, values and energies bit for bit, on consecutive calls whose sizes
shrink (the scratch keeps the previous call's contents), and the oracle on
the same inputs."""
import ctypes

import numpy as np
import pytest

import oracle
import workloads
from _gpu_common import check_energies, log, same_bits, torch_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    L = ctypes.CDLL(sc.library_path())
    vp, u64, f64 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_double
    L.scadles_topk_select_noalloc.restype = ctypes.c_int
    L.scadles_topk_select_noalloc.argtypes = [vp, u64, f64, vp, vp, vp, vp]
    L.scadles_topk_select.restype = ctypes.c_int
    L.scadles_topk_select.argtypes = [vp, u64, f64, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.scadles_workspace_bytes.restype = ctypes.c_size_t
    L.scadles_workspace_bytes.argtypes = [ctypes.c_uint32, u64, ctypes.POINTER(f64)]
    L.scadles_topk_k.restype = u64
    L.scadles_topk_k.argtypes = [u64, f64]
    L.scadles_last_error.restype = ctypes.c_char_p
    return L


def _outputs(torch, dev, k):
    return (torch.empty(k, dtype=torch.uint32, device=dev), torch.empty(k, dtype=torch.float32, device=dev),
            torch.empty(2, dtype=torch.float64, device=dev))


def _both(lib, g_dev, n, ratio):
    """(noalloc outputs, workspace outputs) of one gradient, on the current stream."""
    torch, dev = torch_dev()
    k = lib.scadles_topk_k(n, ratio)
    assert k > 0
    s = torch.cuda.current_stream().cuda_stream
    a = _outputs(torch, dev, k)
    rc = lib.scadles_topk_select_noalloc(g_dev.data_ptr(), n, ratio, a[0].data_ptr(), a[1].data_ptr(),
                                         a[2].data_ptr(), s)
    assert rc == 0, lib.scadles_last_error()
    need = lib.scadles_workspace_bytes(1, n, ctypes.byref(ctypes.c_double(ratio)))
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    b = _outputs(torch, dev, k)
    rc = lib.scadles_topk_select(g_dev.data_ptr(), n, ratio, b[0].data_ptr(), b[1].data_ptr(), b[2].data_ptr(),
                                 ws.data_ptr(), ws.numel(), s)
    assert rc == 0, lib.scadles_last_error()
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in a], [t.cpu().numpy() for t in b], k


def _check(lib, g, ratio, label):
    torch, dev = torch_dev()
    n = g.size
    log(f"noalloc {label}: n={n} ratio={ratio}")
    (ia, va, ea), (ib, vb, eb), k = _both(lib, torch.from_numpy(g).to(dev), n, ratio)
    assert np.array_equal(ia, ib), f"{label}: indices differ between the two entry points"
    assert same_bits(va, vb), f"{label}: values differ"
    assert np.array_equal(ea.view(np.uint64), eb.view(np.uint64)), f"{label}: energies differ"
    idx_o, _, _, _ = oracle.topk_by_threshold(g, k)
    assert np.array_equal(ia, idx_o), f"{label}: indices differ from the oracle"
    assert same_bits(va, g[idx_o]), f"{label}: values differ from the oracle"
    check_energies(label, ea[0], ea[1], oracle.energies_extended(g, idx_o), n, k)


def test_noalloc_matches_workspace_call_shrinking_sizes(lib):
    """Two calls in a row, the second on a smaller input; then the largest
    workload's gradient size (the most scratch a listed workload uses) and a
    smaller one again."""
    s = workloads.spec(2, n=3_000_017, K=2)
    g1 = workloads.gradient(s, 0, 0)
    g2 = workloads.gradient(s, 0, 1)[:700_001].copy()
    _check(lib, g1, 0.01, "first call")
    _check(lib, g2, 0.01, "second call, smaller")
    s5 = workloads.spec(5, K=1, iterations=1)
    g5 = workloads.gradient(s5, 0, 0)
    _check(lib, g5, 0.01, "VGG-19-sized gradient")
    _check(lib, g2[:50_000].copy(), 0.02, "small (exact path) after the largest")


def test_noalloc_rejects_more_than_the_scratch(lib):
    torch, dev = torch_dev()
    n = 143_667_240
    g = torch.zeros(n, dtype=torch.float32, device=dev)
    k = lib.scadles_topk_k(n, 0.1)
    idx, val, en = _outputs(torch, dev, k)
    rc = lib.scadles_topk_select_noalloc(g.data_ptr(), n, 0.1, idx.data_ptr(), val.data_ptr(), en.data_ptr(),
                                         torch.cuda.current_stream().cuda_stream)
    assert rc == 2 and b"scratch" in lib.scadles_last_error()
