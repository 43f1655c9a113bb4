"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times (the fused step). The Top-k oracle here is the O(n) statement
of the same definition (k-th largest magnitude by a library selection, then
the kept set by definition); aggregation and SGD use the plain C oracle over
every element. Indices, values, aggregate and parameters are compared bit for
bit, the energies within the bound of a double sum of their terms. The
largest workload runs all 10 of its iterations with the parameters chained
through the updates."""
import pytest

from _gpu_common import log, run_config, threshold_topk

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def sc():
    import paper_2301_08897_amd as sc
    sc.set_option("force_exact", 0)
    sc.set_option("force_fallback", 0)
    return sc


@pytest.mark.timeout(900)
@pytest.mark.parametrize("config,iters", [(2, 1), (3, 3), (4, 1), (5, 10)])
def test_full_size(sc, config, iters):
    log(f"full-size parity C{config} ({iters} iteration(s))")
    run_config(sc, config, iterations=iters, topk=threshold_topk, threads=8)
