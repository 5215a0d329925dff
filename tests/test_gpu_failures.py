"""Failure handling on the device side of the library: an injected allocation failure at
every allocation of a partition (and of the pattern dump and plan save) returns
DUALGCN_ERR_OOM, leaves no plan, leaks no device memory, and the next call succeeds."""
import os

import numpy as np
import pytest
import torch

from graphgen import small

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _dev(g, device):
    return (torch.from_numpy(np.ascontiguousarray(g.rowptr)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.col)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.val)).to(device))


_calls = [0]


def _with_failure(n, fn):
    # the library counts from each new value of the variable: a distinct suffix per call
    _calls[0] += 1
    os.environ["DUALGCN_TEST_FAIL_ALLOC"] = f"{n} call{_calls[0]}"
    try:
        return fn()
    finally:
        del os.environ["DUALGCN_TEST_FAIL_ALLOC"]


def test_injected_allocation_failures(dg, device):
    g = small.random_graph(3000, 0.004, seed=8)
    rp, c, v = _dev(g, device)
    ref = dg.Plan(rp, c, v, seed=1, walks_per_node=8, walk_len=4)
    ref_perm = ref.export()[0]
    ref.destroy()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    free0 = torch.cuda.mem_get_info()[0]
    failures = 0
    for n in (1, 2):                     # the plan's block, then the build's scratch block
        def build():
            return dg.Plan(rp, c, v, seed=1, walks_per_node=8, walk_len=4)
        with pytest.raises(dg.DualGCNError) as e:
            _with_failure(n, build)
        assert e.value.status == dg.ERR_OOM
        failures += 1
    # the third allocation does not exist: the partition succeeds
    plan = _with_failure(3, lambda: dg.Plan(rp, c, v, seed=1, walks_per_node=8, walk_len=4))
    assert np.array_equal(plan.export()[0], ref_perm)
    with pytest.raises(dg.DualGCNError) as e:
        _with_failure(1, plan.save)
    assert e.value.status == dg.ERR_OOM
    plan.destroy()
    with pytest.raises(dg.DualGCNError) as e:
        _with_failure(1, lambda: dg.arw_patterns(rp, c, v, seed=0, walks_per_node=2, walk_len=3))
    assert e.value.status == dg.ERR_OOM
    # no leak: after the failures, build and release plans; free memory returns
    for _ in range(3):
        p = dg.Plan(rp, c, v, seed=1, walks_per_node=8, walk_len=4)
        assert np.array_equal(p.export()[0], ref_perm)
        p.destroy()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert torch.cuda.mem_get_info()[0] >= free0 - (2 << 20)
    assert failures == 2
