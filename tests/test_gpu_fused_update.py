"""GPU parity of the aggregation fused with the next layer's update,
T = bf16(act(A X)) bf16(W) (dualgcn_spmm_update).

* bit for bit against the two-call route (dualgcn_spmm_act with a bfloat16 output, then
  dualgcn_update of that output), on graphs that reach every path of the SpMM (sparse
  tasks, empty rows, lane-group and wavefront dense rows, a hub row split into parts)
  and every lane-group width (F_in = 32 ... 256);
* against the oracle: |T - T_ref| <= 1e-2 ((|H| + B) |W|) per element, where
  H = act(A X) and B = |A| |X| in float64 -- one bfloat16 rounding of H and of W
  (2^-8 each) and the SpMM's own error, which the bfloat16 rounding may turn into one
  more bfloat16 step -- and, normwise, within 1e-3 of the same chain computed with the
  declared bfloat16 roundings in float64;
* argument checks that need a plan.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from graphgen import configs, dense, small
from test_gpu_parity import TINY, to_dev

pytestmark = pytest.mark.gpu

TOL = 1e-2
DECLARED_TOL = 1e-3


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _empty_runs():
    """3,001 rows, 40% of them empty (one run of about 1,200 empty rows in the processing
    order, cut into tasks of 8), the others 1-19 random columns with values in (0, 1]."""
    gen = np.random.default_rng(17)
    n = 3001
    g = small.from_rows([[] if gen.random() < 0.4 else gen.integers(0, n, gen.integers(1, 20)).tolist()
                         for _ in range(n)])
    g.val[:] = gen.random(g.val.size).astype(np.float32) + np.float32(1e-3)
    return g


GRAPHS = {
    "empty_runs": _empty_runs,
    "gnp257": TINY["gnp257"],
    "rows_dup_empty": TINY["rows_dup_empty"],
    "hub_star": TINY["hub_star"],
    "edgeless7": TINY["edgeless7"],
    "single": TINY["single"],
    "c1": lambda: configs.load_graph("c1"),
    "c2": lambda: configs.load_graph("c2"),
}

_cache = {}


def _graph(name):
    if name not in _cache:
        _cache[name] = GRAPHS[name]()
    return _cache[name]


def _weights(F_in, F_out, seed):
    return dense.glorot(F_in, F_out, seed=seed)


def _two_calls(dg, plan, Xd, Wd, relu):
    H = dg.spmm(plan, Xd, relu=relu, out_bf16=True)
    return dg.update(H, Wd)


@pytest.mark.parametrize("name", sorted(GRAPHS))
@pytest.mark.parametrize("F_in,F_out,relu", [(128, 64, True), (64, 32, False), (32, 32, True),
                                             (256, 64, True), (96, 160, False), (128, 256, True),
                                             (256, 192, False), (256, 224, True)])
def test_fused_equals_two_calls_and_oracle(dg, device, name, F_in, F_out, relu):
    g = _graph(name)
    plan = dg.Plan(*to_dev(g, device), seed=3, walks_per_node=8, walk_len=4)
    X = dense.features_normal(g.n, F_in, seed=F_in + 7, stream_id=41)
    W = _weights(F_in, F_out, seed=F_out + 1)
    Xd, Wd = torch.from_numpy(X).to(device), torch.from_numpy(W).to(device)
    T = dg.spmm_update(plan, Xd, Wd, relu=relu)
    T2 = _two_calls(dg, plan, Xd, Wd, relu)
    got = T.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), T2.cpu().numpy().view(np.uint32)), \
        f"{name} {F_in}->{F_out}: fused and two-call results differ"
    # with H kept: the same T, and H is the plain kernel's bfloat16 output bit for bit
    Hk = torch.full((g.n, F_in), float("nan"), dtype=torch.bfloat16, device=device)
    Tk = dg.spmm_update(plan, Xd, Wd, relu=relu, H=Hk)
    assert torch.equal(Tk, T)
    assert torch.equal(Hk.view(torch.int16), dg.spmm(plan, Xd, relu=relu, out_bf16=True).view(torch.int16))
    # the oracle (rows sampled on the larger graphs)
    rows = np.arange(g.n, dtype=np.int32)
    if g.n > 4096:
        info = plan.info()
        perm = plan.export()[0]
        gen = np.random.default_rng(F_in * 1000 + F_out)
        rows = np.unique(np.concatenate([gen.choice(g.n, 1500, replace=False), perm[-8:],
                                         perm[max(0, info["n_sparse"] - 8):info["n_sparse"] + 8]]))
        rows = rows.astype(np.int32)
    H, B = oracle.spmm(g, X, rows)
    if relu:
        H = np.maximum(H, 0.0)
    Tr = H @ W.astype(np.float64)
    bound = (np.abs(H) + B) @ np.abs(W.astype(np.float64))
    err = np.abs(got[rows].astype(np.float64) - Tr)
    bad = ~(err <= TOL * bound)
    assert not bad.any(), f"{name}: {bad.sum()} outside; worst ratio {np.max(err / np.maximum(bound, 1e-300))}"
    Td = oracle.round_bf16(H) @ oracle.round_bf16(W)
    scale = np.linalg.norm(Td)
    if scale > 0:
        assert np.linalg.norm(got[rows] - Td) <= DECLARED_TOL * scale
    plan.destroy()


def test_fused_on_a_shifted_plan_matches_after_rebuild(dg, device):
    """Two plans of different matrices in turn: nothing of one launch leaks into the next."""
    g1, g2 = _graph("hub_star"), _graph("gnp257")
    W = _weights(128, 64, seed=2)
    Wd = torch.from_numpy(W).to(device)
    for g in (g1, g2, g1):
        plan = dg.Plan(*to_dev(g, device), seed=1, walks_per_node=4, walk_len=3)
        Xd = torch.from_numpy(dense.features_normal(g.n, 128, seed=5, stream_id=42)).to(device)
        T = dg.spmm_update(plan, Xd, Wd, relu=True)
        T2 = _two_calls(dg, plan, Xd, Wd, True)
        assert torch.equal(T, T2)
        plan.destroy()


def test_route_choice(dg, device):
    """Small operands (they fit the memory-side cache) take the two calls when H is given;
    an H that is only 8-byte aligned keeps the fused kernel; both give the same bits."""
    g = _graph("gnp257")
    plan = dg.Plan(*to_dev(g, device), seed=1, walks_per_node=4, walk_len=3)
    assert not dg.spmm_update_route(plan, 128, 64)
    with pytest.raises(dg.DualGCNError):
        dg.spmm_update_route(plan, 48, 64)
    X = torch.from_numpy(dense.features_normal(g.n, 128, seed=5, stream_id=44)).to(device)
    W = torch.from_numpy(_weights(128, 64, seed=6)).to(device)
    T_fused = dg.spmm_update(plan, X, W, relu=True)               # no H: the fused kernel
    H16 = torch.full((g.n, 128), float("nan"), dtype=torch.bfloat16, device=device)
    T_two = dg.spmm_update(plan, X, W, relu=True, H=H16)          # H given: the two calls
    buf = torch.full((g.n * 128 + 4,), float("nan"), dtype=torch.bfloat16, device=device)
    H8 = buf[4:].view(g.n, 128)                                   # 8-byte aligned only
    assert H8.data_ptr() % 16 == 8
    T_h8 = dg.spmm_update(plan, X, W, relu=True, H=H8)
    assert torch.equal(T_two, T_fused) and torch.equal(T_h8, T_fused)
    H_ref = dg.spmm(plan, X, relu=True, out_bf16=True)
    assert torch.equal(H16.view(torch.int16), H_ref.view(torch.int16))
    assert torch.equal(H8.view(torch.int16), H_ref.view(torch.int16))
    plan.destroy()


def test_fused_argument_checks(dg, device):
    g = _graph("gnp257")
    plan = dg.Plan(*to_dev(g, device), seed=1, walks_per_node=4, walk_len=3)
    L = dg.lib()
    X = torch.zeros((g.n, 256), dtype=torch.float32, device=device)
    W = torch.zeros((256, 256), dtype=torch.float32, device=device)
    T = torch.zeros((g.n, 256), dtype=torch.float32, device=device)
    h = plan.handle
    call = L.dualgcn_spmm_update
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 128, 64, dg.RELU, None) == 0
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 128, 64, 2, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 48, 64, 0, None) == dg.ERR_UNSUPPORTED
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 128, 48, 0, None) == dg.ERR_UNSUPPORTED
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 288, 64, 0, None) == dg.ERR_UNSUPPORTED
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 256, 256, 0, None) == dg.ERR_UNSUPPORTED
    # W^T (224 x 264 bfloat16) and the row tiles fit, with the output staging inside the tile
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 256, 224, 0, None) == 0
    assert call(h, X.data_ptr() + 4, W.data_ptr(), T.data_ptr(), None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr() + 4, None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), X.data_ptr(), None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), W.data_ptr(), None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, None, W.data_ptr(), T.data_ptr(), None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(None, X.data_ptr(), W.data_ptr(), T.data_ptr(), None, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    H = torch.zeros((g.n, 128), dtype=torch.bfloat16, device=device)
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), H.data_ptr(), 128, 64, 0, None) == 0
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), H.data_ptr() + 2, 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), T.data_ptr(), 128, 64, 0, None) == dg.ERR_INVALID_ARG
    assert call(h, X.data_ptr(), W.data_ptr(), T.data_ptr(), X.data_ptr(), 128, 64, 0, None) == dg.ERR_INVALID_ARG
    torch.cuda.synchronize()
    with pytest.raises(ValueError):
        dg.spmm_update(plan, X, W[:128])
    plan.destroy()


@pytest.mark.parametrize("force", [1, 2])          # every row sparse / every row dense
@pytest.mark.parametrize("name", ["gnp257", "hub_star", "c1"])
def test_fused_with_forced_paths(dg, device, name, force):
    g = _graph(name)
    plan = dg.Plan(*to_dev(g, device), seed=3, walks_per_node=8, walk_len=4, force_mode=force)
    X = dense.features_normal(g.n, 64, seed=9, stream_id=43)
    W = _weights(64, 96, seed=4)
    Xd, Wd = torch.from_numpy(X).to(device), torch.from_numpy(W).to(device)
    side = torch.cuda.Stream(device=device)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        T = dg.spmm_update(plan, Xd, Wd, relu=True)
    torch.cuda.current_stream().wait_stream(side)
    assert torch.equal(T, _two_calls(dg, plan, Xd, Wd, True))
    plan.destroy()


@pytest.mark.parametrize("name", ["gnp257", "hub_star", "c2"])
def test_fused_with_identity_weights_is_the_bf16_spmm(dg, device, name):
    """W = I: every output is one bf16 value times 1 plus exact zeros, so T holds exactly the
    bfloat16 aggregation the plain kernel writes (as float32)."""
    g = _graph(name)
    plan = dg.Plan(*to_dev(g, device), seed=5, walks_per_node=8, walk_len=4)
    Xd = torch.from_numpy(dense.features_normal(g.n, 128, seed=2, stream_id=44)).to(device)
    I = torch.eye(128, dtype=torch.float32, device=device)
    T = dg.spmm_update(plan, Xd, I, relu=True)
    H = dg.spmm(plan, Xd, relu=True, out_bf16=True)
    assert torch.equal(T, H.float())
    plan.destroy()
