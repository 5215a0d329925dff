"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

* partition (walk patterns, S, K, K*, sums, perm, n_sparse): bit-exact;
* SpMM: |y - y_oracle| <= 1e-5 * sum |a||x| element by element;
* GCN layer (bf16 matrix cores): |y - y_oracle| <= 1e-2 * |A| (|X| |W|).
"""
import numpy as np
import pytest
import torch

import oracle
from graphgen import configs, small, dense

pytestmark = pytest.mark.gpu

SPMM_TOL = 1e-5
GCN_TOL = 1e-2


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def to_dev(g, device):
    return (torch.from_numpy(np.ascontiguousarray(g.rowptr)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.col)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.val)).to(device))


def assert_plan_matches(dg, plan, g, seed, k, d, alpha=(1, 2), beta=(1, 2), force=0):
    perm, S, K = plan.export()
    info = plan.info()
    ref = oracle.partition(g, seed, k, d, alpha, beta, force)
    assert np.array_equal(S, ref["S"]), f"S differs at {np.flatnonzero(S != ref['S'])[:10]}"
    assert np.array_equal(K, ref["K"])
    assert info["s1"] == ref["S1"] and info["s2"] == ref["S2"]
    assert info["kstar"] == ref["kstar"]
    assert info["n_sparse"] == ref["n_sparse"]
    assert np.array_equal(perm, ref["perm"])
    assert (info["alpha_num"], info["alpha_den"]) == tuple(ref["alpha"])
    return ref


def assert_spmm_close(Y, Yr, B, tol=SPMM_TOL, what=""):
    Y = np.asarray(Y, dtype=np.float64)
    err = np.abs(Y - Yr)
    bad = ~(err <= tol * B)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} elements outside {tol} sum|a||x|; first at "
                             f"{tuple(i)}: got {Y[tuple(i)]!r} want {Yr[tuple(i)]!r} bound {B[tuple(i)]!r}")


TINY = {
    "gnp30": lambda: small.random_graph(30, 0.2, seed=1),
    "gnp257": lambda: small.random_graph(257, 0.03, seed=2),
    "star50": lambda: small.star(50, self_loops=True, normalise=True),
    "clique20": lambda: small.clique(20, self_loops=True, normalise=True),
    "path31": lambda: small.path(31, self_loops=True, normalise=True),
    "cycle40": lambda: small.cycle(40, self_loops=True, normalise=True),
    "edgeless7": lambda: small.edgeless(7),
    "single": lambda: small.edgeless(1),
    "rows_dup_empty": lambda: small.from_rows([[1, 1, 2], [], [0, 3, 3, 3], [2], [], [0, 1, 2, 3, 4]]),
    "hub_star": lambda: small.star(10000, self_loops=True, normalise=True),   # one row of 10001 entries
}


# ---------------------------------------------------------------- walks and partition

@pytest.mark.parametrize("name", ["gnp30", "star50", "clique20", "path31", "rows_dup_empty", "single"])
@pytest.mark.parametrize("k,d", [(8, 4), (3, 7), (1, 1), (100, 2), (4, 40)])
def test_walk_patterns_bitexact(dg, device, name, k, d):
    g = TINY[name]()
    rp, c, v = to_dev(g, device)
    P = dg.arw_patterns(rp, c, v, seed=11, walks_per_node=k, walk_len=d).cpu().numpy()
    assert np.array_equal(P, oracle.patterns(g, 11, k, d))


def test_walk_patterns_c1(dg, device):
    g = configs.load_graph("c1")
    rp, c, v = to_dev(g, device)
    P = dg.arw_patterns(rp, c, v, seed=0, walks_per_node=8, walk_len=4).cpu().numpy()
    assert np.array_equal(P, oracle.patterns(g, 0, 8, 4))


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("k,d", [(8, 4), (16, 5), (3, 2), (100, 3)])
def test_partition_bitexact_tiny(dg, device, name, k, d):
    g = TINY[name]()
    plan = dg.Plan(*to_dev(g, device), seed=5, walks_per_node=k, walk_len=d)
    assert_plan_matches(dg, plan, g, 5, k, d)


@pytest.mark.parametrize("alpha,beta", [((0, 1), (1, 2)), ((1, 1), (1, 2)), ((1, 3), (3, 2)),
                                        ((1, 2), (0, 1)), ((2, 5), (7, 3))])
@pytest.mark.parametrize("force", [0, 1, 2])
def test_partition_parameters(dg, device, alpha, beta, force):
    g = small.random_graph(300, 0.02, seed=9)
    plan = dg.Plan(*to_dev(g, device), seed=1, walks_per_node=8, walk_len=4, alpha=alpha,
                   beta=beta, force_mode=force)
    assert_plan_matches(dg, plan, g, 1, 8, 4, alpha, beta, force)


ADAPTIVE_TINY = {
    # deterministic walks: Var(N) = Var(D) (alpha 1/2) and Var(N) = 4 Var(D) (alpha 4/5)
    "pairs": lambda: small.from_rows([[1], [0], [3], [2]] + [[] for _ in range(7)]),
    "triangles": lambda: small.from_rows([[1], [2], [0], [4], [5], [3]] + [[] for _ in range(5)]),
    "edgeless_bare": lambda: small.edgeless(9, self_loops=False, normalise=False),
    "self_loops_only": lambda: small.from_rows([[0] * 3, [1], [2] * 5, [3] * 2]),
}


@pytest.mark.parametrize("name", sorted(TINY) + sorted(ADAPTIVE_TINY))
@pytest.mark.parametrize("q", [1024, 7, 65535])
def test_adaptive_alpha_bitexact_tiny(dg, device, name, q):
    g = (TINY.get(name) or ADAPTIVE_TINY[name])()
    alpha = (dg.ALPHA_ADAPTIVE, q)
    plan = dg.Plan(*to_dev(g, device), seed=7, walks_per_node=8, walk_len=4, alpha=alpha)
    ref = assert_plan_matches(dg, plan, g, 7, 8, 4, alpha)
    if name == "pairs":
        assert ref["alpha"][0] == q // 2
    elif name == "triangles":
        assert ref["alpha"][0] == 4 * q // 5


@pytest.mark.parametrize("name", sorted(TINY) + sorted(ADAPTIVE_TINY))
@pytest.mark.parametrize("q", [1024, 7, 65535])
def test_balanced_alpha_bitexact_tiny(dg, device, name, q):
    g = (TINY.get(name) or ADAPTIVE_TINY[name])()
    alpha = (dg.ALPHA_BALANCED, q)
    plan = dg.Plan(*to_dev(g, device), seed=7, walks_per_node=8, walk_len=4, alpha=alpha)
    ref = assert_plan_matches(dg, plan, g, 7, 8, 4, alpha)
    if name == "pairs":
        assert ref["alpha"][0] == q // 2
    elif name == "triangles":
        assert ref["alpha"][0] == q // 3


@pytest.mark.parametrize("cfg", ["c1", "c2"])
@pytest.mark.parametrize("marker", [0xFFFFFFFF, 0xFFFFFFFE])
def test_adaptive_alpha_bitexact_configs(dg, device, cfg, marker):
    w = configs.WORKLOADS[cfg]
    g = configs.load_graph(cfg)
    alpha = (marker, 1024)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps,
                   alpha=alpha)
    assert_plan_matches(dg, plan, g, 0, w.walks, w.steps, alpha)


@pytest.mark.parametrize("cfg", ["c1", "c2"])
def test_partition_bitexact_configs(dg, device, cfg):
    w = configs.WORKLOADS[cfg]
    g = configs.load_graph(cfg)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    ref = assert_plan_matches(dg, plan, g, 0, w.walks, w.steps)
    assert 0 < ref["n_sparse"] < g.n


@pytest.mark.parametrize("k,d", [(4, 3), (1, 1)])
def test_bad_csr_rejected(dg, device, k, d):
    """Columns are checked by the successor pass where it runs (walks of k d >= 2 nnz / n steps
    per node: 4 x 3 here) and by the validation otherwise (1 x 1)."""
    g = small.random_graph(20, 0.2, seed=3)
    assert (20 * k * d >= 2 * g.nnz) == (k * d == 12)
    rp, c, v = to_dev(g, device)
    for bad in (20, -1, 1 << 30):                    # columns out of range
        c_bad = c.clone()
        c_bad[3] = bad
        with pytest.raises(dg.DualGCNError) as e:
            dg.Plan(rp, c_bad, v, walks_per_node=k, walk_len=d)
        assert e.value.status == dg.ERR_BAD_CSR
    rp_bad = rp.clone()
    rp_bad[5] = rp_bad[6] + 1                        # not monotone
    with pytest.raises(dg.DualGCNError) as e:
        dg.Plan(rp_bad, c, v, walks_per_node=k, walk_len=d)
    assert e.value.status == dg.ERR_BAD_CSR


# ---------------------------------------------------------------- SpMM

@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("force", ["auto", "sparse", "dense"])
@pytest.mark.parametrize("F", [1, 3, 16, 17, 64, 128, 256])
def test_spmm_tiny(dg, device, name, force, F):
    g = TINY[name]()
    X = dense.features_normal(g.n, F, seed=F, stream_id=21)
    plan = dg.Plan(*to_dev(g, device), seed=2, walks_per_node=8, walk_len=4, force_mode=force)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y, Yr, B, what=f"{name} F={F} {force}")


@pytest.mark.parametrize("F", [512, 320, 1000])
def test_spmm_wide_features(dg, device, F):
    g = small.random_graph(150, 0.05, seed=4)
    X = dense.features_normal(g.n, F, seed=1, stream_id=22)
    plan = dg.Plan(*to_dev(g, device), seed=2, walks_per_node=4, walk_len=3)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y, Yr, B, what=f"F={F}")


def test_spmm_poison_and_determinism(dg, device):
    g = configs.load_graph("c1")
    X = torch.from_numpy(configs.load_features("c1")).to(device)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4)
    for force in ["auto", "sparse", "dense"]:
        p = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4, force_mode=force)
        Y1 = torch.full_like(X, float("nan"))
        dg.spmm(p, X, Y1)
        Y2 = torch.full_like(X, float("nan"))
        dg.spmm(p, X, Y2)
        torch.cuda.synchronize()
        assert torch.isfinite(Y1).all()
        assert torch.equal(Y1, Y2)
    del plan


def test_spmm_split_rows_repeat_calls(dg, device):
    """A hub row split over several workgroups: counters are reset between calls."""
    g = small.star(20000, self_loops=True, normalise=True)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=4, walk_len=3)
    info = plan.info()
    # a matrix of about 60,000 entries keeps the largest chunk, 4096 entries
    hub = int(np.diff(g.rowptr).max())                  # 20,001 entries: 5 parts
    assert info["dense_chunk"] == 4096
    assert info["n_split_rows"] == 1 and info["n_split_parts"] == -(-hub // 4096) == 5
    Yr = None
    for F in (128, 64, 128, 17):
        X = dense.features_normal(g.n, F, seed=F, stream_id=23)
        Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
        Yr, B = oracle.spmm(g, X)
        assert_spmm_close(Y, Yr, B, what=f"star F={F}")


def test_spmm_dense_chunk_2048(dg, device):
    """A matrix of 4-8M entries splits its dense rows into 2048-entry parts: 2^19 + 5 nodes of
    about 9 entries each plus 24 hub rows, 12 of about 1,500 entries (one wavefront each) and
    12 of 3,000-9,000 (2 to 5 parts); every row against the oracle, F = 64 and a ragged
    F = 37."""
    from graphgen.csr import Graph, csr_from_pairs, normalised_values
    n = (1 << 19) + 5
    gen = np.random.Generator(np.random.Philox(key=np.array([41, 3], dtype=np.uint64)))
    a, b = gen.integers(0, n, 4 * n), gen.integers(0, n, 4 * n)
    hubs = gen.choice(n, 24, replace=False)
    ha = np.repeat(hubs, [1500] * 12 + [3000, 5000, 8000, 9000] * 3)
    src, dst = np.concatenate([a, ha]), np.concatenate([b, gen.integers(0, n, ha.size)])
    keep = src != dst
    src, dst = src[keep], dst[keep]
    rowptr, col = csr_from_pairs(n, np.concatenate([src, dst, np.arange(n)]),
                                 np.concatenate([dst, src, np.arange(n)]))
    g = Graph(n=n, rowptr=rowptr, col=col, val=normalised_values(rowptr, col), meta={"kind": "hubs"})
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=4, walk_len=3)
    info = plan.info()
    assert (1 << 22) <= g.nnz < (1 << 23) and info["dense_chunk"] == 2048
    assert info["n_split_rows"] == 12
    for F in (64, 37):
        X = dense.features_normal(n, F, seed=F, stream_id=29)
        Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
        Yr, B = oracle.spmm(g, X)
        assert_spmm_close(Y, Yr, B, what=f"chunk 2048 F={F}")
    plan.destroy()


@pytest.mark.parametrize("cfg", ["c1", "c2"])
def test_spmm_configs_full(dg, device, cfg):
    w = configs.WORKLOADS[cfg]
    g = configs.load_graph(cfg)
    X = configs.load_features(cfg)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    # c1 (69,632 entries) keeps 4096-entry parts (no row is split); c2 (1,310,720 entries)
    # splits its 154 rows of 512 entries or more into 512-entry parts
    info = plan.info()
    assert (info["dense_chunk"], info["n_split_rows"]) == {"c1": (4096, 0), "c2": (512, 154)}[cfg]
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y, Yr, B, what=cfg)


@pytest.mark.parametrize("alpha,force", [((1, 2), "auto"), ((0, 1), "auto"), ((1, 1), "auto"),
                                         ((1, 2), "sparse"), ((1, 2), "dense"),
                                         ((0xFFFFFFFF, 1024), "auto"), ((0xFFFFFFFE, 1024), "auto")])
def test_ablation_variants_c2(dg, device, alpha, force):
    """Every partition variant of the ablation: its plan matches the oracle and its SpMM
    (with the variant's schedule) matches the plan-independent oracle product."""
    w = configs.WORKLOADS["c2"]
    g = configs.load_graph("c2")
    X = configs.load_features("c2")
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps,
                   alpha=alpha, force_mode=force)
    assert_plan_matches(dg, plan, g, 0, w.walks, w.steps, alpha, (1, 2),
                        {"auto": 0, "sparse": 1, "dense": 2}[force])
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y, Yr, B, what=f"c2 alpha={alpha} {force}")


@pytest.mark.parametrize("k,d", [(50, 30), (16, 30), (50, 5)])
def test_paper_walk_parameters_c1(dg, device, k, d):
    """The paper's preprocessing uses 50 walks of 30 steps per node: bit-exact patterns and plan."""
    g = configs.load_graph("c1")
    rp, c, v = to_dev(g, device)
    P = dg.arw_patterns(rp, c, v, seed=3, walks_per_node=k, walk_len=d).cpu().numpy()
    assert np.array_equal(P, oracle.patterns(g, 3, k, d))
    plan = dg.Plan(rp, c, v, seed=3, walks_per_node=k, walk_len=d)
    assert_plan_matches(dg, plan, g, 3, k, d)


@pytest.mark.parametrize("k,d", [(1, 1), (3, 8), (2, 9), (128, 3), (129, 2), (256, 2), (300, 9),
                                 (7, 32), (5, 33)])
def test_walk_sum_lane_layouts_c1(dg, device, k, d):
    """Every lane layout of the partition's walk sums, bit-exact: one lane per node, a node's
    last lane with one walk (k odd), up to 64 lanes summed inside a wavefront, nodes whose
    lanes span wavefronts (k = 129, 256, 300), walks of up to 32 steps in lockstep, and the
    one-walk-per-lane kernel beyond; on c1 both with and without successor records
    (k d below and above twice the entries per node)."""
    g = configs.load_graph("c1")
    plan = dg.Plan(*to_dev(g, device), seed=5, walks_per_node=k, walk_len=d)
    assert_plan_matches(dg, plan, g, 5, k, d)
    plan.destroy()


def _sample_rows(g, plan_info_perm, n_sparse, count, seed):
    """Random rows plus the heaviest dense rows and the rows around the region boundary."""
    gen = np.random.default_rng(seed)
    rnd = gen.choice(g.n, size=min(count, g.n), replace=False)
    heavy = plan_info_perm[-min(64, g.n):]
    edge = plan_info_perm[max(0, n_sparse - 32):min(g.n, n_sparse + 32)]
    return np.unique(np.concatenate([rnd, heavy, edge])).astype(np.int32)


@pytest.mark.parametrize("cfg", ["c3"])
def test_config_partition_and_sampled_spmm(dg, device, cfg):
    w = configs.WORKLOADS[cfg]
    g = configs.load_graph(cfg)
    X = configs.load_features(cfg)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    ref = assert_plan_matches(dg, plan, g, 0, w.walks, w.steps)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    rows = _sample_rows(g, ref["perm"], ref["n_sparse"], 20000, seed=1)
    Yr, B = oracle.spmm(g, X, rows)
    assert_spmm_close(Y[rows], Yr, B, what=cfg)


@pytest.mark.parametrize("F", [16, 64, 128, 17])
def test_spmm_act_relu(dg, device, F):
    g = small.random_graph(400, 0.02, seed=12)
    X = dense.features_normal(g.n, F, seed=F, stream_id=28)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device), relu=True).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert (Y >= 0).all()
    assert_spmm_close(Y, np.maximum(Yr, 0.0), B, what=f"relu F={F}")


def _bf16(a):
    """float32 -> bfloat16 (nearest-even) -> float64, done in numpy."""
    u = np.asarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("fin,fout", [(32, 32), (256, 128), (128, 64), (96, 160), (1024, 32),
                                      (256, 256), (64, 256)])
def test_update_alone(dg, device, fin, fout):
    n = 777                                       # ragged against 128-row tiles
    X = dense.features_normal(n, fin, seed=fin, stream_id=29)
    W = dense.glorot(fin, fout, seed=fout, stream_id=30)
    T = dg.update(torch.from_numpy(X).to(device), torch.from_numpy(W).to(device)).cpu().numpy()
    Tr, BT = oracle.xw(X, W)
    assert_spmm_close(T, Tr, BT, tol=GCN_TOL, what=f"update {fin}->{fout}")
    # with both operands rounded to bf16 in numpy the product is reproduced to float32 rounding
    assert np.max(np.abs(T - _bf16(X) @ _bf16(W)) / (BT + 1e-30)) < 1e-5


def _bf16_t(t):
    """torch float32 -> bfloat16 (nearest-even) -> float64 numpy, done with integer ops."""
    return _bf16(t.cpu().numpy())


@pytest.mark.parametrize("F", [128, 64, 16, 12])
def test_spmm_bf16_output_is_rounded_fp32(dg, device, F):
    """DUALGCN_OUT_BF16 stores exactly the nearest-even bfloat16 of the float32 result."""
    g = small.random_graph(500, 0.03, seed=13)
    X = torch.from_numpy(dense.features_normal(g.n, F, seed=F, stream_id=32)).to(device)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4)
    for relu in (False, True):
        Y32 = dg.spmm(plan, X, relu=relu)
        Y16 = dg.spmm(plan, X, relu=relu, out_bf16=True)
        assert Y16.dtype == torch.bfloat16
        assert np.array_equal(Y16.float().cpu().numpy().astype(np.float64), _bf16_t(Y32))


def test_update_bf16_input_is_the_rounding_of_fp32_input(dg, device):
    X = dense.features_normal(777, 128, seed=5, stream_id=33)
    W = dense.glorot(128, 64, seed=5, stream_id=34)
    Xd, Wd = torch.from_numpy(X).to(device), torch.from_numpy(W).to(device)
    T32 = dg.update(Xd, Wd)
    T16 = dg.update(Xd.to(torch.bfloat16), Wd)       # torch's conversion is nearest-even too
    assert torch.equal(T32, T16)


def test_two_layers_through_bf16_intermediate_are_bit_identical(dg, device):
    """Layer 1 writing its output in bfloat16 and layer 2 reading it gives the same bits as
    the float32 intermediate, because the update rounds its input to bfloat16 anyway."""
    g = configs.load_graph("c2")
    X = torch.from_numpy(dense.features_normal(g.n, 256, seed=0, stream_id=27)).to(device)
    W1 = torch.from_numpy(dense.glorot(256, 128, seed=0, stream_id=4)).to(device)
    W2 = torch.from_numpy(dense.glorot(128, 64, seed=0, stream_id=5)).to(device)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=16, walk_len=5)
    H32 = dg.gcn_layer(plan, X, W1, relu=True)
    Y32 = dg.gcn_layer(plan, H32, W2)
    H16 = dg.gcn_layer(plan, X, W1, relu=True, out_bf16=True)
    Y16 = dg.gcn_layer(plan, H16, W2)
    assert H16.dtype == torch.bfloat16 and torch.equal(H16.float(), H32.to(torch.bfloat16).float())
    assert torch.equal(Y16, Y32)
    # the split entry points give the same bits
    T1 = dg.update(X, W1)
    H = dg.spmm(plan, T1, relu=True, out_bf16=True)
    Y = dg.spmm(plan, dg.update(H, W2))
    assert torch.equal(Y, Y32)


# ---------------------------------------------------------------- GCN layer (bf16 MFMA)

@pytest.mark.parametrize("fin,fout", [(32, 32), (64, 32), (256, 128), (128, 64), (96, 160)])
@pytest.mark.parametrize("relu", [False, True])
def test_gcn_layer_small(dg, device, fin, fout, relu):
    g = small.random_graph(333, 0.02, seed=7)
    X = dense.features_normal(g.n, fin, seed=fin, stream_id=24)
    W = dense.glorot(fin, fout, seed=fout, stream_id=25)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4)
    Y = dg.gcn_layer(plan, torch.from_numpy(X).to(device), torch.from_numpy(W).to(device),
                     relu=relu).cpu().numpy()
    Yr, BY = oracle.gcn_layer(g, X, W, relu=relu)
    assert_spmm_close(Y, Yr, BY, tol=GCN_TOL, what=f"gcn {fin}->{fout}")


def test_gcn_layer_identity_graph_is_xw(dg, device):
    """Edgeless graph: A = I, so the layer is the bf16 product itself (ragged n)."""
    g = small.edgeless(1000)
    X = dense.features_normal(g.n, 256, seed=3, stream_id=26)
    W = dense.glorot(256, 128, seed=3)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=2, walk_len=2)
    Y = dg.gcn_layer(plan, torch.from_numpy(X).to(device), torch.from_numpy(W).to(device)).cpu().numpy()
    T, BT = oracle.xw(X, W)
    assert_spmm_close(Y, T, BT, tol=GCN_TOL, what="xw")
    # the bf16 rounding of both operands, done here in numpy, reproduces it much closer
    assert np.max(np.abs(Y - _bf16(X) @ _bf16(W)) / (BT + 1e-30)) < 1e-5


def test_gcn_two_layer_c2_graph(dg, device):
    g = configs.load_graph("c2")
    X = dense.features_normal(g.n, 256, seed=0, stream_id=27)
    W1 = dense.glorot(256, 128, seed=0, stream_id=4)
    W2 = dense.glorot(128, 64, seed=0, stream_id=5)
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=16, walk_len=5)
    H = dg.gcn_layer(plan, torch.from_numpy(X).to(device), torch.from_numpy(W1).to(device), relu=True)
    Y = dg.gcn_layer(plan, H, torch.from_numpy(W2).to(device)).cpu().numpy()
    rows = np.random.default_rng(3).choice(g.n, 300, replace=False).astype(np.int32)
    Yr, bound = oracle.gcn_forward_rows(g, X, [W1, W2], rows)
    assert_spmm_close(Y[rows], Yr, bound, tol=GCN_TOL, what="2-layer")


def test_plan_used_right_away_on_other_streams(dg, device):
    """The partition returns with its sorted copy still queued on its stream; SpMMs launched
    at once on other streams (no synchronisation by the caller) must wait for it."""
    g = configs.load_graph("c2")
    rp, c, v = to_dev(g, device)
    X = torch.from_numpy(dense.features_normal(g.n, 64, seed=3, stream_id=45)).to(device)
    W = torch.from_numpy(dense.glorot(64, 32, seed=6)).to(device)
    ref_plan = dg.Plan(rp, c, v, seed=0, walks_per_node=16, walk_len=5)
    torch.cuda.synchronize()
    Y_ref = dg.spmm(ref_plan, X)
    T_ref = dg.spmm_update(ref_plan, X, W, relu=True)
    torch.cuda.synchronize()
    build, use = torch.cuda.Stream(device=device), torch.cuda.Stream(device=device)
    for _ in range(3):
        plan = dg.Plan(rp, c, v, seed=0, walks_per_node=16, walk_len=5, stream=build)
        with torch.cuda.stream(use):
            Y = dg.spmm(plan, X)
            T = dg.spmm_update(plan, X, W, relu=True)
        use.synchronize()
        assert torch.equal(Y, Y_ref) and torch.equal(T, T_ref)
        plan.destroy()
    ref_plan.destroy()


def test_destroy_waits_for_launches_on_other_streams(dg, device):
    """Destroying a plan while SpMMs that use it are still queued on another stream: the plan's
    memory is reused only after them (a new plan built at once takes the cached block)."""
    g = configs.load_graph("c2")
    rp, c, v = to_dev(g, device)
    X = torch.from_numpy(dense.features_normal(g.n, 256, seed=8, stream_id=46)).to(device)
    ref_plan = dg.Plan(rp, c, v, seed=0, walks_per_node=16, walk_len=5)
    Y_ref = dg.spmm(ref_plan, X)
    torch.cuda.synchronize()
    ref_plan.destroy()
    use = torch.cuda.Stream(device=device)
    for _ in range(2):
        plan = dg.Plan(rp, c, v, seed=0, walks_per_node=16, walk_len=5)
        torch.cuda.synchronize()
        with torch.cuda.stream(use):
            Ys = [dg.spmm(plan, X) for _ in range(4)]
        plan.destroy()                            # must wait for the four launches
        # same size (the cache hands it the block just released), another processing order
        other = dg.Plan(rp, c, v, seed=1, walks_per_node=16, walk_len=5, force_mode="dense")
        use.synchronize()
        for Y in Ys:
            assert torch.equal(Y, Y_ref)
        other.destroy()
