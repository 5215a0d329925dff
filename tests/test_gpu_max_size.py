"""The largest matrix the library accepts: nnz = 2^31 - 2^24 (just under the 2^31 - 2^16
bound), built on the device as a circulant (row r holds columns r + o mod n for 127
fixed offsets, value 1/127).  The partition must cover every row exactly once, and the
SpMM must match the closed form on every row (outputs poisoned with NaN before the call,
so a row no workgroup writes fails): entry indices near 2^31 exercise every 32-bit index
path of the kernels.  The fused layer junction runs on the same plan, every row checked
the same way.  The closed form Y[r] = (1/127) sum over the offsets of X[r + o] is
evaluated in float64 with plain torch gathers on the device, row chunk by row chunk."""
import numpy as np
import pytest
import torch

from graphgen import dense

pytestmark = pytest.mark.gpu

N = 1 << 24
DEG = 127
F = 4


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _x_value(c, f):
    return ((c * (f + 1)) % 97) / 97.0 - 0.5


CHUNK = 1 << 22                                       # rows per closed-form chunk


def _circulant_sums(X, offsets, r0, r1):
    """float64 sums over the offsets of X[r + o mod N] and of |X[r + o mod N]| for rows
    r0 .. r1 - 1 (X as stored, float32, promoted exactly)."""
    rows = torch.arange(r0, r1, device=X.device, dtype=torch.int64)
    s = torch.zeros((r1 - r0, X.shape[1]), dtype=torch.float64, device=X.device)
    a = torch.zeros_like(s)
    for o in offsets:
        xs = X[(rows + int(o)) % N].to(torch.float64)
        s += xs
        a += xs.abs()
    return s, a


def test_max_size_circulant(dg, device):
    offsets = np.unique(np.concatenate([[0], (np.arange(1, DEG) ** 3) % N]))[:DEG]
    assert offsets.size == DEG
    nnz = N * DEG
    assert nnz == 2 ** 31 - 2 ** 24
    off = torch.from_numpy(offsets.astype(np.int64)).to(device)
    rowptr = (torch.arange(N + 1, device=device, dtype=torch.int64) * DEG).to(torch.int32)
    col = torch.empty(nnz, dtype=torch.int32, device=device)
    step = 1 << 20                                   # rows per slice while building
    for r0 in range(0, N, step):
        rows = torch.arange(r0, min(N, r0 + step), device=device, dtype=torch.int64)
        c = torch.sort((rows[:, None] + off[None, :]) % N, dim=1).values
        col[r0 * DEG:(r0 + rows.numel()) * DEG] = c.reshape(-1).to(torch.int32)
        del c, rows
    val = torch.full((nnz,), 1.0 / DEG, dtype=torch.float32, device=device)
    plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=4, walk_len=3)
    info = plan.info()
    assert info["nnz"] == nnz and info["n_sparse"] + info["n_dense"] == N
    perm, S, K = plan.export()
    assert np.array_equal(np.sort(perm), np.arange(N, dtype=np.int32))
    assert S.min() >= 4 and S.max() <= 4 * 4
    Ks = K[perm]
    assert np.all(Ks[1:] >= Ks[:-1])
    # X[c, f] from a closed form; Y[r] = (1/127) sum over the offsets of X[r + o]
    cidx = torch.arange(N, device=device, dtype=torch.int64)
    X = torch.stack([(((cidx * (f + 1)) % 97).to(torch.float32) / 97.0 - 0.5) for f in range(F)], 1)
    X = X.contiguous()
    Y = torch.full((N, F), float("nan"), dtype=torch.float32, device=device)
    dg.spmm(plan, X, Y=Y)
    v32 = float(np.float32(1.0 / DEG))
    for r0 in range(0, N, CHUNK):                    # every row against the closed form
        r1 = min(N, r0 + CHUNK)
        s, a = _circulant_sums(X, offsets, r0, r1)
        err = (Y[r0:r1].to(torch.float64) - v32 * s).abs()
        ok = err <= 1e-5 * (v32 * a) + 1e-30          # False on NaN: an unwritten element
        assert bool(ok.all()), (r0, int((~ok).sum()), float(err.nan_to_num(float("inf")).max()))
        del s, a, err, ok
    rows = np.concatenate([np.random.default_rng(0).choice(N, 2000, replace=False), [0, N - 1]])
    Yh = Y[torch.from_numpy(rows).to(device)].cpu().numpy().astype(np.float64)
    for i, r in enumerate(rows):
        cs = (r + offsets) % N
        for f in range(F):
            xs = np.array([np.float32(_x_value(int(c), f)) for c in cs], dtype=np.float64)
            want = v32 * xs.sum()
            bound = v32 * np.abs(xs).sum()
            assert abs(Yh[i, f] - want) <= 1e-5 * bound + 1e-30, (r, f, Yh[i, f], want)
    del X, Y
    # the fused layer junction at the same size (F_in = F_out = 32, ReLU): bit-identical to
    # the two calls, and within the update's bound of the closed form on every row (and, from
    # host-side values, on the sampled rows)
    FI = 32
    X = torch.stack([(((cidx * (f + 1)) % 97).to(torch.float32) / 97.0 - 0.5) for f in range(FI)],
                    1).contiguous()
    W = dense.glorot(FI, FI, seed=11)
    Wd = torch.from_numpy(W).to(device)
    nan = float("nan")
    T = dg.spmm_update(plan, X, Wd, T=torch.full((N, FI), nan, dtype=torch.float32, device=device),
                       relu=True)
    Hb = dg.spmm(plan, X, Y=torch.full((N, FI), nan, dtype=torch.bfloat16, device=device),
                 relu=True, out_bf16=True)
    T2 = dg.update(Hb, Wd, T=torch.full((N, FI), nan, dtype=torch.float32, device=device))
    assert torch.equal(T, T2)                          # equal, hence no NaN left in either
    del Hb, T2
    W64d = Wd.to(torch.float64)
    for r0 in range(0, N, CHUNK):                    # every row of T within the update's bound
        r1 = min(N, r0 + CHUNK)
        s, a = _circulant_sums(X, offsets, r0, r1)
        H = torch.clamp(v32 * s, min=0.0)
        err = (T[r0:r1].to(torch.float64) - H @ W64d).abs()
        ok = err <= 1e-2 * ((H.abs() + v32 * a) @ W64d.abs())
        assert bool(ok.all()), (r0, int((~ok).sum()))
        del s, a, H, err, ok
    Th = T[torch.from_numpy(rows).to(device)].cpu().numpy().astype(np.float64)
    cs = (rows[:, None].astype(np.int64) + offsets[None, :]) % N              # (rows, DEG)
    xs = np.stack([((cs * (f + 1)) % 97) / 97.0 - 0.5 for f in range(FI)], 2)
    xs = xs.astype(np.float32).astype(np.float64)                             # X as stored
    H = np.maximum(v32 * xs.sum(1), 0.0)
    B = v32 * np.abs(xs).sum(1)
    W64 = W.astype(np.float64)
    err = np.abs(Th - H @ W64)
    assert np.all(err <= 1e-2 * ((np.abs(H) + B) @ np.abs(W64))), float(err.max())
    plan.destroy()
