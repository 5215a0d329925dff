"""dualgcn_weight_grad_noalloc (the weight gradient with its partial products in the
library's static device array, for callers that cannot allocate) against
dualgcn_weight_grad, through the C ABI: bit-identical dW and SGD step on two calls in a
row, the second smaller than the first, and shapes beyond the array refused."""
import numpy as np
import pytest
import torch

import oracle
from graphgen import dense

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _pair(device, n, fin, fout, seed, x_bf16, g_bf16):
    X = torch.from_numpy(dense.features_normal(n, fin, seed=seed)).to(device)
    G = torch.from_numpy(dense.features_normal(n, fout, seed=seed + 1, stream_id=7)).to(device)
    if x_bf16:
        X = X.to(torch.bfloat16)
    if g_bf16:
        G = G.to(torch.bfloat16)
    return X, G


def test_noalloc_weight_grad_matches_workspace_entry(dg, device):
    # c5's layer-1 shape first (n = 2^22, 256 -> 128), then a smaller product with other
    # widths and a ragged row count: each must equal dualgcn_weight_grad bit for bit
    cases = [(1 << 22, 256, 128, False, True), (4133, 128, 64, True, False)]
    for n, fin, fout, xbf, gbf in cases:
        print(f"[no-alloc] n={n} {fin}->{fout} x_bf16={xbf} g_bf16={gbf}", flush=True)
        X, G = _pair(device, n, fin, fout, fin + n % 97, xbf, gbf)
        want = dg.weight_grad(X, G)
        got = torch.full((fin, fout), float("nan"), dtype=torch.float32, device=device)
        dg.weight_grad_noalloc(X, G, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"dW differs from dualgcn_weight_grad at n={n} {fin}->{fout}"
        # and the oracle's bound (1e-2 of sum |x||g| for bfloat16 operands) on the small case
        if n < 10000:
            Xh = X.float().cpu().numpy()
            Gh = G.float().cpu().numpy()
            ref, B = oracle.weight_grad(Xh, Gh)
            assert np.all(np.abs(got.cpu().numpy().astype(np.float64) - ref) <= 1e-2 * B)
        del X, G, want, got
        torch.cuda.empty_cache()


def test_noalloc_sgd_step_matches_workspace_entry(dg, device):
    for n, fin, fout in ((70000, 256, 128), (333, 64, 32)):
        X, G = _pair(device, n, fin, fout, 11 + n, False, False)
        W0 = torch.from_numpy(dense.glorot(fin, fout, seed=3)).to(device)
        Wa, Wb = W0.clone(), W0.clone()
        dWa = dg.weight_grad(X, G, lr=0.05, W=Wa)
        dWb = torch.empty_like(dWa)
        dg.weight_grad_noalloc(X, G, dWb, lr=0.05, W=Wb)
        torch.cuda.synchronize()
        assert torch.equal(dWa, dWb) and torch.equal(Wa, Wb)


def test_noalloc_refuses_partials_beyond_the_array(dg, device):
    # 1024 x 256 partials are 1 MiB each: 65 chunks of 64 rows take 65 workgroups
    # (MI355X holds at least that many at once), 65 MiB > 64 MiB
    X, G = _pair(device, 64 * 65, 1024, 256, 5, True, True)
    dW = torch.zeros((1024, 256), dtype=torch.float32, device=device)
    with pytest.raises(dg.DualGCNError) as e:
        dg.weight_grad_noalloc(X, G, dW)
    assert e.value.status == dg.ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.count_nonzero(dW).item() == 0          # nothing was queued
    # 64 chunks fit exactly (64 MiB)
    X, G = X[:64 * 64], G[:64 * 64]
    dg.weight_grad_noalloc(X, G, dW)
    assert torch.equal(dW, dg.weight_grad(X, G))
