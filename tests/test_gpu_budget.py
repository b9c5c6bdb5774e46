"""GPU parity of the layer budget split (lethe_layer_sparsity with given
sparsities, run on an MI355X): budgets bit-exact against the oracle for up to
256 layers (several layers per lane), ragged per-layer lengths, binding
caps, infeasible and nothing-to-prune sequences, and NaN or out-of-range
sparsities."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("Ly", [1, 7, 64, 65, 130, 256])
def test_budget_split_bit_exact(Ly):
    print("budget split L=%d" % Ly, flush=True)
    sys.stdout.flush()
    rng = np.random.default_rng(70 + Ly)
    B = 6
    cap = 3000
    c = L.LetheCache(Ly, [cap] * B, 2, 1, 64, dtype="bf16", device=DEV)
    n = rng.integers(0, cap + 1, size=(Ly, B)).astype(np.int32)
    n[:, 1] = rng.integers(0, 40, size=Ly)          # many layers below the floors
    n[0, 2] = 0
    c.len.copy_(torch.from_numpy(n).to(DEV))
    S = rng.random((B, Ly)).astype(np.float32)
    S[0, ::3] = np.nan
    S[3, :] = 0.5                                     # equal weights
    S[4, ::2] = np.float32(1.5)
    S[4, 1::2] = np.float32(-0.25)
    S[5, :] = rng.choice([0.0, 1.0, 0.999999, 1e-7], size=Ly).astype(np.float32)
    recent, sink = 24, 4
    tot = n.sum(axis=0).astype(np.int64)
    floors = np.minimum(n, recent + sink).sum(axis=0).astype(np.int64)
    G = np.array([tot[0] // 3, tot[1] + 5, floors[2] - 1, max(floors[3], tot[3] // 2),
                  floors[4] + 1, floors[5] + (tot[5] - floors[5]) // 7], np.int64)
    S_t = torch.from_numpy(S).to(DEV)
    out_S = torch.empty((B, Ly), dtype=torch.float32, device=DEV)
    bud = torch.empty((B, Ly), dtype=torch.int32, device=DEV)
    c.dev_status.zero_()
    L.layer_sparsity(c, torch.from_numpy(G).to(DEV), recent, sink, S_t, out_S, bud)
    torch.cuda.synchronize()
    got = bud.cpu().numpy()
    infeasible = False
    for b in range(B):
        want, inf = oracle.budget_split(n[:, b], S[b], recent, sink, G[b])
        infeasible |= inf
        np.testing.assert_array_equal(got[b], want, err_msg="L=%d b=%d" % (Ly, b))
    assert bool(int(c.dev_status[0]) & L.DEV_INFEASIBLE) == infeasible
    np.testing.assert_array_equal(out_S.cpu().numpy().view(np.uint32), S.view(np.uint32))
