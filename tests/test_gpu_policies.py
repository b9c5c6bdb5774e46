"""GPU parity of the prune policies (run on an MI355X): Lethe, its head-shared
variant and the H2O / StreamingLLM / PyramidKV baselines, each a
parameterisation of the library's kernels (paper_2511_06029_amd/policies.py).

For every policy: decode steps with the policy's gamma against the oracle
(outputs and scores within 1e-3 + 2e-3 |ref|), then one prune round whose
budgets, keep masks and compacted lengths must equal the oracle's given the
device's scores and sparsities, plus what defines each baseline: H2O and
StreamingLLM give every layer the same budget, StreamingLLM keeps exactly its
sinks and window, PyramidKV's budgets above the protected rows follow its
linear progression.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L
from paper_2511_06029_amd import policies

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-3, 2e-3
DEV = "cuda"


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def close(gpu, ref, what):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = ~(np.abs(gpu - ref) <= ATOL + RTOL * np.abs(ref))
    if bad.any():
        i = np.flatnonzero(bad.ravel())[0]
        raise AssertionError("%s: %d mismatches, first at %d: gpu %r ref %r" %
                             (what, bad.sum(), i, gpu.ravel()[i], ref.ravel()[i]))


def f32(t):
    return t.detach().float().cpu().numpy()


@pytest.mark.parametrize("name", policies.POLICY_NAMES)
def test_policy_decode_and_prune_round(name):
    note("policy %s" % name)
    rng = np.random.default_rng(61)
    Ly, HQ, HK, D, steps = 4, 8, 2, 64, 3
    lengths = [300, 777, 1500] if name != "streaming" else [600, 600, 900]
    B = len(lengths)
    pol = policies.get(name, gamma=0.9, sink=2, beta=4.0)
    c = L.LetheCache(Ly, [n + steps for n in lengths], HQ, HK, D, dtype="bf16", device=DEV)
    orc = oracle.OracleCache(Ly, B, HQ, HK, D)
    for l in range(Ly):
        for b, n in enumerate(lengths):
            for h in range(HK):
                s0, _ = c.seg_rows(b, h)
                # Keys carry a per-layer bias direction so attention is peaked.
                u = rng.standard_normal(D).astype(np.float32)
                K = rng.standard_normal((n, D)).astype(np.float32) + np.outer(rng.pareto(1.5, n), u).astype(np.float32) * 0.3
                V = rng.standard_normal((n, D)).astype(np.float32)
                Kt = torch.from_numpy(K).to(DEV).to(torch.bfloat16)
                Vt = torch.from_numpy(V).to(DEV).to(torch.bfloat16)
                c.k[l, s0:s0 + n] = Kt
                c.v[l, s0:s0 + n] = Vt
                orc.set_segment(l, b, h, f32(Kt), f32(Vt))
            c.len[l, b] = n
    ws = c.workspace(L.OP_DECODE)
    scale = 1.0 / math.sqrt(D)
    for t in range(steps):
        for l in range(Ly):
            q = torch.from_numpy(rng.standard_normal((B, HQ, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
            kn = torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
            vn = torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
            out = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
            L.decode_attn_score(c, l, q, kn, vn, pol.gamma, 0.0, out, ws)
            ref = orc.decode_step(l, f32(q), f32(kn), f32(vn), pol.gamma, scale)
            torch.cuda.synchronize()
            close(f32(out), ref, "%s out t%d l%d" % (name, t, l))
    c.flush()
    torch.cuda.synchronize()
    n_now = [n + steps for n in lengths]
    for l in range(Ly):
        for b, n in enumerate(n_now):
            for h in range(HK):
                s0, _ = c.seg_rows(b, h)
                close(f32(c.score[l, s0:s0 + n]), orc.s[l][b][h], "%s scores l%d b%d h%d" % (name, l, b, h))

    # One prune round at a 40% budget (StreamingLLM: one budget for all).
    per_seq = [policies.per_layer_budget(0.4, n) for n in n_now]
    if pol.window_fills:
        per_seq = [min(per_seq)] * B
    rnd = policies.PruneRound(c, pol)
    recent = 16
    r, sk = rnd.budgets(per_seq, recent)
    torch.cuda.synchronize()
    S = rnd.S.cpu().numpy()
    bud = rnd.budget.cpu().numpy()
    s_in = pol.sparsity_in(Ly)
    for b in range(B):
        nl = np.full(Ly, n_now[b], np.int32)
        if s_in is None:
            want_S = np.array([orc.sparsity(l, b) for l in range(Ly)])
            assert np.all(np.abs(S[b] - want_S) <= 1e-6), (name, b)
            given = S[b]
        else:
            given = np.array(s_in, np.float32)
            np.testing.assert_array_equal(S[b], given)
        want, _ = oracle.budget_split(nl, given, r, sk, per_seq[b] * Ly)
        np.testing.assert_array_equal(bud[b], want, err_msg="%s budgets b%d" % (name, b))
        if pol.layer_budget == "uniform":
            assert (bud[b] == per_seq[b]).all()
        if pol.layer_budget == "pyramid":
            # The progression shapes what is left above every layer's
            # protected rows (recent + sink).
            f = min(n_now[b], r + sk)
            prog = np.array(oracle.pyramid_budgets(Ly, per_seq[b] * Ly - Ly * f, pol.beta)) + f
            assert np.all(np.abs(bud[b] - prog) <= 1.0), (bud[b], prog)
    rnd.select(r, sk)
    torch.cuda.synchronize()
    keep = rnd.keep.cpu().numpy()
    kept = {}
    for l in range(Ly):
        for b, n in enumerate(n_now):
            sh = []
            for h in range(HK):
                s0, _ = c.seg_rows(b, h)
                sh.append(f32(c.score[l, s0:s0 + n]))
            for h in range(HK):
                s0, _ = c.seg_rows(b, h)
                got = keep[l, s0:s0 + n].astype(bool)
                if pol.shared:
                    want = oracle.rasr_select_shared(np.stack(sh), bud[b, l], r, sk)
                else:
                    want = oracle.rasr_select(sh[h], bud[b, l], r, sk)
                np.testing.assert_array_equal(got, want, err_msg="%s keep l%d b%d h%d" % (name, l, b, h))
                if pol.window_fills:
                    win = np.zeros(n, bool)
                    win[:sk] = True
                    win[n - r:] = True
                    np.testing.assert_array_equal(got, win)
                kept[l, b] = int(got.sum())
    rnd.compact()
    torch.cuda.synchronize()
    lens = c.len.cpu().numpy()
    for (l, b), k in kept.items():
        assert lens[l, b] == k == min(n_now[b], bud[b, l])
    assert int(c.dev_status[0]) == 0
