"""GPU parity of the causal prefill attention with score seeding (run on an
MI355X) against the oracle: outputs and seeded scores within
1e-3 + 2e-3 |ref| elementwise, on ragged lengths, every group size, both head
dims, chunks with existing scores, empty query sets and the Llama-3-8B prompt
shape; bad sizes are flagged and leave the cache untouched; repeated calls
are bit-identical.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L

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


class Case:
    """A two-layer cache; layer `layer` holds the prompt rows, scores s_init."""

    def __init__(self, D, G, HK, lengths, qlens, seed, s_init=False, layer=1):
        self.rng = np.random.default_rng(seed)
        rng = self.rng
        self.D, self.G, self.HK, self.layer = D, G, HK, layer
        self.lengths, self.qlens = list(lengths), list(qlens)
        self.B = len(lengths)
        self.c = L.LetheCache(2, [n + 3 for n in lengths], HK * G, HK, D, dtype="bf16", device=DEV)
        c = self.c
        self.K, self.V, self.s0 = {}, {}, {}
        for b, n in enumerate(lengths):
            for h in range(HK):
                r0, _ = c.seg_rows(b, h)
                u = rng.standard_normal(D).astype(np.float32)
                K = rng.standard_normal((n, D)).astype(np.float32) + \
                    0.4 * rng.pareto(1.3, size=(n, 1)).astype(np.float32) * u[None]
                V = rng.standard_normal((n, D)).astype(np.float32)
                Kt = torch.from_numpy(K).to(DEV).to(torch.bfloat16)
                Vt = torch.from_numpy(V).to(DEV).to(torch.bfloat16)
                c.k[layer, r0:r0 + n] = Kt
                c.v[layer, r0:r0 + n] = Vt
                s = rng.random(n).astype(np.float32) * 3 if s_init else np.zeros(n, np.float32)
                c.score[layer, r0:r0 + n] = torch.from_numpy(s).to(DEV)
                self.K[b, h], self.V[b, h], self.s0[b, h] = f32(Kt), f32(Vt), s
            c.len[layer, b] = n
            c.len[1 - layer, b] = 0
        # Sentinel scores in the other layer and past the live rows.
        c.score[1 - layer].fill_(7.0)
        self.rows = int(sum(qlens))
        starts = np.concatenate([[0], np.cumsum(qlens)[:-1]]).astype(np.int64)
        self.q_start = torch.from_numpy(starts).to(DEV)
        self.q_len = torch.tensor(qlens, dtype=torch.int32, device=DEV)
        self.starts = starts
        q = rng.standard_normal((max(self.rows, 1), HK * G, D)).astype(np.float32)
        self.q = torch.from_numpy(q[:self.rows]).to(DEV).to(torch.bfloat16).contiguous()
        self.out = torch.full((self.rows, HK * G, D), np.nan, dtype=torch.float32, device=DEV)
        self.ws = c.prefill_workspace(self.rows)
        torch.cuda.synchronize()

    def run(self, max_q=None, max_kv=None, scale=0.0):
        L.prefill_attn_score(self.c, self.layer, self.q, self.q_start, self.q_len,
                             max(self.qlens) if max_q is None else max_q,
                             max(self.lengths) if max_kv is None else max_kv, scale, self.out, self.ws)
        torch.cuda.synchronize()

    def check(self, seqs=None, heads=None):
        c, G, D = self.c, self.G, self.D
        out = f32(self.out)
        qh = f32(self.q)
        scale = 1.0 / math.sqrt(D)
        for b in (range(self.B) if seqs is None else seqs):
            n, ql, r = self.lengths[b], self.qlens[b], int(self.starts[b])
            for h in (range(self.HK) if heads is None else heads):
                o, s = oracle.prefill(qh[r:r + ql, h * G:(h + 1) * G], self.K[b, h], self.V[b, h],
                                      self.s0[b, h].astype(np.float64), scale)
                what = "D%d G%d b%d h%d n%d q%d" % (D, G, b, h, n, ql)
                close(out[r:r + ql, h * G:(h + 1) * G], o, "out " + what)
                r0, r1 = c.seg_rows(b, h)
                close(f32(c.score[self.layer, r0:r0 + n]), s, "scores " + what)
                tail = f32(c.score[self.layer, r0 + n:r1])
                assert np.all(tail == 0.0), "rows past len touched " + what
        assert np.all(f32(c.score[1 - self.layer]) == 7.0)
        assert int(c.dev_status[0]) == 0


LENGTHS = [1, 31, 32, 33, 100, 257, 600]


@pytest.mark.parametrize("D,G,HK", [(128, 4, 2), (64, 2, 3), (128, 7, 1), (128, 8, 2), (128, 1, 4), (64, 5, 1)])
def test_prefill_full_prompts(D, G, HK):
    note("prefill D=%d G=%d HK=%d" % (D, G, HK))
    cs = Case(D, G, HK, LENGTHS, LENGTHS, seed=D + 10 * G + HK)
    cs.run()
    cs.check()


def test_prefill_chunks_with_existing_scores_and_empty_sets():
    note("prefill chunks")
    cs = Case(128, 4, 2, [300, 513, 64, 90, 5], [100, 1, 64, 0, 0], seed=3, s_init=True)
    cs.run()
    cs.check()


def test_prefill_chunked_equals_whole_on_device():
    note("prefill chunked = whole")
    n = 700
    whole = Case(128, 4, 2, [n], [n], seed=4)
    whole.run()
    # Same cache contents, prompt fed as two chunks: rows [0, 300) then the rest.
    ch = Case(128, 4, 2, [n], [n], seed=4)
    c = ch.c
    cut = 300
    c.len[ch.layer, 0] = cut
    q1 = ch.q[:cut].contiguous()
    out1 = torch.empty((cut, 8, 128), dtype=torch.float32, device=DEV)
    ws = c.prefill_workspace(n)
    L.prefill_attn_score(c, ch.layer, q1, torch.zeros(1, dtype=torch.int64, device=DEV),
                         torch.tensor([cut], dtype=torch.int32, device=DEV), cut, cut, 0.0, out1, ws)
    c.len[ch.layer, 0] = n
    q2 = ch.q[cut:].contiguous()
    out2 = torch.empty((n - cut, 8, 128), dtype=torch.float32, device=DEV)
    L.prefill_attn_score(c, ch.layer, q2, torch.zeros(1, dtype=torch.int64, device=DEV),
                         torch.tensor([n - cut], dtype=torch.int32, device=DEV), n - cut, n, 0.0, out2, ws)
    torch.cuda.synchronize()
    close(f32(torch.cat([out1, out2])), f32(whole.out), "chunked out")
    for h in range(2):
        r0, _ = c.seg_rows(0, h)
        close(f32(c.score[ch.layer, r0:r0 + n]), f32(whole.c.score[whole.layer, r0:r0 + n]), "chunked scores")


def test_prefill_is_deterministic():
    note("prefill determinism")
    cs = Case(128, 4, 2, [900, 77], [900, 77], seed=5)
    cs.run()
    out1 = cs.out.clone()
    sc1 = cs.c.score.clone()
    for b, n in enumerate(cs.lengths):
        for h in range(cs.HK):
            r0, _ = cs.c.seg_rows(b, h)
            cs.c.score[cs.layer, r0:r0 + n] = 0.0
    cs.run()
    assert torch.equal(out1.view(torch.int32), cs.out.view(torch.int32))
    assert torch.equal(sc1.view(torch.int32), cs.c.score.view(torch.int32))


def test_prefill_bad_sizes_are_flagged_and_skipped():
    note("prefill bad sizes")
    cs = Case(128, 4, 1, [50, 60, 70], [50, 61, 70], seed=6)   # q_len > len for b = 1
    cs.run(max_q=70, max_kv=70)
    assert int(cs.c.dev_status[0]) & L.DEV_BAD_LAYOUT
    r0, _ = cs.c.seg_rows(1, 0)
    assert np.all(f32(cs.c.score[cs.layer, r0:r0 + 60]) == 0.0)
    assert np.isnan(f32(cs.out[50:111])).all()
    cs.c.dev_status.zero_()
    cs.check(seqs=[0, 2])
    # A bound below a sequence's length also skips it.
    cs2 = Case(64, 2, 1, [40, 80], [40, 80], seed=7)
    cs2.run(max_q=80, max_kv=79)
    assert int(cs2.c.dev_status[0]) & L.DEV_BAD_LAYOUT
    r0, _ = cs2.c.seg_rows(1, 0)
    assert np.all(f32(cs2.c.score[cs2.layer, r0:r0 + 80]) == 0.0)
    cs2.c.dev_status.zero_()
    cs2.check(seqs=[0])


@pytest.mark.timeout(600)
def test_prefill_llama8b_prompt_full_size():
    """Llama-3-8B shapes at a 2048-token prompt, batch 8: every segment's
    seeded mass equals G * qlen; two sampled segments against the oracle."""
    note("prefill llama8b full size")
    B, HK, G, D, T = 8, 8, 4, 128, 2048
    cs = Case(D, G, HK, [T] * B, [T] * B, seed=8)
    cs.run()
    c = cs.c
    for b in range(B):
        for h in range(HK):
            r0, _ = c.seg_rows(b, h)
            mass = float(c.score[cs.layer, r0:r0 + T].double().sum())
            assert abs(mass - G * T) <= 1e-3 * G * T, (b, h, mass)
    assert np.isfinite(f32(cs.out)).all()
    cs.check(seqs=[0], heads=[0])
    cs.check(seqs=[B - 1], heads=[HK - 1])


def test_prefill_then_decode_and_prune():
    """Prompt prefill seeds the scores, decode steps decay and extend them
    (with their deferred updates), then a prune round: the device against the
    oracle's composition of the same steps."""
    note("prefill -> decode -> prune")
    D, G, HK = 128, 4, 2
    lengths = [300, 701]
    cs = Case(D, G, HK, lengths, lengths, seed=9)
    cs.run()
    c, lay = cs.c, cs.layer
    B = len(lengths)
    orc = oracle.OracleCache(2, B, HK * G, HK, D)
    qh = f32(cs.q)
    scale = 1.0 / math.sqrt(D)
    for b, n in enumerate(lengths):
        r = int(cs.starts[b])
        for h in range(HK):
            _, s = oracle.prefill(qh[r:r + n, h * G:(h + 1) * G], cs.K[b, h], cs.V[b, h], None, scale)
            orc.set_segment(lay, b, h, cs.K[b, h], cs.V[b, h], s)
    rng = np.random.default_rng(10)
    ws = c.workspace(L.OP_DECODE)
    gamma = 0.9
    for t in range(3):
        q = torch.from_numpy(rng.standard_normal((B, HK * G, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
        kn = torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
        vn = torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV).to(torch.bfloat16)
        out = torch.empty((B, HK * G, D), dtype=torch.float32, device=DEV)
        L.decode_attn_score(c, lay, q, kn, vn, gamma, 0.0, out, ws)
        ref = orc.decode_step(lay, f32(q), f32(kn), f32(vn), gamma, scale)
        torch.cuda.synchronize()
        close(f32(out), ref, "decode out t%d" % t)
    c.flush()
    torch.cuda.synchronize()
    for b, n in enumerate(lengths):
        for h in range(HK):
            r0, _ = c.seg_rows(b, h)
            close(f32(c.score[lay, r0:r0 + n + 3]), orc.s[lay][b][h], "scores b%d h%d" % (b, h))
    # Prune to 40% per layer, recent 32: masks bit-exact given the device's scores.
    gb = torch.tensor([int(0.4 * (n + 3)) * 2 for n in lengths], dtype=torch.int64, device=DEV)
    S = torch.empty((B, 2), dtype=torch.float32, device=DEV)
    bud = torch.empty((B, 2), dtype=torch.int32, device=DEV)
    L.layer_sparsity(c, gb, 32, 0, None, S, bud)
    keep = torch.zeros((2, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    L.rasr_select(c, bud, 32, 0, keep)
    torch.cuda.synchronize()
    bh = bud.cpu().numpy()
    kh = keep.cpu().numpy()
    for b, n in enumerate(lengths):
        for h in range(HK):
            r0, _ = c.seg_rows(b, h)
            want = oracle.rasr_select(f32(c.score[lay, r0:r0 + n + 3]), bh[b, lay], 32, 0)
            np.testing.assert_array_equal(kh[lay, r0:r0 + n + 3].astype(bool), want)
    L.kv_compact(c, keep, c.workspace(L.OP_COMPACT))
    torch.cuda.synchronize()
    assert [int(c.len[lay, b]) for b in range(B)] == [min(n + 3, int(bh[b, lay])) for b, n in enumerate(lengths)]
    assert int(c.dev_status[0]) == 0
