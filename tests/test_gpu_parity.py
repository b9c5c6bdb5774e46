"""GPU parity of the HIP path against the oracle (run on an MI355X).

Every input comes from the seeded generators in ``workloads``; the oracle
sees the exact values the device holds (bf16 widened to fp32).  Tolerances:
attention outputs and scores |gpu - ref| <= 1e-3 + 2e-3 |ref| elementwise;
selections, budgets and compacted rows bit-exact when both sides get the same
score vectors (ties to the lower row, NaN last, +0 == -0).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L
from workloads import synth

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
    bad &= ~(np.isnan(gpu) & np.isnan(ref))
    if bad.any():
        i = np.flatnonzero(bad.ravel())[0]
        raise AssertionError("%s: %d mismatches, first at %d: gpu %r ref %r" %
                             (what, bad.sum(), i, gpu.ravel()[i], ref.ravel()[i]))


def host(t):
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


class Harness:
    """A device cache plus the oracle's logical copy of the same contents."""

    def __init__(self, L_, caps, HQ, HK, D, dtype):
        self.c = L.LetheCache(L_, caps, HQ, HK, D, dtype=dtype, device=DEV)
        self.orc = oracle.OracleCache(L_, len(caps), HQ, HK, D)
        self.dtype = dtype
        self.ws = self.c.workspace(L.OP_DECODE)

    def store(self, x):
        t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
        return t.to(DEV).to(self.c.tdtype)

    def fill(self, l, b, h, K, V, s=None):
        """K, V float32 arrays (rounded to the storage type first)."""
        n = K.shape[0]
        start, _ = self.c.seg_rows(b, h)
        Kt, Vt = self.store(K), self.store(V)
        self.c.k[l, start:start + n] = Kt
        self.c.v[l, start:start + n] = Vt
        if s is not None:
            self.c.score[l, start:start + n] = torch.from_numpy(np.asarray(s, np.float32)).to(DEV)
        self.orc.set_segment(l, b, h, host(Kt), host(Vt), None if s is None else np.asarray(s, np.float32))

    def set_len(self, l, b, n):
        self.c.len[l, b] = n

    def decode(self, l, q, k_new, v_new, gamma, scale):
        """q, k_new, v_new float32 arrays; returns (gpu out, oracle out)."""
        B, HQ, D = q.shape
        qt = self.store(q)
        kt = None if k_new is None else self.store(k_new)
        vt = None if v_new is None else self.store(v_new)
        out = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
        L.decode_attn_score(self.c, l, qt, kt, vt, gamma, scale, out, self.ws)
        ref = self.orc.decode_step(l, host(qt), None if kt is None else host(kt),
                                   None if vt is None else host(vt), gamma,
                                   scale if scale > 0 else 1 / math.sqrt(D))
        torch.cuda.synchronize()
        return host(out), ref

    def scores(self, l, b, h, n):
        """Current scores of a segment (applies a pending decode step first)."""
        self.c.flush()
        start, _ = self.c.seg_rows(b, h)
        return host(self.c.score[l, start:start + n])

    def check_scores(self, l):
        for b in range(self.c.B):
            n = int(self.c.len[l, b])
            assert n == self.orc.length(l, b), (l, b, n, self.orc.length(l, b))
            for h in range(self.c.HK):
                close(self.scores(l, b, h, n), self.orc.s[l][b][h], "scores l%d b%d h%d" % (l, b, h))


# ---------------------------------------------------------------------------
# Decode step
# ---------------------------------------------------------------------------

def test_tiny_case_end_to_end():
    """The small fp32 case: 512 cached rows, 16 decode steps, one prune to 256
    rows with a recent window of 32."""
    note("tiny case: decode x16")
    d = synth.tiny_case(seed=1)
    HQ, HK, D = 4, 2, 64
    H = Harness(1, [528], HQ, HK, D, "f32")
    for h in range(HK):
        H.fill(0, 0, h, d["K0"][0, h], d["V0"][0, h])
    H.set_len(0, 0, 512)
    scale = 1 / math.sqrt(D)
    for t in range(16):
        out, ref = H.decode(0, d["q"][t], d["k_new"][t], d["v_new"][t], 0.99, scale)
        close(out, ref, "out step %d" % t)
        if t % 4 == 3 and t < 15:  # other steps fold into the next call's pass
            H.check_scores(0)
    assert int(H.c.dev_status[0]) == 0

    note("tiny case: prune round")
    # The last step's score update is still pending: layer_sparsity applies it.
    c = H.c
    gb = torch.tensor([256], dtype=torch.int64, device=DEV)
    S = torch.empty((1, 1), dtype=torch.float32, device=DEV)
    bud = torch.empty((1, 1), dtype=torch.int32, device=DEV)
    L.layer_sparsity(c, gb, 32, 0, None, S, bud)
    torch.cuda.synchronize()
    S_ref = H.orc.sparsity(0, 0)
    assert abs(float(S[0, 0]) - S_ref) <= 1e-5
    assert int(bud[0, 0]) == 256
    H.check_scores(0)
    # Heavy hitters dominate the accumulated score.
    for h in range(HK):
        s = H.scores(0, 0, h, 528)
        top = set(np.argsort(-s[:512])[:8].tolist())
        assert len(top & set(d["heavy"][h].tolist())) >= 6
    keep = torch.zeros((1, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    # The scores the selection ranks are the device's own (checked against
    # the oracle's above): on them the keep mask is bit-exact.
    s_dev = [H.scores(0, 0, h, 528).astype(np.float32) for h in range(HK)]
    L.rasr_select(c, bud, 32, 0, keep)
    torch.cuda.synchronize()
    for h in range(HK):
        start, _ = c.seg_rows(0, h)
        kg = host(keep[0, start:start + 528]).astype(bool)
        ko = oracle.rasr_select(s_dev[h], 256, 32, 0)
        np.testing.assert_array_equal(kg, ko)
        assert kg.sum() == 256 and kg[-32:].all()
    ws = c.workspace(L.OP_COMPACT)
    k_before, v_before = host(c.k[0]).copy(), host(c.v[0]).copy()
    s_before = host(c.score[0]).copy()
    L.kv_compact(c, keep, ws)
    torch.cuda.synchronize()
    assert int(c.len[0, 0]) == 256
    for h in range(HK):
        start, _ = c.seg_rows(0, h)
        kg = host(keep[0, start:start + 528]).astype(bool)
        seg = slice(start, start + 528)
        np.testing.assert_array_equal(host(c.k[0, start:start + 256]), oracle.compact(k_before[seg], kg))
        np.testing.assert_array_equal(host(c.v[0, start:start + 256]), oracle.compact(v_before[seg], kg))
        np.testing.assert_array_equal(host(c.score[0, start:start + 256]), oracle.compact(s_before[seg], kg))
    assert int(c.dev_status[0]) == 0


SHAPES = [
    # dtype, D, G, HK, lengths, append
    ("bf16", 128, 4, 2, [0, 1, 63, 64, 65, 700], True),
    ("bf16", 128, 7, 2, [5, 129, 2000], True),
    ("bf16", 128, 8, 1, [333, 1], False),
    ("bf16", 64, 2, 3, [1, 17, 1025], True),
    ("bf16", 64, 1, 2, [200, 0], False),
    ("f32", 64, 2, 2, [512, 3], True),
    ("f32", 128, 5, 1, [77, 300], True),
    ("bf16", 128, 3, 4, [4096, 17, 2500, 1], True),
]


@pytest.mark.parametrize("dtype,D,G,HK,lengths,append", SHAPES)
def test_decode_matches_oracle(dtype, D, G, HK, lengths, append):
    note("decode %s D=%d G=%d HK=%d lengths=%s append=%s" % (dtype, D, G, HK, lengths, append))
    rng = np.random.default_rng(len(lengths) * 1000 + D + G)
    B = len(lengths)
    caps = [n + 4 for n in lengths]  # room for the four appended rows
    H = Harness(2, caps, G * HK, HK, D, dtype)
    for l in range(2):
        for b, n in enumerate(lengths):
            for h in range(HK):
                K = (rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)))).astype(np.float32)
                H.fill(l, b, h, K, rng.standard_normal((n, D)).astype(np.float32),
                       synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    # Steps 1 and 2 apply the previous step's score update inside the decode
    # call; the checks after steps 2 and 3 apply it through the flush.
    for step, gamma in enumerate((0.99, 0.5, 1.0, 0.8)):
        for l in range(2):
            q = (2 * rng.standard_normal((B, G * HK, D))).astype(np.float32)
            kn = rng.standard_normal((B, HK, D)).astype(np.float32) if append else None
            vn = rng.standard_normal((B, HK, D)).astype(np.float32) if append else None
            out, ref = H.decode(l, q, kn, vn, gamma, 0.0 if step == 0 else 0.07)
            close(out, ref, "out step %d layer %d" % (step, l))
        if step >= 2:
            for l in range(2):
                H.check_scores(l)
    assert int(H.c.dev_status[0]) == 0


@pytest.mark.parametrize("env", [{"LETHE_DECODE_BLOCKS": "1"}, {"LETHE_DECODE_BLOCKS": "8192"},
                                 {"LETHE_DECODE_DETERMINISTIC": "1"},
                                 {"LETHE_DECODE_BLOCKS": "8192", "LETHE_DECODE_DETERMINISTIC": "1"}])
@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[3], SHAPES[5], SHAPES[7]])
def test_decode_chunking_extremes(env, shape, monkeypatch):
    """One block per segment (the block writes its output itself) and up to 64
    blocks per segment, many of which find no step left."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    test_decode_matches_oracle(*shape)


def test_decode_deterministic_and_empty(monkeypatch):
    """With the fixed step schedule repeated calls are bit-identical."""
    note("decode determinism")
    monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    rng = np.random.default_rng(7)
    lengths = [1000, 0, 3000]
    H = Harness(1, [4000] * 3, 32, 8, 128, "bf16")
    for b, n in enumerate(lengths):
        for h in range(8):
            H.fill(0, b, h, rng.standard_normal((n, 128)).astype(np.float32),
                   rng.standard_normal((n, 128)).astype(np.float32))
        H.set_len(0, b, n)
    q = H.store(rng.standard_normal((3, 32, 128)))
    outs, scores = [], []
    base_score = H.c.score.clone()
    for _ in range(2):
        H.c.score.copy_(base_score)
        H.c.reset_state()
        out = torch.empty((3, 32, 128), dtype=torch.float32, device=DEV)
        L.decode_attn_score(H.c, 0, q, None, None, 0.9, 0.0, out, H.ws)
        torch.cuda.synchronize()
        # The step's score update is pending until a flush.
        np.testing.assert_array_equal(host(H.c.score), host(base_score))
        H.c.flush()
        torch.cuda.synchronize()
        outs.append(host(out))
        scores.append(host(H.c.score))
    np.testing.assert_array_equal(outs[0], outs[1])
    np.testing.assert_array_equal(scores[0], scores[1])
    assert not outs[0][1].any()          # empty sequence: zero output
    assert not np.array_equal(scores[0], host(base_score))


@pytest.mark.parametrize("dtype,D,G,HK", [("bf16", 128, 4, 8), ("bf16", 64, 7, 2), ("f32", 64, 2, 2)])
def test_flush_applies_once(dtype, D, G, HK):
    """A flush applies the pending step of every (layer, sequence) and leaves
    none: a second flush changes nothing, and the next decode step applies
    only its own predecessor."""
    note("flush once %s D=%d G=%d HK=%d" % (dtype, D, G, HK))
    rng = np.random.default_rng(21 + D + G)
    lengths = [300, 0, 1000]
    H = Harness(3, [n + 4 for n in lengths], G * HK, HK, D, dtype)
    for l in range(3):
        for b, n in enumerate(lengths):
            for h in range(HK):
                H.fill(l, b, h, rng.standard_normal((n, D)).astype(np.float32),
                       rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    B = len(lengths)
    for step in range(2):
        for l in (0, 2):  # layer 1 has no pending step
            q = rng.standard_normal((B, G * HK, D)).astype(np.float32)
            kn = rng.standard_normal((B, HK, D)).astype(np.float32)
            out, ref = H.decode(l, q, kn, kn, 0.9, 0.0)
            close(out, ref, "out step %d layer %d" % (step, l))
        H.c.flush()
        torch.cuda.synchronize()
        first = host(H.c.score).copy()
        H.c.flush()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(H.c.score), first)
        for l in range(3):
            H.check_scores(l)
    assert int(H.c.dev_status[0]) == 0


def test_decode_append_overflow_is_flagged_and_skipped():
    note("decode overflow")
    rng = np.random.default_rng(8)
    H = Harness(1, [10, 10], 8, 2, 64, "bf16")
    for b, n in enumerate([10, 4]):
        for h in range(2):
            H.fill(0, b, h, rng.standard_normal((n, 64)).astype(np.float32),
                   rng.standard_normal((n, 64)).astype(np.float32), np.ones(n, np.float32))
        H.set_len(0, b, n)
    k_before = host(H.c.k).copy()
    q = H.store(rng.standard_normal((2, 8, 64)))
    kn = H.store(rng.standard_normal((2, 2, 64)))
    out = torch.empty((2, 8, 64), dtype=torch.float32, device=DEV)
    L.decode_attn_score(H.c, 0, q, kn, kn, 0.5, 0.0, out, H.ws)
    H.c.flush()
    torch.cuda.synchronize()
    assert int(H.c.dev_status[0]) & L.DEV_APPEND_OVERFLOW
    assert np.isnan(host(out)[0]).all() and not np.isnan(host(out)[1]).any()
    assert H.c.len.cpu().tolist() == [[10, 5]]
    s0, _ = H.c.seg_rows(0, 0)
    np.testing.assert_array_equal(host(H.c.k)[0, s0:s0 + 20], k_before[0, s0:s0 + 20])
    assert (host(H.c.score)[0, s0:s0 + 10] == 1.0).all()


# ---------------------------------------------------------------------------
# Prune round pieces, bit-exact on identical score vectors
# ---------------------------------------------------------------------------

def _prune_harness(lengths, L_, HK, seed, kind):
    rng = np.random.default_rng(seed)
    caps = [n + 5 for n in lengths]
    H = Harness(L_, caps, HK * 2, HK, 128, "bf16")
    for l in range(L_):
        for b, n in enumerate(lengths):
            for h in range(HK):
                H.fill(l, b, h, rng.standard_normal((n, 128)).astype(np.float32),
                       rng.standard_normal((n, 128)).astype(np.float32),
                       synth.score_vector(rng, n, kind))
            H.set_len(l, b, n)
    return H, rng


@pytest.mark.parametrize("kind", ["zipf", "ties", "special"])
def test_select_bit_exact(kind):
    note("select %s" % kind)
    # Up to 8192 candidates a segment's keys stay in registers; the longer
    # segments take the path that re-reads them.
    lengths = [0, 1, 2, 64, 65, 300, 1000, 5000, 9000, 20000]
    H, rng = _prune_harness(lengths, 3, 2, 11, kind)
    c = H.c
    B, L_ = len(lengths), 3
    budgets = np.zeros((B, L_), np.int32)
    for b, n in enumerate(lengths):
        for l in range(L_):
            budgets[b, l] = [0, 1, n // 3, n // 2, n - 1, n, n + 7, 40][(b + 3 * l) % 8]
    for recent, sink in ((0, 0), (32, 4), (64, 0), (3000, 2)):
        bud = torch.from_numpy(budgets).to(DEV)
        keep = torch.full((L_, c.rows_per_layer), 7, dtype=torch.uint8, device=DEV)
        L.rasr_select(c, bud, recent, sink, keep)
        torch.cuda.synchronize()
        kh = host(keep)
        for l in range(L_):
            for b, n in enumerate(lengths):
                for h in range(2):
                    start, _ = c.seg_rows(b, h)
                    want = oracle.rasr_select(H.orc.s[l][b][h].astype(np.float32), budgets[b, l], recent, sink)
                    got = kh[l, start:start + n]
                    assert set(np.unique(got).tolist()) <= {0, 1}
                    np.testing.assert_array_equal(got.astype(bool), want, err_msg="l%d b%d h%d" % (l, b, h))


def test_max_batch_decode_and_prune():
    """The largest batch the library takes (1024 sequences): the decode's
    blocks per segment are capped by its workspace, and the prune kernels
    run thousands of segments.  Every sequence is checked."""
    note("max batch")
    rng = np.random.default_rng(31)
    B, HK, G, D = 1024, 2, 4, 64
    lengths = rng.integers(0, 48, B).tolist()
    H = Harness(1, [n + 2 for n in lengths], G * HK, HK, D, "bf16")
    K = rng.standard_normal((sum(lengths) * HK + 1, D)).astype(np.float32)
    V = rng.standard_normal((sum(lengths) * HK + 1, D)).astype(np.float32)
    r = 0
    for b, n in enumerate(lengths):
        for h in range(HK):
            H.fill(0, b, h, K[r:r + n], V[r:r + n], synth.score_vector(rng, n, "zipf"))
            r += n
        H.set_len(0, b, n)
    for step in range(2):
        q = rng.standard_normal((B, G * HK, D)).astype(np.float32)
        kn = rng.standard_normal((B, HK, D)).astype(np.float32)
        out, ref = H.decode(0, q, kn, kn, 0.9, 0.0)
        close(out, ref, "out step %d" % step)
    H.check_scores(0)
    c = H.c
    bud = torch.from_numpy(np.array([[max(0, n + 2 - 5)] for n in lengths], np.int32)).to(DEV)
    keep = torch.zeros((1, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    L.rasr_select(c, bud, 3, 1, keep)
    torch.cuda.synchronize()
    kh = host(keep)
    sc = host(c.score)
    k_before = host(c.k).copy()
    bh = host(bud)
    for b, n in enumerate(lengths):
        for h in range(HK):
            s0, _ = c.seg_rows(b, h)
            want = oracle.rasr_select(sc[0, s0:s0 + n + 2], int(bh[b, 0]), 3, 1)
            np.testing.assert_array_equal(kh[0, s0:s0 + n + 2].astype(bool), want, err_msg="b%d h%d" % (b, h))
    L.kv_compact(c, keep, c.workspace(L.OP_COMPACT))
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0
    lens = host(c.len)
    for b, n in enumerate(lengths):
        for h in range(HK):
            s0, _ = c.seg_rows(b, h)
            km = kh[0, s0:s0 + n + 2].astype(bool)
            m = int(km.sum())
            assert lens[0, b] == m
            np.testing.assert_array_equal(host(c.k)[0, s0:s0 + m], k_before[0, s0:s0 + n + 2][km])


MASKS = ["random", "first_evicted", "alternate", "last_only", "all", "none", "prefix_kept", "newest_evicted",
         "front_evicted"]


@pytest.mark.parametrize("mask", MASKS)
def test_compact_bit_exact(mask):
    note("compact %s" % mask)
    # Rows move in 256-row tiles; a tile's stores wait for the earlier tiles
    # whose rows they overwrite (up to 35 of them in the 9001-row segment).
    lengths = [1, 2, 63, 64, 65, 700, 3000, 9001]
    H, rng = _prune_harness(lengths, 2, 2, 12, "zipf")
    c = H.c
    keep = np.zeros((2, c.rows_per_layer), np.uint8)
    for l in range(2):
        for b, n in enumerate(lengths):
            start, _ = c.seg_rows(b, 0)
            j = np.arange(n)
            if mask == "random":
                m = rng.random(n) < 0.35
            elif mask == "first_evicted":
                m = j > 0
            elif mask == "alternate":
                m = j % 2 == 1
            elif mask == "last_only":
                m = j == n - 1
            elif mask == "all":
                m = np.ones(n, bool)
            elif mask == "none":
                m = np.zeros(n, bool)
            elif mask == "newest_evicted":
                # Steady state of the decode loop: a few evictions, all among
                # the newest quarter of the rows.
                m = ~((j >= 3 * n // 4) & (rng.random(n) < 0.04))
            elif mask == "front_evicted":
                m = j >= min(600, n // 2)
            else:
                m = j < (n + 1) // 2
            for h in range(2):
                s, _ = c.seg_rows(b, h)
                keep[l, s:s + n] = m
    kt = torch.from_numpy(keep).to(DEV)
    ws = c.workspace(L.OP_COMPACT)
    L.kv_compact(c, kt, ws)
    torch.cuda.synchronize()
    kk = c.k.view(torch.int16).cpu().numpy()
    vv = c.v.view(torch.int16).cpu().numpy()
    ss = c.score.cpu().numpy()
    for l in range(2):
        for b, n in enumerate(lengths):
            s0, _ = c.seg_rows(b, 0)
            cnt = int(keep[l, s0:s0 + n].sum())
            assert int(c.len[l, b]) == cnt
            for h in range(2):
                s, _ = c.seg_rows(b, h)
                m = keep[l, s:s + n].astype(bool)
                want_k = oracle.compact(torch.from_numpy(H.orc.K[l][b][h]).to(torch.bfloat16).view(torch.int16).numpy(), m)
                want_v = oracle.compact(torch.from_numpy(H.orc.V[l][b][h]).to(torch.bfloat16).view(torch.int16).numpy(), m)
                want_s = oracle.compact(H.orc.s[l][b][h].astype(np.float32), m)
                np.testing.assert_array_equal(kk[l, s:s + cnt], want_k)
                np.testing.assert_array_equal(vv[l, s:s + cnt], want_v)
                np.testing.assert_array_equal(ss[l, s:s + cnt].view(np.uint32), want_s.view(np.uint32))
    assert int(c.dev_status[0]) == 0


@pytest.mark.parametrize("dtype,D", [("bf16", 64), ("f32", 128), ("f32", 64)])
@pytest.mark.parametrize("mask", ["random", "front_evicted", "newest_evicted"])
def test_compact_row_widths(dtype, D, mask):
    """Compaction of 128-, 256- and 512-byte rows (its three move kernels) on
    segments of several tiles, bit-exact against the oracle's gather."""
    note("compact %s D=%d %s" % (dtype, D, mask))
    lengths = [0, 1, 300, 3000, 9001]
    rng = np.random.default_rng(21 + D)
    H = Harness(2, [n + 3 for n in lengths], 2 * 2, 2, D, dtype)
    c = H.c
    for l in range(2):
        for b, n in enumerate(lengths):
            for h in range(2):
                H.fill(l, b, h, rng.standard_normal((n, D)).astype(np.float32),
                       rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    keep = np.zeros((2, c.rows_per_layer), np.uint8)
    for l in range(2):
        for b, n in enumerate(lengths):
            j = np.arange(n)
            if mask == "random":
                m = rng.random(n) < 0.3
            elif mask == "front_evicted":
                m = j >= min(700, n // 2)
            else:
                m = ~((j >= 3 * n // 4) & (rng.random(n) < 0.05))
            for h in range(2):
                s0, _ = c.seg_rows(b, h)
                keep[l, s0:s0 + n] = m
    k_before = c.k.cpu().clone()
    v_before = c.v.cpu().clone()
    s_before = c.score.cpu().numpy().copy()
    L.kv_compact(c, torch.from_numpy(keep).to(DEV), c.workspace(L.OP_COMPACT))
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0
    bits = torch.int16 if dtype == "bf16" else torch.int32
    kk, vv = c.k.cpu().view(bits).numpy(), c.v.cpu().view(bits).numpy()
    kb, vb = k_before.view(bits).numpy(), v_before.view(bits).numpy()
    ss = c.score.cpu().numpy()
    for l in range(2):
        for b, n in enumerate(lengths):
            s0, _ = c.seg_rows(b, 0)
            cnt = int(keep[l, s0:s0 + n].sum())
            assert int(c.len[l, b]) == cnt
            for h in range(2):
                s0, _ = c.seg_rows(b, h)
                m = keep[l, s0:s0 + n].astype(bool)
                np.testing.assert_array_equal(kk[l, s0:s0 + cnt], oracle.compact(kb[l, s0:s0 + n], m))
                np.testing.assert_array_equal(vv[l, s0:s0 + cnt], oracle.compact(vb[l, s0:s0 + n], m))
                np.testing.assert_array_equal(ss[l, s0:s0 + cnt].view(np.uint32),
                                              oracle.compact(s_before[l, s0:s0 + n], m).view(np.uint32))


def test_sparsity_and_budgets():
    note("sparsity + budgets")
    lengths = [0, 1, 5, 300, 2000, 4097]
    L_ = 6
    H, rng = _prune_harness(lengths, L_, 4, 13, "zipf")
    c = H.c
    B = len(lengths)
    gb_host = np.array([int(0.3 * n * L_) for n in lengths], np.int64)
    gb = torch.from_numpy(gb_host).to(DEV)
    S = torch.empty((B, L_), dtype=torch.float32, device=DEV)
    bud = torch.empty((B, L_), dtype=torch.int32, device=DEV)
    for recent, sink in ((16, 0), (64, 4)):
        L.layer_sparsity(c, gb, recent, sink, None, S, bud)
        torch.cuda.synchronize()
        Sh, bh = host(S), host(bud)
        for b in range(B):
            Sref = np.array([H.orc.sparsity(l, b) for l in range(L_)])
            assert np.all(np.abs(Sh[b] - Sref) <= 1e-6), (b, Sh[b], Sref)
            n = np.array([lengths[b]] * L_, np.int32)
            want, inf = oracle.budget_split(n, Sref.astype(np.float32), recent, sink, gb_host[b])
            if np.array_equal(Sref.astype(np.float32), Sh[b]):
                np.testing.assert_array_equal(bh[b], want)
            else:   # an fp32 rounding flip of S may move a token between layers
                assert bh[b].sum() == want.sum() and np.abs(bh[b] - want).max() <= 2
    # Given identical layer sparsities (sparsity_in), budgets are bit-exact.
    S_in = rng.random((B, L_)).astype(np.float32)
    S_in[0, 0] = np.nan
    S_in[1, :] = 0.5
    L.layer_sparsity(c, gb, 8, 2, torch.from_numpy(S_in).to(DEV), S, bud)
    torch.cuda.synchronize()
    for b in range(B):
        want, _ = oracle.budget_split(np.array([lengths[b]] * L_, np.int32), S_in[b], 8, 2, gb_host[b])
        np.testing.assert_array_equal(host(bud)[b], want)
    np.testing.assert_array_equal(host(S).view(np.uint32), S_in.view(np.uint32))


def test_infeasible_budget_flag():
    note("infeasible budget")
    H, _ = _prune_harness([500, 500], 2, 2, 14, "zipf")
    c = H.c
    gb = torch.tensor([100, 800], dtype=torch.int64, device=DEV)
    S = torch.empty((2, 2), dtype=torch.float32, device=DEV)
    bud = torch.empty((2, 2), dtype=torch.int32, device=DEV)
    L.layer_sparsity(c, gb, 64, 0, None, S, bud)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) & L.DEV_INFEASIBLE
    assert host(bud)[0].tolist() == [500, 500]
    assert int(host(bud)[1].sum()) == 800
