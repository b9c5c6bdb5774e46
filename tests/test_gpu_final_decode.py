"""The settling decode call (lethe_decode_attn_score_final) on an MI355X.

It must give the same out and len as lethe_decode_attn_score, and scores
bit-identical to that call followed by lethe_score_flush (same fixed split of
the rows), leave nothing pending, and keep the oracle's tolerance
(|gpu - ref| <= 1e-3 + 2e-3 |ref|).  A sequence skipped for append overflow
keeps its earlier pending step, as in the deferred call.
"""
import math
import sys

import numpy as np
import pytest
import torch

from paper_2511_06029_amd import lethe as L
from workloads import synth

from test_gpu_parity import DEV, Harness, close, host

pytestmark = pytest.mark.gpu


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def twin(c):
    """A second device cache with the same geometry, contents and state."""
    t = L.LetheCache(c.L, c.caps, c.HQ, c.HK, c.D, dtype="bf16" if c.dtype_code == L.BF16 else "f32", device=DEV)
    for name in ("k", "v", "score", "len", "state", "dev_status"):
        getattr(t, name).copy_(getattr(c, name))
    return t


def live_scores(c):
    """Scores of every live row, segment by segment (host arrays)."""
    lens = c.len.cpu().numpy()
    sc = host(c.score)
    out = []
    for l in range(c.L):
        for b in range(c.B):
            for h in range(c.HK):
                s0, _ = c.seg_rows(b, h)
                out.append(sc[l, s0:s0 + int(lens[l, b])])
    return out


def assert_same(a, b, what):
    assert len(a) == len(b)
    for i, (x, y) in enumerate(zip(a, b)):
        np.testing.assert_array_equal(x, y, err_msg="%s, segment %d" % (what, i))


CASES = [
    # dtype, D, G, HK, lengths, spare rows per sequence, append
    ("bf16", 128, 4, 2, [0, 1, 63, 64, 700], [4] * 5, True),
    ("bf16", 128, 7, 4, [5, 2000, 129], [4] * 3, True),
    ("bf16", 128, 8, 1, [333, 1], [4] * 2, False),
    ("bf16", 64, 2, 3, [1, 17, 1025], [4] * 3, True),
    ("bf16", 128, 4, 2, [300, 40], [4, 2], True),   # sequence 1 is full at the settling step
    ("f32", 64, 2, 2, [512, 3], [4] * 2, True),
    ("f32", 128, 5, 1, [77, 300], [4] * 2, True),
]


@pytest.mark.parametrize("dtype,D,G,HK,lengths,spare,append", CASES)
def test_final_equals_deferred_plus_flush(dtype, D, G, HK, lengths, spare, append, monkeypatch):
    note("settling decode %s D=%d G=%d HK=%d lengths=%s spare=%s append=%s" % (dtype, D, G, HK, lengths, spare, append))
    monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    rng = np.random.default_rng(sum(lengths) + 13 * D + G)
    B = len(lengths)
    # Two appends fill a sequence with two spare rows; the oracle has no
    # capacity, so such a case is checked against the deferred call only.
    overflow = append and min(spare) < 3
    H = Harness(2, [n + e for n, e in zip(lengths, spare)], G * HK, HK, D, dtype)
    for l in range(2):
        for b, n in enumerate(lengths):
            for h in range(HK):
                K = (rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)))).astype(np.float32)
                H.fill(l, b, h, K, rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    A = H.c
    Bc = twin(A)
    ws_a = A.workspace(L.OP_DECODE_FINAL)
    ws_b = Bc.workspace(L.OP_DECODE)
    scale = 1 / math.sqrt(D)

    # Two deferred steps on both copies (the oracle follows A), then the
    # settling step on A against deferred + flush on B, then one more deferred
    # step on both: nothing of the settling step may be applied twice.
    for step, (gamma, mode) in enumerate([(0.9, "deferred"), (0.5, "deferred"), (0.99, "final"), (0.8, "deferred")]):
        for l in range(2):
            q = H.store(2 * rng.standard_normal((B, G * HK, D)))
            kn = H.store(rng.standard_normal((B, HK, D))) if append else None
            vn = H.store(rng.standard_normal((B, HK, D))) if append else None
            out_a = torch.empty((B, G * HK, D), dtype=torch.float32, device=DEV)
            out_b = torch.empty_like(out_a)
            if mode == "final":
                L.decode_attn_score_final(A, l, q, kn, vn, gamma, scale, out_a, ws_a)
            else:
                L.decode_attn_score(A, l, q, kn, vn, gamma, scale, out_a, H.ws)
            L.decode_attn_score(Bc, l, q, kn, vn, gamma, scale, out_b, ws_b)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(host(out_a), host(out_b), err_msg="out step %d layer %d" % (step, l))
            if not overflow:
                ref = H.orc.decode_step(l, host(q), None if kn is None else host(kn),
                                        None if vn is None else host(vn), gamma, scale)
                close(host(out_a), ref, "out step %d layer %d" % (step, l))
        if mode == "final":
            Bc.flush()
            torch.cuda.synchronize()
            assert A.len.cpu().tolist() == Bc.len.cpu().tolist()
            if not overflow:
                # Settled without a flush, and a flush then changes nothing.
                assert_same(live_scores(A), live_scores(Bc), "scores after the settling step")
            # A skipped sequence kept its earlier pending step on both copies.
            A.flush()
            torch.cuda.synchronize()
            assert_same(live_scores(A), live_scores(Bc), "scores after flushing both")
    A.flush()
    Bc.flush()
    torch.cuda.synchronize()
    assert_same(live_scores(A), live_scores(Bc), "scores at the end")
    assert int(A.dev_status[0]) == int(Bc.dev_status[0])
    assert bool(int(A.dev_status[0]) & L.DEV_APPEND_OVERFLOW) == overflow
    if not overflow:
        for l in range(2):
            H.check_scores(l)


def test_final_default_split_against_oracle():
    """Dynamic row split (the default launch) on a larger group: tolerance only."""
    note("settling decode, default split")
    rng = np.random.default_rng(5)
    lengths = [4096, 17, 2500, 1]
    HK, G, D = 4, 7, 128
    H = Harness(1, [n + 2 for n in lengths], G * HK, HK, D, "bf16")
    for b, n in enumerate(lengths):
        for h in range(HK):
            H.fill(0, b, h, rng.standard_normal((n, D)).astype(np.float32),
                   rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
        H.set_len(0, b, n)
    ws = H.c.workspace(L.OP_DECODE_FINAL)
    B = len(lengths)
    for step, final in enumerate((False, True)):
        q = H.store(2 * rng.standard_normal((B, G * HK, D)))
        kn = H.store(rng.standard_normal((B, HK, D)))
        vn = H.store(rng.standard_normal((B, HK, D)))
        out = torch.empty((B, G * HK, D), dtype=torch.float32, device=DEV)
        fn = L.decode_attn_score_final if final else L.decode_attn_score
        fn(H.c, 0, q, kn, vn, 0.95, 0.0, out, ws)
        ref = H.orc.decode_step(0, host(q), host(kn), host(vn), 0.95, 1 / math.sqrt(D))
        torch.cuda.synchronize()
        close(host(out), ref, "out step %d" % step)
    # Settled: the scores are current without a flush.
    for b in range(B):
        n = int(H.c.len[0, b])
        for h in range(HK):
            s0, _ = H.c.seg_rows(b, h)
            close(host(H.c.score[0, s0:s0 + n]), H.orc.s[0][b][h], "scores b%d h%d" % (b, h))
    assert int(H.c.dev_status[0]) == 0


def test_final_workspace_is_checked():
    H = Harness(1, [100], 8, 2, 128, "bf16")
    small = H.c.workspace(L.OP_DECODE)
    assert L.workspace_bytes(H.c, L.OP_DECODE_FINAL) >= small.numel() + 100 * 2 * 8 * 4
    q = torch.zeros((1, 8, 128), dtype=torch.bfloat16, device=DEV)
    out = torch.empty((1, 8, 128), dtype=torch.float32, device=DEV)
    with pytest.raises(L.LetheError):
        L.decode_attn_score_final(H.c, 0, q, None, None, 0.9, 0.0, out, small)
