"""Decode tiling on an MI355X: segments of very different lengths split into
chunks by the layer's tiling hints (lengths the flush and the compaction
record in the decode state).

Checked against the oracle (|gpu - ref| <= 1e-3 + 2e-3 |ref|): the flat
split (no hints yet), the hinted split, hints that no longer match the
lengths (the split then only balances worse), several block targets, the
adaptive chunk count at its extremes (one step a chunk, the fewest chunks,
always the most) and the fixed step schedule.  With the fixed schedule repeated calls on twin caches
are bit-identical.
"""
import math
import sys

import numpy as np
import pytest
import torch

from paper_2511_06029_amd import lethe as L
from workloads import synth

from test_gpu_final_decode import assert_same, live_scores, twin
from test_gpu_parity import DEV, Harness, close, host

pytestmark = pytest.mark.gpu


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


LENGTHS = [1, 7, 20000, 33, 4096, 0, 900, 12000, 64, 65]


def ragged(rng, lengths=LENGTHS, HK=2, G=4, D=128, spare=40, room=None):
    """room[b]: rows sequence b may grow to (default its length)."""
    room = room or {}
    H = Harness(1, [max(n, room.get(b, 0)) + spare for b, n in enumerate(lengths)], G * HK, HK, D, "bf16")
    for b, n in enumerate(lengths):
        for h in range(HK):
            H.fill(0, b, h, rng.standard_normal((n, D)).astype(np.float32),
                   rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
        H.set_len(0, b, n)
    return H


def step(H, rng, gamma=0.95):
    B, HQ, D, HK = H.c.B, H.c.HQ, H.c.D, H.c.HK
    q = 2 * rng.standard_normal((B, HQ, D))
    kn = rng.standard_normal((B, HK, D))
    vn = rng.standard_normal((B, HK, D))
    out, ref = H.decode(0, q.astype(np.float32), kn.astype(np.float32), vn.astype(np.float32), gamma, 0.0)
    return out, ref


@pytest.mark.parametrize("env", [{}, {"LETHE_DECODE_BLOCKS": "1"}, {"LETHE_DECODE_BLOCKS": "3"},
                                 {"LETHE_DECODE_BLOCKS": "8192"}, {"LETHE_DECODE_DETERMINISTIC": "1"},
                                 {"LETHE_DECODE_DETERMINISTIC": "1", "LETHE_DECODE_BLOCKS": "3"},
                                 {"LETHE_DECODE_STEPS_PER_CHUNK": "1"},
                                 {"LETHE_DECODE_STEPS_PER_CHUNK": "100000", "LETHE_DECODE_MIN_CHUNKS": "1"},
                                 {"LETHE_DECODE_MIN_CHUNKS": "100000"}],
                         ids=["default", "blocks1", "blocks3", "blocks8192", "fixed", "fixed-blocks3",
                              "adaptive-1step", "adaptive-fewest", "adaptive-all"])
def test_tiling_flat_hinted_and_stale(env, monkeypatch):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    rng = np.random.default_rng(11)
    note("tiling %s: flat split (hints 0)" % env)
    H = ragged(rng, room={1: 9000})
    out, ref = step(H, rng)
    close(out, ref, "flat split")
    note("tiling %s: hinted split" % env)
    H.c.flush()  # records the lengths as hints
    for t in range(2):
        out, ref = step(H, rng)
        close(out, ref, "hinted split, step %d" % t)
    H.check_scores(0)  # flushes, hints current again
    note("tiling %s: stale hints" % env)
    # Lengths change after the flush (as a caller editing len would): the
    # longest sequence shrinks to 5 rows, a short one grows to 9000.
    for b, n in ((2, 5), (1, 9000)):
        for h in range(H.c.HK):
            H.fill(0, b, h, rng.standard_normal((n, H.c.D)).astype(np.float32),
                   rng.standard_normal((n, H.c.D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
        H.set_len(0, b, n)
    torch.cuda.synchronize()
    for t in range(2):
        out, ref = step(H, rng)
        close(out, ref, "stale hints, step %d" % t)
    H.check_scores(0)
    assert int(H.c.dev_status[0]) == 0


def test_fixed_schedule_is_bit_reproducible(monkeypatch):
    """Twin caches, the same calls, the fixed step schedule: out and scores
    identical bit for bit (the flat split, then the hinted one)."""
    monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    rng = np.random.default_rng(12)
    note("tiling: reproducibility")
    H = ragged(rng, HK=4, G=7)
    A = H.c
    Tw = twin(A)
    ws_t = Tw.workspace(L.OP_DECODE)
    B, HQ, D, HK = A.B, A.HQ, A.D, A.HK
    for t in range(4):
        if t == 2:
            A.flush()
            Tw.flush()
        q = H.store(2 * rng.standard_normal((B, HQ, D)))
        kn = H.store(rng.standard_normal((B, HK, D)))
        vn = H.store(rng.standard_normal((B, HK, D)))
        oa = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
        ob = torch.empty_like(oa)
        L.decode_attn_score(A, 0, q, kn, vn, 0.9, 0.0, oa, H.ws)
        L.decode_attn_score(Tw, 0, q, kn, vn, 0.9, 0.0, ob, ws_t)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(oa), host(ob), err_msg="out step %d" % t)
    A.flush()
    Tw.flush()
    torch.cuda.synchronize()
    assert_same(live_scores(A), live_scores(Tw), "scores")


@pytest.mark.parametrize("nseq", [65, 128, 129, 256, 300])
def test_sequence_counts_plan_paths(nseq):
    """The block plan reads the hints of 64 sequences a round: with the chosen
    sequence's words in the same round up to 256 sequences (two rounds up to
    128, four up to 256), and in 16 rounds and a second load above that.
    Lengths log-uniform 1 .. 3000, one of them empty; the first step splits
    flat, the later ones by the hints the flush records."""
    rng = np.random.default_rng(13 + nseq)
    lengths = [int(x) for x in np.exp(rng.uniform(0, math.log(3000), size=nseq))]
    lengths[5] = 0
    note("tiling: %d sequences" % nseq)
    HK, G, D = 1, 4, 64
    H = Harness(1, [n + 4 for n in lengths], G * HK, HK, D, "bf16")
    for b, n in enumerate(lengths):
        H.fill(0, b, 0, rng.standard_normal((n, D)).astype(np.float32),
               rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
        H.set_len(0, b, n)
    for t in range(3):
        if t == 1:
            H.c.flush()
        q = 2 * rng.standard_normal((len(lengths), G * HK, D))
        kn = rng.standard_normal((len(lengths), HK, D))
        vn = rng.standard_normal((len(lengths), HK, D))
        out, ref = H.decode(0, q.astype(np.float32), kn.astype(np.float32), vn.astype(np.float32), 0.9, 0.0)
        close(out, ref, "%d sequences, step %d" % (nseq, t))
    H.check_scores(0)
    assert int(H.c.dev_status[0]) == 0
