"""Checkpoint -> restore -> continue on an MI355X.

Under the fixed step schedule (LETHE_DECODE_DETERMINISTIC=1) a trajectory of
decode steps, a Lethe prune round and more decode steps is run three ways:
uninterrupted twice, and interrupted by checkpoints (the cache's K, V, scores,
lengths and decode state written to a safetensors file on the host, then
loaded into a freshly allocated cache) once in the middle of a decode run
(a score update pending) and once right after the prune round.  All three
must give the same outputs, rows, scores and decode state bit for bit.  What
has to survive a restart is the accumulated score vector (Eq. 5) and the
pending step the decode state holds; the state stores values only, no
addresses, so it moves with the rest of the cache.
"""
import math
import sys

import numpy as np
import pytest
import torch
from safetensors.torch import load_file, save_file

from paper_2511_06029_amd import lethe as L
from paper_2511_06029_amd import policies
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"
LAYERS, HQ, HK, D = 3, 16, 4, 128
LENGTHS = [300, 1500, 4000, 77]
STEPS = 40
PRUNE_AT = 20  # the round runs after step PRUNE_AT - 1
CHECKPOINTS = (10, PRUNE_AT)  # restart before these steps (the second right after the round)
FIELDS = ("k", "v", "score", "len", "state", "dev_status")


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def inputs():
    rng = np.random.default_rng(2024)
    B = len(LENGTHS)
    q = [[torch.from_numpy((2 * rng.standard_normal((B, HQ, D))).astype(np.float32)).to(DEV, torch.bfloat16)
          for _ in range(LAYERS)] for _ in range(STEPS)]
    kn = [[torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV, torch.bfloat16)
           for _ in range(LAYERS)] for _ in range(STEPS)]
    vn = [[torch.from_numpy(rng.standard_normal((B, HK, D)).astype(np.float32)).to(DEV, torch.bfloat16)
           for _ in range(LAYERS)] for _ in range(STEPS)]
    return q, kn, vn


def new_cache():
    return L.LetheCache(LAYERS, [n + STEPS + 8 for n in LENGTHS], HQ, HK, D, dtype="bf16", device=DEV)


def filled_cache():
    rng = np.random.default_rng(7)
    c = new_cache()
    k = np.zeros((LAYERS, c.rows_per_layer, D), np.float32)
    v = np.zeros_like(k)
    s = np.zeros((LAYERS, c.rows_per_layer), np.float32)
    for l in range(LAYERS):
        for b, n in enumerate(LENGTHS):
            for h in range(HK):
                r0, _ = c.seg_rows(b, h)
                k[l, r0:r0 + n] = rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)))
                v[l, r0:r0 + n] = rng.standard_normal((n, D))
                s[l, r0:r0 + n] = synth.score_vector(rng, n, "zipf")
    c.k.copy_(torch.from_numpy(k))
    c.v.copy_(torch.from_numpy(v))
    c.score.copy_(torch.from_numpy(s))
    c.len.copy_(torch.tensor([LENGTHS] * LAYERS, dtype=torch.int32))
    return c


def run(c, t0, t1, data, outs):
    """Decode steps t0 .. t1 - 1; the prune round follows step PRUNE_AT - 1."""
    q, kn, vn = data
    ws = c.workspace(L.OP_DECODE)
    prune = policies.PruneRound(c, policies.get("lethe", gamma=0.99))
    scale = 1 / math.sqrt(D)
    for t in range(t0, t1):
        for l in range(LAYERS):
            o = torch.empty((c.B, HQ, D), dtype=torch.float32, device=DEV)
            L.decode_attn_score(c, l, q[t][l], kn[t][l], vn[t][l], 0.99, scale, o, ws)
            outs.append(o)
        if t == PRUNE_AT - 1:
            lens = c.len.cpu().numpy()
            per_seq = [policies.per_layer_budget(0.4, int(lens[0, b])) for b in range(c.B)]
            prune(per_seq, 16)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0


def checkpoint(c, path):
    torch.cuda.synchronize()
    save_file({f: getattr(c, f).detach().cpu().contiguous() for f in FIELDS}, str(path))


def restore(path):
    c = new_cache()
    saved = load_file(str(path))
    for f in FIELDS:
        getattr(c, f).copy_(saved[f])
    torch.cuda.synchronize()
    return c


def bits(t):
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.numpy()


def assert_same_run(a_outs, a_cache, b_outs, b_cache, what):
    assert len(a_outs) == len(b_outs)
    for i, (x, y) in enumerate(zip(a_outs, b_outs)):
        np.testing.assert_array_equal(bits(y), bits(x), err_msg="%s: output %d" % (what, i))
    for f in FIELDS:
        np.testing.assert_array_equal(bits(getattr(b_cache, f)), bits(getattr(a_cache, f)),
                                      err_msg="%s: %s" % (what, f))


def test_checkpoint_restore_continue(monkeypatch, tmp_path):
    monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    data = inputs()
    note("resume: uninterrupted runs")
    ref_c, ref_outs = filled_cache(), []
    run(ref_c, 0, STEPS, data, ref_outs)
    again_c, again_outs = filled_cache(), []
    run(again_c, 0, STEPS, data, again_outs)
    assert_same_run(ref_outs, ref_c, again_outs, again_c, "repeat")
    assert int(ref_c.len[0, 0]) < LENGTHS[0] + STEPS  # the round evicted rows

    note("resume: interrupted by checkpoints before steps %s" % (CHECKPOINTS,))
    c, outs, t = filled_cache(), [], 0
    for i, stop in enumerate(CHECKPOINTS):
        run(c, t, stop, data, outs)
        path = tmp_path / ("lethe_%d.safetensors" % i)
        checkpoint(c, path)
        del c
        c = restore(path)
        t = stop
    run(c, t, STEPS, data, outs)
    assert_same_run(ref_outs, ref_c, outs, c, "resumed")
