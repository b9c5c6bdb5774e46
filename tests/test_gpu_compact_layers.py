"""Compaction over a range of layers (lethe_kv_compact_layers) on an MI355X.

Compacting layer by layer must leave what one lethe_kv_compact call leaves:
the same len, the kept K and V rows and their scores bit for bit.  It must
also allow the next decode step to run on another stream, each layer's
decode call waiting only for that layer's compaction: under the fixed step
schedule (LETHE_DECODE_DETERMINISTIC=1) the outputs, rows and pending state
then match the serial order bit for bit, and the outputs match the oracle
(compaction of its own rows, then its decode step).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L

from test_gpu_final_decode import twin
from test_gpu_fused_compact import keep_tensor, make, mask_of, raw_rows
from test_gpu_parity import DEV, close, host

pytestmark = pytest.mark.gpu


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def pending_step(H, rng, scale):
    """One deferred decode step on every layer, so a score update is pending."""
    c = H.c
    for l in range(c.L):
        q = (2 * rng.standard_normal((c.B, c.HQ, c.D))).astype(np.float32)
        kn = rng.standard_normal((c.B, c.HK, c.D)).astype(np.float32)
        vn = rng.standard_normal((c.B, c.HK, c.D)).astype(np.float32)
        out, ref = H.decode(l, q, kn, vn, 0.9, scale)
        close(out, ref, "first step layer %d" % l)


def compact_oracle(H, masks):
    c = H.c
    for l in range(c.L):
        for b in range(c.B):
            for h in range(c.HK):
                m = masks[l][b]
                H.orc.K[l][b][h] = oracle.compact(H.orc.K[l][b][h], m)
                H.orc.V[l][b][h] = oracle.compact(H.orc.V[l][b][h], m)
                H.orc.s[l][b][h] = oracle.compact(H.orc.s[l][b][h], m)


def same_rows(c, T):
    la, lb = host(c.len), host(T.len)
    np.testing.assert_array_equal(la, lb)
    for i, (x, y) in enumerate(zip(raw_rows(c, la), raw_rows(T, lb))):
        np.testing.assert_array_equal(y[0], x[0], err_msg="K rows, segment %d" % i)
        np.testing.assert_array_equal(y[1], x[1], err_msg="V rows, segment %d" % i)
        np.testing.assert_array_equal(y[2], x[2], err_msg="scores, segment %d" % i)


@pytest.mark.parametrize("ranges", [[(0, 1), (1, 1), (2, 1), (3, 1)], [(0, 3), (3, 1)], [(2, 2), (0, 2)]])
def test_compact_layers_matches_whole(ranges):
    note("layer-range compaction %s" % ranges)
    rng = np.random.default_rng(11 + len(ranges))
    H = make(rng, [0, 1, 33, 700, 3000, 9001], 128, 4, 2, layers=4)
    c = H.c
    pending_step(H, rng, 1 / math.sqrt(128))
    lens = [[int(c.len[l, b]) for b in range(c.B)] for l in range(c.L)]
    kinds = ["random", "newest_evicted", "front_evicted", "alternate", "none", "all", "first_evicted"]
    masks = [[mask_of(kinds[(l + 2 * b) % len(kinds)], lens[l][b], rng) for b in range(c.B)] for l in range(c.L)]
    kt = keep_tensor(c, masks)
    T = twin(c)
    L.kv_compact(c, kt, c.workspace(L.OP_COMPACT))
    ws = T.workspace(L.OP_COMPACT)
    for l0, n in ranges:
        L.kv_compact_layers(T, l0, n, kt, ws)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0 and int(T.dev_status[0]) == 0
    same_rows(c, T)
    for l in range(c.L):
        for b in range(c.B):
            assert int(T.len[l, b]) == int(masks[l][b].sum())
    # Both sides had the pending step applied to the rows they kept.
    np.testing.assert_array_equal(host(T.state), host(c.state))


def test_compact_layers_overlapping_next_step(monkeypatch):
    """Layer l compacted on a side stream while the main stream runs the
    decode calls of the layers before it."""
    monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    note("layer-range compaction overlapping the next decode step")
    rng = np.random.default_rng(5)
    H = make(rng, [2, 64, 1500, 5000, 9001, 130], 128, 7, 4, layers=6)
    c = H.c
    B, HQ, HK, D = c.B, c.HQ, c.HK, c.D
    scale = 1 / math.sqrt(D)
    pending_step(H, rng, scale)
    lens = [[int(c.len[l, b]) for b in range(B)] for l in range(c.L)]
    kinds = ["random", "newest_evicted", "front_evicted", "alternate", "prefix_kept"]
    masks = [[mask_of(kinds[(3 * l + b) % len(kinds)], lens[l][b], rng) for b in range(B)] for l in range(c.L)]
    kt = keep_tensor(c, masks)
    T = twin(c)
    compact_oracle(H, masks)
    qs = [H.store(2 * rng.standard_normal((B, HQ, D))) for _ in range(c.L)]
    kns = [H.store(rng.standard_normal((B, HK, D))) for _ in range(c.L)]
    vns = [H.store(rng.standard_normal((B, HK, D))) for _ in range(c.L)]
    # Serial: whole compaction, then the decode step.
    L.kv_compact(c, kt, c.workspace(L.OP_COMPACT))
    outs_a = []
    for l in range(c.L):
        o = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
        L.decode_attn_score(c, l, qs[l], kns[l], vns[l], 0.95, scale, o, H.ws)
        outs_a.append(o)
    # Overlapped: compactions on a side stream, each decode call waiting for
    # its layer's compaction only.
    ws_c = T.workspace(L.OP_COMPACT)
    ws_d = T.workspace(L.OP_DECODE)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream(device=DEV)
    ready = torch.cuda.Event()
    ready.record(main)
    side.wait_event(ready)
    done = []
    for l in range(c.L):
        L.kv_compact_layers(T, l, 1, kt, ws_c, stream=side)
        e = torch.cuda.Event()
        e.record(side)
        done.append(e)
    outs_b = []
    for l in range(c.L):
        main.wait_event(done[l])
        o = torch.full((B, HQ, D), float("nan"), dtype=torch.float32, device=DEV)
        L.decode_attn_score(T, l, qs[l], kns[l], vns[l], 0.95, scale, o, ws_d)
        outs_b.append(o)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0 and int(T.dev_status[0]) == 0
    for l in range(c.L):
        np.testing.assert_array_equal(host(outs_b[l]).view(np.uint32), host(outs_a[l]).view(np.uint32),
                                      err_msg="out layer %d" % l)
        ref = H.orc.decode_step(l, host(qs[l]), host(kns[l]), host(vns[l]), 0.95, scale)
        close(host(outs_b[l]), ref, "overlapped out layer %d" % l)
    same_rows(c, T)
    np.testing.assert_array_equal(host(T.state), host(c.state))
    for l in range(c.L):
        H.check_scores(l)


def test_compact_layers_range_errors():
    note("layer-range compaction, argument errors")
    rng = np.random.default_rng(9)
    H = make(rng, [10, 20], 128, 4, 2, layers=3)
    c = H.c
    kt = keep_tensor(c, [[np.ones(10, bool), np.ones(20, bool)] for _ in range(3)])
    ws = c.workspace(L.OP_COMPACT)
    before = host(c.len).copy()
    for l0, n in [(-1, 1), (0, 4), (3, 1), (2, 2), (0, -1)]:
        with pytest.raises(L.LetheError):
            L.kv_compact_layers(c, l0, n, kt, ws)
    L.kv_compact_layers(c, 1, 0, kt, ws)  # nothing to do
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(c.len), before)
    assert int(c.dev_status[0]) == 0
