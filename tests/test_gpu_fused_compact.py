"""Compaction carried out by the next decode step (lethe_kv_compact_plan +
lethe_decode_attn_score_compact) on an MI355X.

On twin caches it must leave what lethe_kv_compact followed by
lethe_decode_attn_score leaves: the same len, the kept K and V rows and
their scores bit for bit (a pending score update applied to the kept rows on
both sides), and outputs within the decode tolerance of each other and of the
oracle (compaction of its own rows, then its decode step).  Masks cover the
adversarial shapes of the compaction tests; edge cases: nothing kept, nothing
evicted, a plan made before the lengths changed, heads keeping different
counts, fp32 caches.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L
from workloads import synth

from test_gpu_final_decode import twin
from test_gpu_parity import DEV, Harness, close, host

pytestmark = pytest.mark.gpu


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def make(rng, lengths, D, G, HK, layers=2, spare=4):
    H = Harness(layers, [n + spare for n in lengths], G * HK, HK, D, "bf16")
    for l in range(layers):
        for b, n in enumerate(lengths):
            for h in range(HK):
                K = (rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)))).astype(np.float32)
                H.fill(l, b, h, K, rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    return H


def mask_of(kind, n, rng):
    j = np.arange(n)
    if kind == "random":
        return rng.random(n) < 0.35
    if kind == "first_evicted":
        return j > 0
    if kind == "alternate":
        return j % 2 == 1
    if kind == "last_only":
        return j == n - 1
    if kind == "all":
        return np.ones(n, bool)
    if kind == "none":
        return np.zeros(n, bool)
    if kind == "newest_evicted":
        return ~((j >= 3 * n // 4) & (rng.random(n) < 0.04))
    if kind == "front_evicted":
        return j >= min(600, n // 2)
    return j < (n + 1) // 2  # prefix_kept


def keep_tensor(c, masks):
    """masks[l][b]: bool (n,), the same for every KV head."""
    keep = np.zeros((c.L, c.rows_per_layer), np.uint8)
    for l in range(c.L):
        for b in range(c.B):
            for h in range(c.HK):
                s, _ = c.seg_rows(b, h)
                keep[l, s:s + len(masks[l][b])] = masks[l][b]
    return torch.from_numpy(keep).to(DEV)


def raw_rows(c, lengths_after):
    """K and V as int16 patterns and scores as uint32, rows [0, len) of every segment."""
    kk = c.k.view(torch.int16).cpu().numpy()
    vv = c.v.view(torch.int16).cpu().numpy()
    ss = c.score.cpu().numpy().view(np.uint32)
    out = []
    for l in range(c.L):
        for b in range(c.B):
            n = int(lengths_after[l][b])
            for h in range(c.HK):
                s, _ = c.seg_rows(b, h)
                out.append((kk[l, s:s + n].copy(), vv[l, s:s + n].copy(), ss[l, s:s + n].copy()))
    return out


def run_case(rng, lengths, D, G, HK, kinds, append=True):
    """A deferred decode step on the harness (so a score update is pending),
    then eager compaction + decode on the harness cache and plan + compacting
    decode on its twin; the oracle follows the harness."""
    H = make(rng, lengths, D, G, HK)
    c = H.c
    B, HQ = c.B, c.HQ
    scale = 1 / math.sqrt(D)
    for l in range(c.L):
        q = (2 * rng.standard_normal((B, HQ, D))).astype(np.float32)
        kn = rng.standard_normal((B, HK, D)).astype(np.float32)
        vn = rng.standard_normal((B, HK, D)).astype(np.float32)
        out, ref = H.decode(l, q, kn, vn, 0.9, scale)
        close(out, ref, "first step layer %d" % l)
    lens = [[int(c.len[l, b]) for b in range(B)] for l in range(c.L)]
    masks = [[mask_of(kinds[(l + b) % len(kinds)], lens[l][b], rng) for b in range(B)] for l in range(c.L)]
    kt = keep_tensor(c, masks)
    T = twin(c)
    plan = T.workspace(L.OP_COMPACT_PLAN)
    ws_t = T.workspace(L.OP_DECODE)
    L.kv_compact(c, kt, c.workspace(L.OP_COMPACT))
    L.kv_compact_plan(T, kt, plan)
    # The oracle: its pending-free scores compact with the rows.
    for l in range(c.L):
        for b in range(B):
            for h in range(HK):
                m = masks[l][b]
                H.orc.K[l][b][h] = oracle.compact(H.orc.K[l][b][h], m)
                H.orc.V[l][b][h] = oracle.compact(H.orc.V[l][b][h], m)
                H.orc.s[l][b][h] = oracle.compact(H.orc.s[l][b][h], m)
    for l in range(c.L):
        q = H.store(2 * rng.standard_normal((B, HQ, D)))
        kn = H.store(rng.standard_normal((B, HK, D))) if append else None
        vn = H.store(rng.standard_normal((B, HK, D))) if append else None
        oa = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
        ob = torch.full_like(oa, float("nan"))
        L.decode_attn_score(c, l, q, kn, vn, 0.95, scale, oa, H.ws)
        L.decode_attn_score_compact(T, l, q, kn, vn, 0.95, scale, ob, plan, ws_t)
        ref = H.orc.decode_step(l, host(q), None if kn is None else host(kn), None if vn is None else host(vn),
                                0.95, scale)
        torch.cuda.synchronize()
        close(host(oa), ref, "eager out layer %d" % l)
        close(host(ob), ref, "fused out layer %d" % l)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0 and int(T.dev_status[0]) == 0, (int(c.dev_status[0]), int(T.dev_status[0]))
    la, lb = host(c.len), host(T.len)
    np.testing.assert_array_equal(la, lb)
    for l in range(c.L):
        for b in range(B):
            assert la[l, b] == int(masks[l][b].sum()) + (1 if append else 0)
    # Rows and scores (this step's update still pending on both) bit for bit.
    for i, (x, y) in enumerate(zip(raw_rows(c, la), raw_rows(T, lb))):
        np.testing.assert_array_equal(y[0], x[0], err_msg="K rows, segment %d" % i)
        np.testing.assert_array_equal(y[1], x[1], err_msg="V rows, segment %d" % i)
        np.testing.assert_array_equal(y[2], x[2], err_msg="scores, segment %d" % i)
    # Scores with this step applied: each side against the oracle.
    T.flush()
    torch.cuda.synchronize()
    for l in range(c.L):
        for b in range(B):
            n = int(lb[l, b])
            for h in range(HK):
                s0, _ = T.seg_rows(b, h)
                close(host(T.score[l, s0:s0 + n]), H.orc.s[l][b][h], "fused scores l%d b%d h%d" % (l, b, h))
    H.check_scores(0)
    H.check_scores(1)


MASKS = ["random", "first_evicted", "alternate", "last_only", "all", "none", "prefix_kept", "newest_evicted",
         "front_evicted"]


@pytest.mark.parametrize("mask", MASKS)
def test_fused_compaction_masks(mask):
    note("fused compaction, mask %s" % mask)
    rng = np.random.default_rng(100 + MASKS.index(mask))
    run_case(rng, [1, 2, 31, 32, 33, 700, 3000, 9001], 128, 4, 2, [mask])


@pytest.mark.parametrize("D,G,HK", [(128, 7, 4), (64, 2, 3), (128, 8, 1), (64, 1, 2)])
def test_fused_compaction_shapes(D, G, HK):
    note("fused compaction D=%d G=%d HK=%d" % (D, G, HK))
    rng = np.random.default_rng(7 * D + G + HK)
    run_case(rng, [0, 5, 64, 65, 1500, 4097], D, G, HK, ["random", "newest_evicted", "front_evicted", "alternate"])


@pytest.mark.parametrize("env", [{"LETHE_DECODE_BLOCKS": "1"}, {"LETHE_DECODE_BLOCKS": "8192"}])
def test_fused_compaction_chunking(env, monkeypatch):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    note("fused compaction %s" % env)
    rng = np.random.default_rng(31)
    run_case(rng, [40, 2000, 9001], 128, 4, 2, ["random", "front_evicted", "newest_evicted"])


def test_fused_compaction_no_append_keep_none():
    """No new row and nothing kept: len becomes 0 and out is 0."""
    note("fused compaction, nothing kept, no append")
    rng = np.random.default_rng(41)
    run_case(rng, [300, 33], 128, 4, 2, ["none"], append=False)


def test_fused_compaction_stale_and_mismatched_plans():
    """A plan made before a decode step appended rows, and heads keeping
    different counts: those sequences are skipped and flagged, the rest
    compact."""
    note("fused compaction, stale and invalid plans")
    rng = np.random.default_rng(43)
    lengths = [500, 800, 1200]
    H = make(rng, lengths, 128, 4, 2, layers=1, spare=8)
    c = H.c
    masks = [[mask_of("random", n, rng) for n in lengths]]
    keep = keep_tensor(c, masks)
    # Sequence 2: head 1 keeps one row fewer than head 0.
    s1, _ = c.seg_rows(2, 1)
    row = s1 + int(np.flatnonzero(masks[0][2])[0])
    keep[0, row] = 0
    plan = c.workspace(L.OP_COMPACT_PLAN)
    L.kv_compact_plan(c, keep, plan)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) & L.DEV_HEAD_MISMATCH
    c.dev_status.zero_()
    B, HQ, HK, D = 3, 8, 2, 128
    q = H.store(rng.standard_normal((B, HQ, D)))
    kn = H.store(rng.standard_normal((B, HK, D)))
    vn = H.store(rng.standard_normal((B, HK, D)))
    out = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
    # Sequence 0's length changes after the plan (made stale).
    c.len[0, 0] = lengths[0] - 1
    L.decode_attn_score_compact(c, 0, q, kn, vn, 0.9, 0.0, out, plan, H.ws)
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) & L.DEV_BAD_LAYOUT
    lens = host(c.len)[0].tolist()
    assert lens == [lengths[0] - 1, int(masks[0][1].sum()) + 1, lengths[2]]
    o = host(out)
    assert np.isnan(o[0]).all() and np.isnan(o[2]).all() and np.isfinite(o[1]).all()


def test_fused_compaction_rejects_fp32():
    c = L.LetheCache(1, [64], 4, 2, 64, dtype="f32", device=DEV)
    plan = c.workspace(L.OP_COMPACT_PLAN)
    ws = c.workspace(L.OP_DECODE)
    q = torch.zeros((1, 4, 64), dtype=torch.float32, device=DEV)
    out = torch.empty((1, 4, 64), dtype=torch.float32, device=DEV)
    with pytest.raises(L.LetheError) as e:
        L.decode_attn_score_compact(c, 0, q, None, None, 0.9, 0.0, out, plan, ws)
    assert e.value.status == L.ERR_UNSUPPORTED
