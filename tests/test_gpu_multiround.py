"""Several decode intervals and prune rounds in a row against the oracle (run
on an MI355X).

The serving loop of Section 4: decode steps whose score updates (Eq. 5) stay
pending from one call to the next, the settling call that closes each
interval, then a prune round (Hoyer sparsity and budgets, Eqs. 1-4; RASR
selection, Section 4.2; compaction), and decoding again on the compacted
cache with the tiling hints the compaction rewrote.  Three rounds, each
compaction carried out one of three ways: whole cache in the round, layer by
layer on a second stream with each layer's next decode step waiting for its
own layer, or by the next decode step itself.  The kept sets come from RASR
per KV head, RASR on the head-summed score (one set per layer and sequence),
or Algorithm 1 with its size trigger, whose eviction thresholds carry over
from round to round on the device.

The oracle follows every step; after a round it drops the rows the device's
keep mask drops, from its own K, V and score arrays, so that it goes on
independently of the device's arithmetic.  Checked every step: outputs within
1e-3 + 2e-3 |ref|.  Every interval's end: lengths and K, V rows bit for bit,
scores within the output tolerance.  Every round: sparsities against the
oracle's on the device's scores (1e-6) and on its own (1e-4), budgets, keep
masks, breakpoints and thresholds bit-exact given the device's sparsities and
scores.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L

from test_gpu_parity import DEV, Harness, close, host

pytestmark = pytest.mark.gpu

LAYERS, G, HK, D = 3, 4, 2, 128
LENGTHS = [700, 2500, 0, 33, 1300]
STEPS, ROUNDS = 8, 3          # steps per interval, prune rounds
RECENT, SINK, KEEP_FRAC = 16, 2, 0.6
SEGMENTS, TAU = 8, 3.0        # Algorithm 1's cut points and ratio


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def make(rng):
    caps = [n + STEPS * (ROUNDS + 1) + 3 for n in LENGTHS]
    H = Harness(LAYERS, caps, G * HK, HK, D, "bf16")
    for l in range(LAYERS):
        for b, n in enumerate(LENGTHS):
            for h in range(HK):
                # Keys of mixed norms, so that a few rows draw most attention.
                K = (rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)) ** 4)).astype(np.float32)
                H.fill(l, b, h, K, rng.standard_normal((n, D)).astype(np.float32))
            H.set_len(l, b, n)
    return H


def check_rows(H):
    """Lengths and K, V rows bit for bit (bf16 widened on both sides)."""
    c = H.c
    lens = host(c.len)
    for l in range(c.L):
        for b in range(c.B):
            n = int(lens[l, b])
            assert n == H.orc.length(l, b), (l, b, n, H.orc.length(l, b))
            for h in range(c.HK):
                s, _ = c.seg_rows(b, h)
                np.testing.assert_array_equal(host(c.k[l, s:s + n]), H.orc.K[l][b][h], err_msg="K l%d b%d h%d" % (l, b, h))
                np.testing.assert_array_equal(host(c.v[l, s:s + n]), H.orc.V[l][b][h], err_msg="V l%d b%d h%d" % (l, b, h))


def interval(H, rng, ctx, r):
    """STEPS decode steps per layer; the last one settles its own update."""
    c, B, HQ = H.c, H.c.B, H.c.HQ
    scale = 1 / math.sqrt(D)
    gamma = (0.97, 0.9, 1.0, 0.8)[r % 4]
    for t in range(STEPS):
        for l in range(LAYERS):
            q = H.store(2 * rng.standard_normal((B, HQ, D)))
            kn = H.store(rng.standard_normal((B, HK, D)))
            vn = H.store(rng.standard_normal((B, HK, D)))
            out = torch.full((B, HQ, D), float("nan"), dtype=torch.float32, device=DEV)
            if t == 0 and ctx.get("plan") is not None:
                L.decode_attn_score_compact(c, l, q, kn, vn, gamma, scale, out, ctx["plan"], H.ws)
            else:
                if t == 0 and ctx.get("done") is not None:
                    torch.cuda.current_stream().wait_event(ctx["done"][l])
                if t == STEPS - 1:
                    L.decode_attn_score_final(c, l, q, kn, vn, gamma, scale, out, ctx["ws_final"])
                else:
                    L.decode_attn_score(c, l, q, kn, vn, gamma, scale, out, H.ws)
            ref = H.orc.decode_step(l, host(q), host(kn), host(vn), gamma, scale)
            torch.cuda.synchronize()
            close(host(out), ref, "round %d step %d layer %d" % (r, t, l))
        if t == 0:
            ctx["plan"] = ctx["done"] = None
    check_rows(H)
    # The settling call left nothing pending: the stored scores are current.
    for l in range(LAYERS):
        for b in range(B):
            n = H.orc.length(l, b)
            for h in range(HK):
                s, _ = c.seg_rows(b, h)
                close(host(c.score[l, s:s + n]), H.orc.s[l][b][h], "scores round %d l%d b%d h%d" % (r, l, b, h))


def prune(H, ctx, mode, rule, r):
    c, B = H.c, H.c.B
    lens = host(c.len).astype(np.int64)
    keep = torch.full((LAYERS, c.rows_per_layer), 7, dtype=torch.uint8, device=DEV)
    if rule == "shrink":
        thr = host(ctx["evict"]).copy()
        bp = torch.full((LAYERS, B), 99, dtype=torch.int32, device=DEV)
        L.segmented_shrink(c, SEGMENTS, TAU, RECENT, SINK, ctx["evict"], bp, keep)
    else:
        gb_host = np.zeros(B, np.int64)
        for b in range(B):
            protected = sum(min(int(lens[l, b]), RECENT + SINK) for l in range(LAYERS))
            gb_host[b] = max(int(KEEP_FRAC * lens[:, b].sum()), protected)
        gb = torch.from_numpy(gb_host).to(DEV)
        S = torch.empty((B, LAYERS), dtype=torch.float32, device=DEV)
        bud = torch.empty((B, LAYERS), dtype=torch.int32, device=DEV)
        L.layer_sparsity(c, gb, RECENT, SINK, None, S, bud)
        (L.rasr_select_shared if rule == "shared" else L.rasr_select)(c, bud, RECENT, SINK, keep)
    torch.cuda.synchronize()
    kh = host(keep)
    score = host(c.score)
    masks = {}
    for b in range(B):
        heads = {}
        for l in range(LAYERS):
            n = int(lens[l, b])
            heads[l] = np.stack([score[l, s:s + n] for s, _ in (c.seg_rows(b, h) for h in range(HK))])
        if rule == "shrink":
            evh, bph = host(ctx["evict"]), host(bp)
            for l in range(LAYERS):
                want, wbp, wlev = oracle.segmented_shrink(oracle.head_sum_f32(heads[l]), SEGMENTS, TAU, RECENT, SINK,
                                                          thr[l, b])
                assert (int(bph[l, b]), int(evh[l, b])) == (wbp, wlev), (r, l, b, thr[l, b])
                ctx["cuts"] += wbp >= 0
                for h in range(HK):
                    masks[l, b, h] = want
        else:
            Sh, bh = host(S), host(bud)
            for l in range(LAYERS):
                S_dev_scores = oracle.layer_sparsity(heads[l])
                assert abs(Sh[b, l] - S_dev_scores) <= 1e-6, (r, b, l, Sh[b, l], S_dev_scores)
                assert abs(Sh[b, l] - H.orc.sparsity(l, b)) <= 1e-4, (r, b, l, Sh[b, l], H.orc.sparsity(l, b))
            want, infeasible = oracle.budget_split(lens[:, b].astype(np.int32), Sh[b], RECENT, SINK, gb_host[b])
            assert not infeasible
            np.testing.assert_array_equal(bh[b], want, err_msg="budgets round %d b%d" % (r, b))
            for l in range(LAYERS):
                for h in range(HK):
                    if rule == "shared":
                        masks[l, b, h] = oracle.rasr_select_shared(heads[l], int(bh[b, l]), RECENT, SINK)
                    else:
                        masks[l, b, h] = oracle.rasr_select(heads[l][h], int(bh[b, l]), RECENT, SINK)
        for l in range(LAYERS):
            n = int(lens[l, b])
            for h in range(HK):
                s, _ = c.seg_rows(b, h)
                np.testing.assert_array_equal(kh[l, s:s + n], masks[l, b, h].astype(np.uint8),
                                              err_msg="keep round %d l%d b%d h%d" % (r, l, b, h))
    note("round %d: %d of %d rows kept" % (r, sum(int(m.sum()) for m in masks.values()), int(lens.sum()) * HK))
    if mode == "eager":
        L.kv_compact(c, keep, ctx["ws_c"])
    elif mode == "layers":
        # Each layer's compaction on a second stream; each layer's next decode
        # step waits for its own layer only.
        main, side = torch.cuda.current_stream(), ctx["side"]
        ready = torch.cuda.Event()
        ready.record(main)
        side.wait_event(ready)
        done = [torch.cuda.Event() for _ in range(LAYERS)]
        for l in range(LAYERS):
            L.kv_compact_layers(c, l, 1, keep, ctx["ws_c"], stream=side)
            done[l].record(side)
        ctx["done"] = done
        ctx["keep_alive"] = keep      # in use on the side stream
    else:
        L.kv_compact_plan(c, keep, ctx["ws_c"])
        ctx["plan"] = ctx["ws_c"]
    for (l, b, h), m in masks.items():
        H.orc.K[l][b][h] = oracle.compact(H.orc.K[l][b][h], m)
        H.orc.V[l][b][h] = oracle.compact(H.orc.V[l][b][h], m)
        H.orc.s[l][b][h] = oracle.compact(H.orc.s[l][b][h], m)


@pytest.mark.parametrize("rule", ["rasr", "shared", "shrink"])
@pytest.mark.parametrize("mode", ["eager", "layers", "fused"])
def test_decode_prune_rounds(mode, rule):
    note("multi-round %s %s" % (mode, rule))
    rng = np.random.default_rng(31 + 3 * ["eager", "layers", "fused"].index(mode) + ["rasr", "shared", "shrink"].index(rule))
    H = make(rng)
    c = H.c
    # Size-trigger thresholds: pruning from the first round on, once past
    # 1000 tokens, and never (above any length here).
    thr = np.tile(np.array([0, 1000, 1 << 20, 0, 1000], np.int32), (LAYERS, 1))
    ctx = {"ws_final": c.workspace(L.OP_DECODE_FINAL), "plan": None, "done": None,
           "ws_c": c.workspace(L.OP_COMPACT_PLAN if mode == "fused" else L.OP_COMPACT),
           "side": torch.cuda.Stream(device=DEV) if mode == "layers" else None,
           "evict": torch.from_numpy(thr).to(DEV), "cuts": 0}
    for r in range(ROUNDS):
        interval(H, rng, ctx, r)
        prune(H, ctx, mode, rule, r)
    interval(H, rng, ctx, ROUNDS)
    assert int(c.dev_status[0]) == 0, L.dev_status_names(int(c.dev_status[0]))
    if rule == "shrink":
        assert ctx["cuts"] > 0          # some rounds found a breakpoint
    else:
        # The long sequences were pruned below what they would hold unpruned.
        lens = host(c.len)
        for b, n in enumerate(LENGTHS):
            if n > 100:
                assert (lens[:, b] < n + STEPS * (ROUNDS + 1)).all(), (b, lens[:, b])
