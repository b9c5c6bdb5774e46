"""GPU parity of the head-shared kept sets (run on an MI355X): RASR on the
head-summed score (lethe_rasr_select_shared) and Algorithm 1's segmented
shrinking with the size trigger (lethe_segmented_shrink), each followed by
compaction.  Given the same fp32 scores, keep masks, breakpoints, updated
thresholds and compacted rows must match the oracle bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2511_06029_amd import lethe as L
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def scores_of(rng, n, kind):
    if kind == "geometric":   # ranked values 2^0, 2^-1, ... at shuffled rows
        a = np.empty(n, np.float32)
        a[rng.permutation(n)] = np.float32(2.0) ** -np.minimum(np.arange(n), 120).astype(np.float32)
        return a
    if kind == "zero":
        return np.zeros(n, np.float32)
    return synth.score_vector(rng, n, kind)


def make_cache(lengths, L_, HK, seed, kind, D=64):
    """Cache with random bf16 K/V rows and scores from the seeded generator;
    returns (cache, scores)."""
    rng = np.random.default_rng(seed)
    caps = [n + 3 for n in lengths]
    c = L.LetheCache(L_, caps, HK, HK, D, dtype="bf16", device=DEV)
    s = {}
    for l in range(L_):
        for b, n in enumerate(lengths):
            for h in range(HK):
                v = scores_of(rng, n, kind)
                if kind == "ties" and h % 2:    # heads that cancel into exact ties
                    v = v[::-1].copy()
                s[l, b, h] = v
                start, _ = c.seg_rows(b, h)
                c.score[l, start:start + n] = torch.from_numpy(v).to(DEV)
                c.k[l, start:start + n] = torch.from_numpy(rng.standard_normal((n, D), np.float32)).to(DEV)
                c.v[l, start:start + n] = torch.from_numpy(rng.standard_normal((n, D), np.float32)).to(DEV)
            c.len[l, b] = n
    torch.cuda.synchronize()
    return c, s


def masks_of(c, keep, lengths, L_, HK):
    kh = keep.cpu().numpy()
    out = {}
    for l in range(L_):
        for b, n in enumerate(lengths):
            for h in range(HK):
                start, _ = c.seg_rows(b, h)
                got = kh[l, start:start + n]
                assert set(np.unique(got).tolist()) <= {0, 1}
                out[l, b, h] = got.astype(bool)
    return out


LENGTHS = [0, 1, 2, 63, 64, 65, 300, 1000, 4097]


@pytest.mark.parametrize("HK", [1, 3, 8])
@pytest.mark.parametrize("kind", ["zipf", "ties", "special"])
def test_rasr_select_shared_bit_exact(kind, HK):
    note("shared select %s HK=%d" % (kind, HK))
    L_ = 2
    c, s = make_cache(LENGTHS, L_, HK, 21 + HK, kind)
    B = len(LENGTHS)
    budgets = np.zeros((B, L_), np.int32)
    for b, n in enumerate(LENGTHS):
        for l in range(L_):
            budgets[b, l] = [0, 1, n // 3, n // 2, n - 1, n, n + 7, 40, -5][(b + 3 * l) % 9]
    for recent, sink in ((0, 0), (32, 4), (3000, 2)):
        keep = torch.full((L_, c.rows_per_layer), 7, dtype=torch.uint8, device=DEV)
        L.rasr_select_shared(c, torch.from_numpy(budgets).to(DEV), recent, sink, keep)
        torch.cuda.synchronize()
        got = masks_of(c, keep, LENGTHS, L_, HK)
        for l in range(L_):
            for b, n in enumerate(LENGTHS):
                sh = np.stack([s[l, b, h] for h in range(HK)]) if n else np.zeros((HK, 0), np.float32)
                want = oracle.rasr_select_shared(sh, budgets[b, l], recent, sink)
                for h in range(HK):
                    np.testing.assert_array_equal(got[l, b, h], want, err_msg="l%d b%d h%d" % (l, b, h))
    assert int(c.dev_status[0]) == 0


SHRINK_PARAMS = [(10, 400.0, 16, 0), (8, 2.0, 0, 0), (64, 30.0, 32, 4), (3, 1e6, 5, 2), (1, 4.0, 8, 1),
                 (1000, 1.0001, 7, 3)]


@pytest.mark.parametrize("kind", ["zipf", "geometric", "ties", "special", "zero"])
def test_segmented_shrink_bit_exact(kind):
    note("shrink %s" % kind)
    L_, HK = 3, 4
    c, s = make_cache(LENGTHS, L_, HK, 31, kind)
    B = len(LENGTHS)
    for segments, tau, recent, sink in SHRINK_PARAMS:
        # Thresholds below, at and above the length, and negative.
        thr = np.zeros((L_, B), np.int32)
        for l in range(L_):
            for b, n in enumerate(LENGTHS):
                thr[l, b] = [0, n - 1, n, n + 4, -3, n // 2, 2 ** 30 + 7][(l * B + b) % 7]
        ev = torch.from_numpy(thr).to(DEV)
        bp = torch.full((L_, B), 99, dtype=torch.int32, device=DEV)
        keep = torch.full((L_, c.rows_per_layer), 7, dtype=torch.uint8, device=DEV)
        L.segmented_shrink(c, segments, tau, recent, sink, ev, bp, keep)
        torch.cuda.synchronize()
        got = masks_of(c, keep, LENGTHS, L_, HK)
        evh, bph = ev.cpu().numpy(), bp.cpu().numpy()
        for l in range(L_):
            for b, n in enumerate(LENGTHS):
                a = oracle.head_sum_f32(np.stack([s[l, b, h] for h in range(HK)]) if n else
                                        np.zeros((HK, 0), np.float32))
                want, wbp, wlev = oracle.segmented_shrink(a, segments, tau, recent, sink, thr[l, b])
                what = "%s D=%d tau=%g l%d b%d n=%d thr=%d" % (kind, segments, tau, l, b, n, thr[l, b])
                assert (int(bph[l, b]), int(evh[l, b])) == (wbp, wlev), what
                for h in range(HK):
                    np.testing.assert_array_equal(got[l, b, h], want, err_msg=what)
    # Without a breakpoint array the thresholds still update.
    thr = np.zeros((L_, B), np.int32)
    ev = torch.from_numpy(thr).to(DEV)
    keep = torch.zeros((L_, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    L.segmented_shrink(c, 10, 400.0, 16, 0, ev, None, keep)
    torch.cuda.synchronize()
    for l in range(L_):
        for b, n in enumerate(LENGTHS):
            a = oracle.head_sum_f32(np.stack([s[l, b, h] for h in range(HK)]) if n else np.zeros((HK, 0), np.float32))
            assert int(ev[l, b]) == oracle.segmented_shrink(a, 10, 400.0, 16, 0, 0)[2]
    assert int(c.dev_status[0]) == 0


@pytest.mark.parametrize("rule", ["shared", "shrink"])
def test_shared_mask_compaction_end_to_end(rule):
    """Select, compact, then check every head's rows, scores and len."""
    note("shared-mask compaction %s" % rule)
    lengths = [5, 200, 2049, 40000]
    L_, HK = 2, 8
    c, s = make_cache(lengths, L_, HK, 41, "zipf", D=128)
    B = len(lengths)
    keep = torch.zeros((L_, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    recent, sink = 64, 4
    if rule == "shared":
        bud = np.array([[max(n // 3, 0)] * L_ for n in lengths], np.int32)
        L.rasr_select_shared(c, torch.from_numpy(bud).to(DEV), recent, sink, keep)
    else:
        thr = np.full((L_, B), 100, np.int32)
        L.segmented_shrink(c, 20, 50.0, recent, sink, torch.from_numpy(thr).to(DEV), None, keep)
    k_before = c.k.view(torch.int16).cpu().numpy()
    v_before = c.v.view(torch.int16).cpu().numpy()
    L.kv_compact(c, keep, c.workspace(L.OP_COMPACT))
    torch.cuda.synchronize()
    assert int(c.dev_status[0]) == 0
    lens = c.len.cpu().numpy()
    kk = c.k.view(torch.int16).cpu().numpy()
    vv = c.v.view(torch.int16).cpu().numpy()
    ss = c.score.cpu().numpy()
    for l in range(L_):
        for b, n in enumerate(lengths):
            sh = np.stack([s[l, b, h] for h in range(HK)])
            if rule == "shared":
                m = oracle.rasr_select_shared(sh, n // 3, recent, sink)
            else:
                m = oracle.segmented_shrink(oracle.head_sum_f32(sh), 20, 50.0, recent, sink, 100)[0]
            kept = np.flatnonzero(m)
            assert lens[l, b] == len(kept), (l, b)
            for h in range(HK):
                start, _ = c.seg_rows(b, h)
                e = start + len(kept)
                np.testing.assert_array_equal(kk[l, start:e], oracle.compact(k_before[l, start:start + n], m))
                np.testing.assert_array_equal(vv[l, start:e], oracle.compact(v_before[l, start:start + n], m))
                np.testing.assert_array_equal(ss[l, start:e].view(np.uint32),
                                              oracle.compact(s[l, b, h], m).view(np.uint32))


def test_shrink_large_segments_and_many_blocks():
    """64k-row sequences (several radix passes over large ranges) and a grid of
    more (layer, sequence) blocks than CUs."""
    note("shrink large")
    lengths = [65536, 1, 30000] + [700] * 125
    L_, HK = 3, 2
    c, s = make_cache(lengths, L_, HK, 51, "zipf", D=64)
    B = len(lengths)
    thr = np.zeros((L_, B), np.int32)
    ev = torch.from_numpy(thr).to(DEV)
    bp = torch.empty((L_, B), dtype=torch.int32, device=DEV)
    keep = torch.zeros((L_, c.rows_per_layer), dtype=torch.uint8, device=DEV)
    L.segmented_shrink(c, 100, 400.0, 128, 4, ev, bp, keep)
    torch.cuda.synchronize()
    got = masks_of(c, keep, lengths, L_, HK)
    bph, evh = bp.cpu().numpy(), ev.cpu().numpy()
    for l in range(L_):
        for b in list(range(4)) + [B - 1]:
            a = oracle.head_sum_f32(np.stack([s[l, b, h] for h in range(HK)]))
            want, wbp, wlev = oracle.segmented_shrink(a, 100, 400.0, 128, 4, 0)
            assert (int(bph[l, b]), int(evh[l, b])) == (wbp, wlev), (l, b)
            for h in range(HK):
                np.testing.assert_array_equal(got[l, b, h], want)
