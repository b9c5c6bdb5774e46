"""Pins of the oracle to facts other than itself (CPU only).

The paper prints no worked example and no intermediate values for any step,
so every pin here is a closed form, an invariant, a special case that reduces
to an independent library routine (torch's scaled_dot_product_attention,
numpy's lexsort), or exact rational arithmetic.  Each is chosen so that a
plausible slip in the oracle (a dropped term, a wrong axis, a sign, an
off-by-one in a window) fails at least one test.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from workloads import synth

RNG = np.random.default_rng


# --------------------------------------------------------------------------
# Eq. 1 (Hoyer sparsity)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n", [2, 3, 7, 64, 1000])
def test_hoyer_one_hot_is_one(n):
    a = np.zeros(n)
    a[n // 3] = 2.5
    assert oracle.hoyer(a) == pytest.approx(1.0, abs=1e-12)


@pytest.mark.parametrize("n", [2, 5, 128, 4097])
def test_hoyer_uniform_is_zero(n):
    assert oracle.hoyer(np.full(n, 0.37)) == pytest.approx(0.0, abs=1e-12)


@pytest.mark.parametrize("n,k", [(4, 2), (100, 1), (100, 7), (1024, 512), (9, 8)])
def test_hoyer_k_equal_nonzeros_closed_form(n, k):
    a = np.zeros(n)
    a[RNG(n * 31 + k).choice(n, k, replace=False)] = 1.7
    want = (math.sqrt(n) - math.sqrt(k)) / (math.sqrt(n) - 1)
    assert oracle.hoyer(a) == pytest.approx(want, abs=1e-12)


def test_hoyer_scale_and_permutation_invariant():
    a = RNG(3).random(333) ** 4
    S = oracle.hoyer(a)
    assert 0.0 < S < 1.0
    assert oracle.hoyer(a * 1e-7) == pytest.approx(S, rel=1e-12)
    assert oracle.hoyer(a * 3e5) == pytest.approx(S, rel=1e-12)
    assert oracle.hoyer(a[RNG(4).permutation(333)]) == pytest.approx(S, rel=1e-12)


def test_hoyer_degenerate():
    assert oracle.hoyer(np.array([])) == 0.0
    assert oracle.hoyer(np.array([5.0])) == 0.0
    assert oracle.hoyer(np.zeros(10)) == 0.0


def test_layer_sparsity_sums_heads_before_hoyer():
    # Splitting one score vector across heads in arbitrary proportions must not
    # change the layer sparsity (Eq. 2 sums heads first); a per-head Hoyer
    # average would.
    rng = RNG(5)
    a = rng.random(200) ** 6
    t = rng.random(200)
    heads = np.stack([a * t, a * (1 - t) * 0.5, a * (1 - t) * 0.5])
    assert oracle.layer_sparsity(heads) == pytest.approx(oracle.hoyer(a), rel=1e-12)
    per_head_mean = np.mean([oracle.hoyer(h) for h in heads])
    assert abs(per_head_mean - oracle.hoyer(a)) > 1e-3


# --------------------------------------------------------------------------
# Decode attention and Eq. 5
# --------------------------------------------------------------------------

def _sdpa(q, K, V, scale):
    """torch's attention in float64 on the CPU: q (G, D), K/V (n, D)."""
    qt = torch.from_numpy(np.asarray(q, np.float64))[None, :, None, :]     # (1, G, 1, D)
    Kt = torch.from_numpy(np.asarray(K, np.float64))[None, None].expand(1, q.shape[0], -1, -1)
    Vt = torch.from_numpy(np.asarray(V, np.float64))[None, None].expand(1, q.shape[0], -1, -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, Kt.contiguous(), Vt.contiguous(), scale=scale)
    return o[0, :, 0, :].numpy()


@pytest.mark.parametrize("n,D,G", [(1, 64, 2), (5, 64, 1), (37, 64, 4), (129, 128, 7), (300, 128, 8)])
def test_attend_matches_library_attention(n, D, G):
    rng = RNG(n * 7 + G)
    q, K, V = synth.random_segment(rng, n, D, G, scale_k=2.0)
    scale = 1 / math.sqrt(D)
    out, s = oracle.attend(q, K, V, None, 0.9, scale)
    np.testing.assert_allclose(out, _sdpa(q, K, V, scale), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("n,G", [(3, 1), (40, 4), (64, 7)])
def test_score_increment_is_attention_probabilities(n, G):
    # With one-hot value rows the attention output *is* the probability
    # vector, so the library routine exposes p; Eq. 5 adds sum_g p_g.
    D = 64
    rng = RNG(11 + n)
    q, K, _ = synth.random_segment(rng, n, D, G, scale_k=3.0)
    V = np.zeros((n, D), np.float32)
    V[np.arange(n), np.arange(n)] = 1.0
    scale = 1 / math.sqrt(D)
    p = _sdpa(q, K, V, scale)[:, :n]                         # (G, n)
    s_in = rng.random(n)
    gamma = 0.75
    _, s_out = oracle.attend(q, K, V, s_in, gamma, scale)
    np.testing.assert_allclose(s_out, gamma * s_in + p.sum(axis=0), rtol=1e-12, atol=1e-14)


def test_two_token_closed_form():
    D = 64
    rng = RNG(12)
    q, K, V = synth.random_segment(rng, 2, D, 1)
    scale = 0.3
    x = scale * (K.astype(np.float64) @ q[0].astype(np.float64))
    p1 = 1 / (1 + math.exp(-(x[1] - x[0])))
    out, s = oracle.attend(q, K, V, None, 0.5, scale)
    assert s[1] == pytest.approx(p1, rel=1e-12)
    assert s[0] == pytest.approx(1 - p1, rel=1e-12)
    V64 = V.astype(np.float64)
    np.testing.assert_allclose(out[0], (1 - p1) * V64[0] + p1 * V64[1], rtol=1e-11, atol=1e-12)


def test_zero_query_gives_uniform_attention():
    n, D, G = 50, 128, 4
    rng = RNG(13)
    _, K, V = synth.random_segment(rng, n, D, G)
    out, s = oracle.attend(np.zeros((G, D), np.float32), K, V, np.ones(n), 0.5, 0.1)
    for g in range(G):
        np.testing.assert_allclose(out[g], V.astype(np.float64).mean(axis=0), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(s, 0.5 + G / n, rtol=1e-13)


def test_single_row_and_empty():
    D, G = 64, 3
    rng = RNG(14)
    q, K, V = synth.random_segment(rng, 1, D, G)
    out, s = oracle.attend(q, K, V, np.array([2.0]), 0.25, 0.125)
    np.testing.assert_allclose(out, np.repeat(V.astype(np.float64), G, axis=0), rtol=0, atol=0)
    assert s[0] == pytest.approx(0.5 + G, rel=1e-15)
    out0, s0 = oracle.attend(q, K[:0], V[:0], None, 0.9, 0.125)
    assert out0.shape == (G, D) and not out0.any() and s0.shape == (0,)


def test_mass_invariant_and_decay_closed_form():
    # From zero scores, with no pruning and no appends, t steps give
    # sum_j s_t[j] = G (1 - gamma^t) / (1 - gamma); gamma = 1 gives G t.
    n, D, G = 97, 64, 4
    rng = RNG(15)
    _, K, V = synth.random_segment(rng, n, D, G)
    for gamma in (0.5, 0.9, 0.99, 1.0):
        s = np.zeros(n)
        for t in range(1, 13):
            q = rng.standard_normal((G, D)).astype(np.float32)
            _, s = oracle.attend(q, K, V, s, gamma, 1 / 8)
            want = G * t if gamma == 1.0 else G * (1 - gamma ** t) / (1 - gamma)
            assert s.sum() == pytest.approx(want, rel=1e-12)
            assert (s >= 0).all()


def test_gamma_one_is_cumulative_attention():
    # gamma = 1 is plain accumulated attention (the heavy-hitter score of H2O).
    n, D, G = 30, 64, 2
    rng = RNG(16)
    _, K, _ = synth.random_segment(rng, n, D, G, scale_k=2.0)
    V = np.zeros((n, D), np.float32)
    V[np.arange(n), np.arange(n)] = 1.0
    s = np.zeros(n)
    acc = np.zeros(n)
    for t in range(6):
        q = rng.standard_normal((G, D)).astype(np.float32)
        acc += _sdpa(q, K, V, 0.125)[:, :n].sum(axis=0)
        _, s = oracle.attend(q, K, V, s, 1.0, 0.125)
    np.testing.assert_allclose(s, acc, rtol=1e-12)


def test_cache_gqa_mapping_matches_repeat_interleave():
    # Eq. 3: keys repeated H_Q/H_KV times along the head axis (interleaved):
    # query head i reads KV head i // G.
    L, B, HQ, HK, D = 1, 2, 8, 2, 64
    G = HQ // HK
    rng = RNG(17)
    cache = oracle.OracleCache(L, B, HQ, HK, D)
    Ks = rng.standard_normal((B, HK, 20, D)).astype(np.float32)
    Vs = rng.standard_normal((B, HK, 20, D)).astype(np.float32)
    for b in range(B):
        for h in range(HK):
            cache.set_segment(0, b, h, Ks[b, h], Vs[b, h])
    q = rng.standard_normal((B, HQ, D)).astype(np.float32)
    out = cache.decode_step(0, q, None, None, 0.9, 1 / 8)
    Kr = torch.from_numpy(Ks.astype(np.float64)).repeat_interleave(G, dim=1)
    Vr = torch.from_numpy(Vs.astype(np.float64)).repeat_interleave(G, dim=1)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q.astype(np.float64))[:, :, None, :], Kr, Vr, scale=1 / 8)[:, :, 0, :]
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_cache_append_attends_to_new_token():
    L, B, HQ, HK, D = 1, 1, 2, 1, 64
    cache = oracle.OracleCache(L, B, HQ, HK, D)
    rng = RNG(18)
    q = rng.standard_normal((1, HQ, D)).astype(np.float32)
    kn = rng.standard_normal((1, HK, D)).astype(np.float32)
    vn = rng.standard_normal((1, HK, D)).astype(np.float32)
    out = cache.decode_step(0, q, kn, vn, 0.9, 0.125)
    np.testing.assert_array_equal(out[0], np.repeat(vn[0].astype(np.float64), HQ, axis=0))
    assert cache.s[0][0][0].tolist() == [2.0]


# --------------------------------------------------------------------------
# Budget split (reading of the paper's layerwise allocation)
# --------------------------------------------------------------------------

def _weights32(S):
    S = np.clip(np.nan_to_num(np.asarray(S, np.float32), nan=0.0), 0, 1).astype(np.float32)
    return 1 + np.floor((np.float32(1.0) - S) * np.float32(16777216.0)).astype(np.int64)


def _budget_cases():
    rng = RNG(21)
    cases = []
    for _ in range(300):
        L = int(rng.integers(1, 40))
        n = rng.integers(0, 3000, size=L).astype(np.int32)
        if rng.random() < 0.3:
            n[:] = n[0]
        S = rng.random(L).astype(np.float32)
        if rng.random() < 0.2:
            S[rng.integers(0, L)] = np.float32(rng.choice([0.0, 1.0, np.nan]))
        recent = int(rng.integers(0, 300))
        sink = int(rng.integers(0, 8))
        frac = rng.uniform(0.05, 1.1)
        Gb = int(frac * n.sum())
        cases.append((n, S, recent, sink, Gb))
    return cases


def test_budget_invariants():
    for n, S, recent, sink, Gb in _budget_cases():
        b, infeasible = oracle.budget_split(n, S, recent, sink, Gb)
        f = np.minimum(n, recent + sink)
        if n.sum() <= Gb:
            assert not infeasible and (b == n).all()
        elif f.sum() > Gb:
            assert infeasible and (b == n).all()
        else:
            assert not infeasible
            assert int(b.sum()) == Gb
            assert (b >= f).all() and (b <= n).all()


def test_budget_hamilton_quota_rule_exact_rational():
    # When no cap binds, each layer receives floor or ceil of its exact
    # proportional quota R * w_l / W (Hamilton's largest-remainder property),
    # and the ceil goes to the largest fractional parts, ties to lower l.
    rng = RNG(22)
    checked = 0
    for _ in range(400):
        L = int(rng.integers(1, 40))
        n = [int(x) for x in rng.integers(500, 5000, size=L)]
        S = rng.random(L).astype(np.float32)
        if rng.random() < 0.3:
            S[:] = S[0]
        recent, sink = int(rng.integers(0, 200)), int(rng.integers(0, 8))
        Gb = int(rng.uniform(0.1, 0.3) * sum(n))
        f = [min(x, recent + sink) for x in n]
        if sum(f) > Gb:
            continue
        A = [l for l in range(L) if n[l] > f[l]]
        w = [int(x) for x in _weights32(S)]
        R = Gb - sum(f)
        W = sum(w[l] for l in A)
        quota = {l: Fraction(R * w[l], W) for l in A}
        if any(f[l] + math.ceil(quota[l]) > n[l] - 1 for l in A):
            continue                           # a cap may bind: covered elsewhere
        b, inf = oracle.budget_split(np.array(n, np.int32), S, recent, sink, Gb)
        assert not inf and int(b.sum()) == Gb
        for l in A:
            assert math.floor(quota[l]) <= int(b[l]) - f[l] <= math.ceil(quota[l])
        frac = {l: quota[l] - math.floor(quota[l]) for l in A}
        up = [l for l in A if int(b[l]) - f[l] > math.floor(quota[l])]
        down = [l for l in A if int(b[l]) - f[l] == math.floor(quota[l]) and frac[l] > 0]
        for u in up:
            for d in down:
                assert frac[u] > frac[d] or (frac[u] == frac[d] and u < d)
        checked += 1
    assert checked > 100


def test_budget_equal_sparsity_splits_evenly():
    L = 7
    n = np.full(L, 1000, np.int32)
    S = np.full(L, 0.8, np.float32)
    # Floors 16 each leave 3003 - 112 = 2891 = 7 * 413: an exact split.
    b, _ = oracle.budget_split(n, S, 16, 0, 3003)
    assert b.tolist() == [429] * 7
    # 2893 = 7 * 413 + 2: equal remainders, so the two leftover rows go to the
    # two lowest layers.
    b, _ = oracle.budget_split(n, S, 16, 0, 3005)
    assert b.tolist() == [430, 430, 429, 429, 429, 429, 429]


def test_budget_denser_layers_get_more():
    L = 6
    n = np.full(L, 4000, np.int32)
    S = np.array([0.9, 0.2, 0.5, 0.95, 0.0, 0.7], np.float32)
    b, _ = oracle.budget_split(n, S, 64, 4, 6000)
    order = np.argsort(S, kind="stable")
    assert all(b[order[i]] >= b[order[i + 1]] for i in range(L - 1))
    assert b.sum() == 6000


def test_budget_caps_redistribute():
    n = np.array([10, 5000, 5000, 300], np.int32)
    S = np.zeros(4, np.float32)
    b, inf = oracle.budget_split(n, S, 8, 0, 4000)
    assert not inf and b.sum() == 4000 and b[0] == 10 and b[3] == 300
    assert abs(int(b[1]) - int(b[2])) <= 1


# --------------------------------------------------------------------------
# RASR selection and compaction
# --------------------------------------------------------------------------

def _select_cases():
    rng = RNG(31)
    for kind in ("zipf", "ties", "special", "uniform"):
        for n in (0, 1, 2, 5, 31, 64, 257, 1000):
            for k in sorted({0, 1, n // 3, n // 2, max(n - 1, 0), n, n + 5}):
                for recent, sink in ((0, 0), (3, 0), (16, 4), (n + 2, 1)):
                    yield synth.score_vector(rng, n, kind), k, recent, sink


def _order_key_rank(s, cand):
    """Library ordering of candidates: numpy lexsort by (-value, index) with
    NaN last (numpy sorts NaN after every number) and -0 == +0."""
    v = -s[cand].astype(np.float64)
    return cand[np.lexsort((cand, v))]


def test_select_matches_library_sort_and_invariants():
    for s, k, recent, sink in _select_cases():
        n = len(s)
        keep = oracle.rasr_select(s, k, recent, sink)
        assert keep.shape == (n,)
        assert keep.sum() == min(n, max(k, 0))
        if k >= n:
            assert keep.all()
            continue
        r = min(recent, k)
        sk = min(sink, k - r)
        m = k - r - sk
        assert keep[n - r:].all() and keep[:sk].all()
        cand = np.arange(sk, n - r)
        ranked = _order_key_rank(s, cand)
        want = np.zeros(n, bool)
        want[:sk] = True
        want[n - r:] = True
        want[ranked[:m]] = True
        np.testing.assert_array_equal(keep, want)


def test_select_streaming_case_ignores_scores():
    # budget = recent + sink: the kept set is the StreamingLLM set whatever s is.
    rng = RNG(32)
    for _ in range(20):
        s = synth.score_vector(rng, 500, "zipf")
        keep = oracle.rasr_select(s, 68, 64, 4)
        want = np.zeros(500, bool)
        want[:4] = True
        want[-64:] = True
        np.testing.assert_array_equal(keep, want)


def test_select_ties_lower_index_nan_last_signed_zero():
    s = np.array([1.0, np.nan, 1.0, -0.0, 0.0, 2.0, 1.0], np.float32)
    keep = oracle.rasr_select(s, 3, 0, 0)
    assert keep.tolist() == [True, False, True, False, False, True, False]
    keep = oracle.rasr_select(s, 5, 0, 0)
    assert keep.tolist() == [True, False, True, True, False, True, True]
    keep = oracle.rasr_select(s, 6, 0, 0)
    assert keep.tolist() == [True, False, True, True, True, True, True]


def test_select_budget_smaller_than_window():
    s = np.arange(10, dtype=np.float32)
    keep = oracle.rasr_select(s, 3, 5, 2)
    assert keep.tolist() == [False] * 7 + [True] * 3


def test_compact_preserves_order_and_bytes():
    rng = RNG(33)
    rows = rng.integers(0, 2 ** 16, size=(100, 64), dtype=np.uint16)
    keep = rng.random(100) < 0.4
    out = oracle.compact(rows, keep)
    idx = np.flatnonzero(keep)
    assert out.shape == (len(idx), 64)
    for i, j in enumerate(idx):
        assert (out[i] == rows[j]).all()
    np.testing.assert_array_equal(oracle.compact(rows, np.ones(100, bool)), rows)


def test_prune_round_keeps_exactly_the_budgets():
    L, B, HQ, HK, D = 3, 2, 4, 2, 64
    rng = RNG(34)
    cache = oracle.OracleCache(L, B, HQ, HK, D)
    for l in range(L):
        for b in range(B):
            for h in range(HK):
                n = 200 + 50 * l
                cache.set_segment(l, b, h, rng.standard_normal((n, D)), rng.standard_normal((n, D)),
                                  synth.score_vector(rng, n, "zipf").astype(np.float64))
    Gb = [300, 450]
    S, budget, inf = cache.prune_round(Gb, 16, 2)
    assert not inf.any()
    for b in range(B):
        assert budget[b].sum() == Gb[b]
        for l in range(L):
            for h in range(HK):
                assert cache.K[l][b][h].shape[0] == budget[b, l]


def _rank_keep(s32, k, recent, sink):
    """Independent selection on fp32 scores: the protected windows (recent
    first, then sinks, both within k), then the rest by numpy's lexsort on
    (score descending with NaN last, row ascending)."""
    n = len(s32)
    keep = np.zeros(n, bool)
    if k >= n:
        keep[:] = True
        return keep
    k = max(k, 0)
    r = min(recent, k)
    sk = min(sink, k - r)
    keep[n - r:] = True
    keep[:sk] = True
    cand = np.arange(sk, n - r)
    v = s32[cand].astype(np.float64)
    nan = np.isnan(v)
    order = np.lexsort((cand, np.where(nan, 0.0, -v), nan))
    keep[cand[order[:k - r - sk]]] = True
    return keep


@pytest.mark.parametrize("given_sparsity", [False, True])
def test_prune_round_composition(given_sparsity):
    """The whole round against its parts recomposed independently: each
    (layer, sequence)'s sparsity from its own heads' summed scores (Hoyer in
    numpy), the split fed those values in fp32, each head's kept set from its
    own fp32 scores and its layer's budget, and K, V and scores compacted with
    the same mask.  Segments carry distinct values, so a crossed layer,
    sequence or head shows."""
    L, B, HQ, HK, D = 4, 3, 6, 3, 16
    rng = RNG(77)
    cache = oracle.OracleCache(L, B, HQ, HK, D)
    orig = {}
    for l in range(L):
        for b in range(B):
            n = 60 + 37 * l + 11 * b
            for h in range(HK):
                K = rng.standard_normal((n, D)).astype(np.float32) + 100 * l + 10 * b + h
                V = rng.standard_normal((n, D)).astype(np.float32) - 100 * l - 10 * b - h
                s = synth.score_vector(rng, n, "zipf").astype(np.float64) * (1 + 0.3 * h + 0.1 * l)
                s[rng.integers(0, n, 3)] = s[0]  # some ties
                cache.set_segment(l, b, h, K, V, s)
                orig[l, b, h] = (K.copy(), V.copy(), s.copy())
    recent, sink = 8, 2
    Gb = [L * 40, L * 55, L * 30]
    s_in = None
    if given_sparsity:
        s_in = [[float(rng.random()) for _ in range(L)] for _ in range(B)]
    S, budget, inf = cache.prune_round(Gb, recent, sink, sparsity_in=s_in)
    for b in range(B):
        S_ind = np.zeros(L)
        for l in range(L):
            if given_sparsity:
                S_ind[l] = s_in[b][l]
            else:
                a = sum(orig[l, b, h][2] for h in range(HK))
                n = len(a)
                l1, l2 = np.abs(a).sum(), math.sqrt((a * a).sum())
                S_ind[l] = min(max((math.sqrt(n) - l1 / l2) / (math.sqrt(n) - 1), 0.0), 1.0)
        np.testing.assert_allclose(S[b], S_ind, rtol=1e-12, atol=1e-14)
        n_l = np.array([len(orig[l, b, 0][2]) for l in range(L)], np.int32)
        bud, infb = oracle.budget_split(n_l, S_ind.astype(np.float32), recent, sink, Gb[b])
        np.testing.assert_array_equal(budget[b], bud)
        assert inf[b] == infb
        for l in range(L):
            for h in range(HK):
                K, V, s = orig[l, b, h]
                keep = _rank_keep(s.astype(np.float32), int(budget[b, l]), recent, sink)
                np.testing.assert_array_equal(cache.K[l][b][h], K[keep])
                np.testing.assert_array_equal(cache.V[l][b][h], V[keep])
                np.testing.assert_array_equal(cache.s[l][b][h], s[keep])
