"""Property tests of the oracle (hypothesis, CPU only).

Each property follows from the definitions the oracle implements, not from
its code, and is checked over generated shapes, lengths, ties and NaNs:

* RASR selection: exactly min(k, n) rows kept; the recent window and the
  sinks inside the budget kept; every kept candidate ranks above every
  evicted one (score descending, NaN last, lower index first).
* Budget split: nothing pruned when the sequence fits; infeasible floors keep
  everything; otherwise the budgets sum exactly to the global budget, stay
  between floor and cap, and a denser layer never gets more than one row
  less (above its floor) than a sparser uncapped one.
* Decode attention with the Eq. 5 update: outputs are convex combinations of
  the V rows; the update adds exactly one unit of attention per query head;
  permuting the rows permutes the scores and leaves the outputs unchanged;
  identical keys spread attention evenly.
* Hoyer sparsity (Eq. 1): in [0, 1], 1 for a one-hot vector, 0 for a constant
  one, and invariant under positive scaling.
* Compaction keeps the kept rows in order.
"""
import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle

SETTINGS = settings(max_examples=80, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def rank_key(s, j):
    v = float(s[j])
    return (1, 0.0, j) if math.isnan(v) else (0, -v, j)


@st.composite
def score_vectors(draw):
    n = draw(st.integers(0, 200))
    kind = draw(st.sampled_from(["ties", "floats", "nan"]))
    if kind == "ties":
        vals = draw(st.lists(st.integers(0, 3), min_size=n, max_size=n))
        return np.array(vals, np.float32)
    vals = draw(st.lists(st.floats(-1e3, 1e3, allow_nan=False, width=32), min_size=n, max_size=n))
    s = np.array(vals, np.float32)
    if kind == "nan" and n:
        idx = draw(st.lists(st.integers(0, n - 1), max_size=max(1, n // 4)))
        s[idx] = np.nan
    return s


@SETTINGS
@given(s=score_vectors(), k=st.integers(0, 220), recent=st.integers(0, 40), sink=st.integers(0, 8))
def test_rasr_select_properties(s, k, recent, sink):
    n = len(s)
    keep = oracle.rasr_select(s, k, recent, sink)
    assert keep.shape == (n,)
    assert keep.sum() == min(k, n)
    if k >= n:
        return
    r = min(recent, k)
    sk = min(sink, k - r)
    assert keep[n - r:].all() and keep[:sk].all()
    cand = np.arange(sk, n - r)
    kept = [j for j in cand if keep[j]]
    evicted = [j for j in cand if not keep[j]]
    if kept and evicted:
        worst_kept = max(rank_key(s, j) for j in kept)
        best_evicted = min(rank_key(s, j) for j in evicted)
        assert worst_kept < best_evicted


@st.composite
def budget_cases(draw):
    L = draw(st.integers(1, 12))
    n = draw(st.lists(st.integers(0, 3000), min_size=L, max_size=L))
    S = draw(st.lists(st.one_of(st.floats(-0.5, 1.5, width=32), st.just(float("nan"))), min_size=L, max_size=L))
    recent = draw(st.integers(0, 300))
    sink = draw(st.integers(0, 8))
    total = draw(st.integers(0, sum(n) + 100))
    return np.array(n, np.int32), np.array(S, np.float32), recent, sink, total


def density_weight(S):
    """1 + floor((1 - S clamped to [0, 1], NaN as 0) * 2^24), in fp32."""
    Sc = np.where(np.isnan(S), np.float32(0), np.clip(S, np.float32(0), np.float32(1))).astype(np.float32)
    return 1 + np.floor((np.float32(1) - Sc) * np.float32(16777216.0)).astype(np.int64)


@SETTINGS
@given(case=budget_cases())
def test_budget_split_properties(case):
    n, S, recent, sink, total = case
    b, infeasible = oracle.budget_split(n, S, recent, sink, total)
    f = np.minimum(n, recent + sink)
    if n.sum() <= total:
        assert not infeasible
        np.testing.assert_array_equal(b, n)
        return
    if f.sum() > total:
        assert infeasible
        np.testing.assert_array_equal(b, n)
        return
    assert not infeasible
    assert int(b.sum()) == total
    assert (b >= f).all() and (b <= n).all()
    w = density_weight(S)
    free = (b > f) & (b < n)  # layers neither at their floor nor capped
    idx = np.flatnonzero((n > f) & (b < n))
    for l in idx:
        for m in idx:
            if w[l] > w[m] and free[m]:
                assert b[l] - f[l] >= b[m] - f[m] - 1, (l, m, b, f, w)


@st.composite
def attention_cases(draw):
    n = draw(st.integers(1, 96))
    G = draw(st.integers(1, 8))
    D = draw(st.sampled_from([4, 16, 64]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    gamma = draw(st.floats(0.05, 1.0))
    return n, G, D, seed, gamma


@SETTINGS
@given(case=attention_cases())
def test_attend_properties(case):
    n, G, D, seed, gamma = case
    rng = np.random.default_rng(seed)
    q = (2 * rng.standard_normal((G, D))).astype(np.float32)
    K = rng.standard_normal((n, D)).astype(np.float32)
    V = rng.standard_normal((n, D)).astype(np.float32)
    s_in = rng.random(n) * 5
    scale = 1 / math.sqrt(D)
    out, s_out = oracle.attend(q, K, V, s_in, gamma, scale)
    lo, hi = V.min(axis=0).astype(np.float64), V.max(axis=0).astype(np.float64)
    assert (out >= lo - 1e-9).all() and (out <= hi + 1e-9).all()
    added = s_out - gamma * s_in
    assert (added >= -1e-12).all()
    assert abs(added.sum() - G) <= 1e-9 * G
    perm = rng.permutation(n)
    out_p, s_out_p = oracle.attend(q, K[perm], V[perm], s_in[perm], gamma, scale)
    np.testing.assert_allclose(out_p, out, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s_out_p, s_out[perm], rtol=1e-12, atol=1e-12)
    # Identical keys: every row gets 1/n of each head's attention.
    Kc = np.repeat(K[:1], n, axis=0)
    out_c, s_c = oracle.attend(q, Kc, V, None, gamma, scale)
    np.testing.assert_allclose(out_c, np.repeat(V.astype(np.float64).mean(axis=0)[None], G, axis=0),
                               rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s_c, np.full(n, G / n), rtol=1e-10)


@SETTINGS
@given(a=st.lists(st.floats(0, 1e4, allow_nan=False), min_size=0, max_size=100), c=st.floats(1e-3, 1e3))
def test_hoyer_properties(a, c):
    a = np.array(a, np.float64)
    h = oracle.hoyer(a)
    assert 0.0 <= h <= 1.0 + 1e-12
    if len(a) > 1 and a.sum() > 0:
        assert abs(oracle.hoyer(c * a) - h) <= 1e-9
    if len(a) > 1:
        one_hot = np.zeros(len(a))
        one_hot[len(a) // 2] = 3.0
        assert abs(oracle.hoyer(one_hot) - 1.0) <= 1e-12
        assert abs(oracle.hoyer(np.full(len(a), 2.5))) <= 1e-12


@SETTINGS
@given(keep=st.lists(st.booleans(), min_size=0, max_size=300))
def test_compact_keeps_order(keep):
    keep = np.array(keep, bool)
    rows = np.arange(len(keep) * 3, dtype=np.int64).reshape(len(keep), 3)
    out = oracle.compact(rows, keep)
    assert out.shape == (int(keep.sum()), 3)
    if len(out) > 1:
        assert (np.diff(out[:, 0]) > 0).all()
    assert set(out[:, 0].tolist()) == {3 * j for j in np.flatnonzero(keep)}
