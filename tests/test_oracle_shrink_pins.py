"""Pins of the oracle's head-shared selection and of Algorithm 1 (segmented
token shrinking with the size trigger) to facts other than the oracle itself
(CPU only).

The paper prints Algorithm 1 but no worked example, so the pins are closed
forms (geometric score vectors whose breakpoint follows from powers of two),
special cases (uniform, all-zero and one-hot scores, an untriggered cache,
no cut points), an independent route to the breakpoint (the ratio test is
monotone along the ranking, so the breakpoint is the first cut at or after the
number of tokens whose tau-scaled score exceeds the head), numpy's lexsort for
the ranking, and numpy's own fp32 additions for the head sum.
"""
import numpy as np
import pytest

import oracle
from workloads import synth

RNG = np.random.default_rng
NOT_TRIGGERED, NO_BREAKPOINT = oracle.SHRINK_NOT_TRIGGERED, oracle.SHRINK_NO_BREAKPOINT


def _ranked(a):
    """Indices of a in the order (value desc, index asc), NaN last, -0 == +0,
    by numpy's lexsort on fp64 values (numpy sorts NaN after numbers)."""
    idx = np.arange(len(a))
    return idx[np.lexsort((idx, -a.astype(np.float64)))]


# --------------------------------------------------------------------------
# Head-summed selection score (Eq. 2 over KV heads) and the shared RASR mask
# --------------------------------------------------------------------------

def test_head_sum_rounds_in_fp32_after_each_head():
    # 1 + 2^-24 rounds back to 1 (ties to even) at every step in fp32, while an
    # exact sum would be 1 + 2^-23, a representable fp32 value.
    s = np.array([[1.0], [2.0 ** -24], [2.0 ** -24]], np.float32)
    assert oracle.head_sum_f32(s)[0] == np.float32(1.0)
    # Summed in the other order the small terms combine first.
    assert oracle.head_sum_f32(s[::-1].copy())[0] == np.float32(1.0 + 2.0 ** -23)


def test_head_sum_matches_numpy_fp32_additions():
    rng = RNG(41)
    for H in (1, 2, 3, 7, 8):
        s = rng.random((H, 333)).astype(np.float32) * rng.choice([1e-3, 1.0, 1e3], size=(H, 1)).astype(np.float32)
        want = s[0].copy()
        for h in range(1, H):
            want = np.add(want, s[h], dtype=np.float32)
        np.testing.assert_array_equal(oracle.head_sum_f32(s), want)


def test_shared_select_single_head_is_per_segment_select():
    rng = RNG(42)
    for n in (0, 1, 17, 300):
        s = synth.score_vector(rng, n, "zipf")
        for k, recent, sink in ((n // 2, 8, 2), (n, 0, 0), (3, 16, 4)):
            np.testing.assert_array_equal(oracle.rasr_select_shared(s[None], k, recent, sink),
                                          oracle.rasr_select(s, k, recent, sink))


def test_shared_select_identical_heads_is_per_segment_select():
    # Four equal heads sum exactly to 4 s, which ranks like s.
    rng = RNG(43)
    s = synth.score_vector(rng, 500, "zipf")
    np.testing.assert_array_equal(oracle.rasr_select_shared(np.stack([s] * 4), 200, 32, 4),
                                  oracle.rasr_select(s, 200, 32, 4))


def test_shared_select_ranks_the_head_sum():
    rng = RNG(44)
    for n in (64, 257, 1000):
        s = np.stack([synth.score_vector(rng, n, "zipf") for _ in range(4)])
        a = ((s[0] + s[1]) + s[2]) + s[3]
        k, recent, sink = n // 3, 16, 4
        keep = oracle.rasr_select_shared(s, k, recent, sink)
        assert keep.sum() == k
        cand = np.arange(sink, n - recent)
        top = cand[np.lexsort((cand, -a[cand].astype(np.float64)))][:k - recent - sink]
        want = np.zeros(n, bool)
        want[:sink] = want[n - recent:] = True
        want[top] = True
        np.testing.assert_array_equal(keep, want)


# --------------------------------------------------------------------------
# Algorithm 1: segmented token shrinking
# --------------------------------------------------------------------------

def _geometric(n, rng):
    """Scores 2^0, 2^-1, ..., 2^-(n-1) at shuffled positions: the c-th ranked
    value is 2^-c, so the head-to-cut ratio at cut c is exactly 2^c."""
    perm = rng.permutation(n)
    a = np.empty(n, np.float32)
    a[perm] = np.float32(2.0) ** -np.arange(n, dtype=np.float32)
    return a, perm


@pytest.mark.parametrize("n,D,tau", [(64, 8, 400.0), (100, 10, 400.0), (100, 10, 2.0), (50, 4, 1e6),
                                     (37, 5, 3.0), (90, 3, 2.0 ** 40), (20, 20, 1.5)])
def test_shrink_geometric_closed_form(n, D, tau):
    rng = RNG(n * 7 + D)
    a, perm = _geometric(n, rng)
    recent, sink, L0 = 3, 2, 5
    keep, bp, lev = oracle.segmented_shrink(a, D, tau, recent, sink, L0)
    cuts = [(n * d) // D for d in range(1, D)]
    hits = [c for c in cuts if 2.0 ** c >= tau]
    if not hits:
        assert bp == NO_BREAKPOINT and keep.all() and lev == 2 * L0
        return
    want_bp = hits[0]
    assert bp == want_bp
    want = np.zeros(n, bool)
    want[:sink] = True
    want[n - recent:] = True
    want[perm[:want_bp]] = True          # positions of 2^0 ... 2^-(bp-1)
    np.testing.assert_array_equal(keep, want)
    assert lev == max(L0, want_bp + recent)


def test_shrink_reads_breakpoint_as_ratio_reaching_tau():
    # Ratio 2^8 at the first cut is below tau = 400, 2^16 at the second is
    # above: the breakpoint is the second cut (a literal "<= tau" test would
    # stop at the first).
    a, _ = _geometric(64, RNG(5))
    _, bp, _ = oracle.segmented_shrink(a, 8, 400.0, 0, 0, 0)
    assert bp == 16
    # tau exactly equal to a ratio counts as reaching it.
    _, bp, _ = oracle.segmented_shrink(a, 8, 256.0, 0, 0, 0)
    assert bp == 8
    _, bp, _ = oracle.segmented_shrink(a, 8, float(np.nextafter(np.float32(256.0), np.float32(1e9))), 0, 0, 0)
    assert bp == 16


def test_shrink_uniform_and_zero_scores_delay_pruning():
    for a in (np.full(200, 0.25, np.float32), np.zeros(200, np.float32)):
        keep, bp, lev = oracle.segmented_shrink(a, 10, 4.0, 16, 4, 150)
        assert bp == NO_BREAKPOINT and keep.all() and lev == 300


def test_shrink_one_hot_cuts_at_first_nonzero_cut():
    n, D, hot = 120, 6, 77
    a = np.zeros(n, np.float32)
    a[hot] = 3.0
    keep, bp, lev = oracle.segmented_shrink(a, D, 400.0, 10, 2, 0)
    assert bp == n // D                           # v_cut = 0 gives an infinite ratio
    want = np.zeros(n, bool)
    want[:2] = True
    want[n - 10:] = True
    want[hot] = True
    zeros_in_order = [j for j in range(n) if j != hot][:bp - 1]   # ties by index
    want[zeros_in_order] = True
    np.testing.assert_array_equal(keep, want)
    assert lev == bp + 10


def test_shrink_cut_at_rank_zero_never_qualifies():
    # n < D puts the first cuts at rank 0, where the ratio is 1 < tau.
    a = np.array([5.0, 0.0, 0.0], np.float32)
    _, bp, _ = oracle.segmented_shrink(a, 8, 2.0, 0, 0, 0)
    assert bp == (3 * 3) // 8 == 1


def test_shrink_not_triggered_at_or_below_threshold():
    a, _ = _geometric(64, RNG(6))
    for L0 in (64, 65, 1000):
        keep, bp, lev = oracle.segmented_shrink(a, 8, 2.0, 4, 4, L0)
        assert bp == NOT_TRIGGERED and keep.all() and lev == L0
    keep, bp, lev = oracle.segmented_shrink(a, 8, 2.0, 4, 4, 63)
    assert bp >= 0 and not keep.all()
    # A negative threshold counts as zero; an empty cache is never triggered.
    _, bp, lev = oracle.segmented_shrink(np.zeros(0, np.float32), 8, 2.0, 4, 4, -7)
    assert bp == NOT_TRIGGERED and lev == 0


def test_shrink_threshold_update_saturates():
    a = np.ones(10, np.float32)
    _, bp, lev = oracle.segmented_shrink(a, 4, 2.0, 0, 0, 5)
    assert bp == NO_BREAKPOINT and lev == 10
    g, _ = _geometric(64, RNG(8))
    _, bp, lev = oracle.segmented_shrink(g, 8, 2.0, 2 ** 31 - 1, 0, 0)
    assert bp == 8 and lev == 2 ** 31 - 1          # bp + recent saturates


def test_shrink_no_cut_points_and_full_windows():
    a, _ = _geometric(40, RNG(7))
    keep, bp, lev = oracle.segmented_shrink(a, 1, 2.0, 0, 0, 3)     # D = 1: no cuts
    assert bp == NO_BREAKPOINT and keep.all() and lev == 6
    keep, bp, lev = oracle.segmented_shrink(a, 4, 2.0, 100, 0, 0)    # recent covers all
    assert bp == 10 and keep.all() and lev == 110


def test_shrink_nan_cut_is_not_a_breakpoint():
    a = np.array([8.0] + [np.nan] * 7, np.float32)   # ranks 1.. are NaN
    keep, bp, _ = oracle.segmented_shrink(a, 4, 2.0, 0, 0, 0)
    assert bp == NO_BREAKPOINT and keep.all()
    a = np.array([8.0, 1.0, 1.0, 1.0, np.nan, np.nan, np.nan, np.nan], np.float32)
    keep, bp, _ = oracle.segmented_shrink(a, 4, 2.0, 0, 0, 0)
    assert bp == 2 and keep.tolist() == [True, True] + [False] * 6


def _independent_breakpoint(a, D, tau):
    """The ratio test holds on a suffix of the ranking (values never increase
    along it): ranks [cnt, n - nnan) where cnt counts the values whose
    tau-scaled size exceeds the head.  The breakpoint is the first cut there."""
    n = len(a)
    finite = a[~np.isnan(a)].astype(np.float64)
    if finite.size == 0:
        return NO_BREAKPOINT
    head = finite.max()
    if not head > 0:
        return NO_BREAKPOINT
    cnt = int(np.sum(float(tau) * finite > head))
    nnan = n - finite.size
    for d in range(1, D):
        c = (n * d) // D
        if cnt <= c < n - nnan:
            return c
    return NO_BREAKPOINT


def test_shrink_matches_threshold_route_and_library_ranking():
    rng = RNG(45)
    for kind in ("zipf", "ties", "special", "uniform"):
        for n in (1, 2, 5, 31, 64, 257, 1000):
            for D, tau in ((2, 2.0), (10, 400.0), (16, 8.0), (64, 1.25)):
                for recent, sink in ((0, 0), (8, 2), (n + 3, 1)):
                    a = synth.score_vector(rng, n, kind)
                    keep, bp, lev = oracle.segmented_shrink(a, D, tau, recent, sink, 0)
                    assert bp == _independent_breakpoint(a, D, tau), (kind, n, D, tau)
                    if bp < 0:
                        assert keep.all() and lev == 0
                        continue
                    want = np.zeros(n, bool)
                    want[:min(sink, n)] = True
                    want[max(n - recent, 0):] = True
                    want[_ranked(a)[:bp]] = True
                    np.testing.assert_array_equal(keep, want)
                    assert lev == bp + recent


def test_shrink_scale_invariant_by_powers_of_two():
    rng = RNG(46)
    a = synth.score_vector(rng, 500, "zipf")
    base = oracle.segmented_shrink(a, 10, 30.0, 16, 4, 0)
    for e in (-20, -3, 5, 40):
        got = oracle.segmented_shrink(a * np.float32(2.0 ** e), 10, 30.0, 16, 4, 0)
        np.testing.assert_array_equal(got[0], base[0])
        assert got[1:] == base[1:]


# --------------------------------------------------------------------------
# Baseline policies: PyramidKV's layer budgets
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,total,beta", [(32, 32 * 1000, 20.0), (28, 5000, 10.0), (2, 100, 4.0), (1, 77, 20.0)])
def test_pyramid_budgets_progression(L, total, beta):
    k = oracle.pyramid_budgets(L, total, beta)
    assert len(k) == L
    assert abs(sum(k) - total) <= 1e-9 * total          # the budgets add up to the total
    if L > 1:
        assert abs(k[-1] - total / (beta * L)) <= 1e-9 * total
        steps = np.diff(k)
        assert np.all(steps < 0) and np.allclose(steps, steps[0])   # linear, falling with depth
        assert abs(k[0] / k[-1] - (2 * beta - 1)) <= 1e-9 * beta    # first : last = 2 beta - 1
