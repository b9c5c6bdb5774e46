"""Pins of the oracle's prefill attention with score seeding (Eq. 2 summed over
the query heads of a KV group and the prompt's query positions) to facts other
than the oracle itself (CPU only): torch's fp64 attention with a causal mask
(a library routine) for the outputs, torch's softmax for the attention matrix
whose sums seed the scores, the harmonic closed form of a zero query, the
mass invariant, the reduction to the (separately pinned) decode step at one
query, and chunked prefill equal to one call.
"""
import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng


def _inputs(rng, n, qlen, D, G, bias=0.0):
    q = rng.standard_normal((qlen, G, D)).astype(np.float32)
    K = rng.standard_normal((n, D)).astype(np.float32)
    if bias:
        K += bias * rng.pareto(1.5, size=(n, 1)).astype(np.float32) * q[:, 0].mean(0)[None]
    V = rng.standard_normal((n, D)).astype(np.float32)
    return q, K, V


def _mask(n, qlen):
    """mask[i, j]: query i (position n - qlen + i) may attend row j."""
    pos = np.arange(n - qlen, n)[:, None]
    return np.arange(n)[None, :] <= pos


@pytest.mark.parametrize("n,qlen,D,G", [(1, 1, 64, 1), (9, 9, 64, 2), (40, 13, 64, 4), (130, 130, 128, 7),
                                         (257, 64, 128, 8)])
def test_prefill_matches_library_attention(n, qlen, D, G):
    rng = RNG(n + 7 * qlen)
    q, K, V = _inputs(rng, n, qlen, D, G, bias=0.5)
    scale = 1.0 / np.sqrt(D)
    s_in = rng.random(n)
    out, s = oracle.prefill(q, K, V, s_in, scale)
    mask = torch.from_numpy(_mask(n, qlen))
    qt = torch.from_numpy(q.astype(np.float64)).permute(1, 0, 2)       # (G, qlen, D)
    Kt = torch.from_numpy(K.astype(np.float64))[None].expand(G, n, D)
    Vt = torch.from_numpy(V.astype(np.float64))[None].expand(G, n, D)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, attn_mask=mask, scale=scale)
    np.testing.assert_allclose(out, ref.permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-12)
    logits = (qt @ Kt.transpose(1, 2)) * scale
    A = torch.softmax(logits.masked_fill(~mask, float("-inf")), dim=-1)   # (G, qlen, n)
    np.testing.assert_allclose(s, s_in + A.sum(dim=(0, 1)).numpy(), rtol=1e-10, atol=1e-12)


def test_prefill_mass_and_causality():
    rng = RNG(3)
    n, qlen, D, G = 300, 120, 64, 4
    q, K, V = _inputs(rng, n, qlen, D, G, bias=1.0)
    _, s = oracle.prefill(q, K, V, None, 0.125)
    assert abs(s.sum() - G * qlen) < 1e-9          # every query distributes one unit per head
    assert np.all(s >= 0)
    # The newest row is seen only by the newest query, whose own logit it holds.
    _, s1 = oracle.prefill(q[-1:], K, V, None, 0.125)
    assert abs(s[-1] - s1[-1]) < 1e-12


@pytest.mark.parametrize("n,qlen", [(1, 1), (10, 10), (50, 17), (200, 1)])
def test_prefill_zero_query_harmonic_closed_form(n, qlen):
    rng = RNG(5)
    G, D = 3, 64
    _, K, V = _inputs(rng, n, qlen, D, G)
    q = np.zeros((qlen, G, D), np.float32)
    out, s = oracle.prefill(q, K, V, None, 0.3)
    first = n - qlen
    for j in range(n):
        want = G * sum(1.0 / (p + 1) for p in range(max(j, first), n))
        assert abs(s[j] - want) < 1e-12
    for i in range(qlen):
        p = first + i
        np.testing.assert_allclose(out[i], np.broadcast_to(V[:p + 1].astype(np.float64).mean(0), (G, D)),
                                   rtol=1e-12, atol=1e-13)


def test_prefill_single_query_is_the_decode_step_without_decay():
    rng = RNG(6)
    n, D, G = 77, 128, 4
    q, K, V = _inputs(rng, n, 1, D, G)
    s_in = rng.random(n)
    out, s = oracle.prefill(q, K, V, s_in, 0.09)
    o_dec, s_dec = oracle.attend(q[0], K, V, s_in, 1.0, 0.09)
    np.testing.assert_allclose(out[0], o_dec, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(s, s_dec, rtol=1e-13, atol=1e-14)


def test_prefill_chunked_equals_whole():
    rng = RNG(8)
    n, D, G = 150, 64, 2
    q, K, V = _inputs(rng, n, n, D, G, bias=0.7)
    out, s = oracle.prefill(q, K, V, None, 0.2)
    cut = 61
    o1, s1 = oracle.prefill(q[:cut], K[:cut], V[:cut], None, 0.2)
    s1 = np.concatenate([s1, np.zeros(n - cut)])
    o2, s2 = oracle.prefill(q[cut:], K, V, s1, 0.2)
    np.testing.assert_allclose(np.concatenate([o1, o2]), out, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(s2, s, rtol=1e-13, atol=1e-14)


def test_prefill_empty_query_set():
    rng = RNG(9)
    q, K, V = _inputs(rng, 20, 0, 64, 4)
    s_in = rng.random(20)
    out, s = oracle.prefill(q, K, V, s_in, 0.1)
    assert out.shape == (0, 4, 64)
    np.testing.assert_array_equal(s, s_in)
