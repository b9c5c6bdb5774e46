"""oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow CPU reference for the Lethe hot path (arXiv 2511.06029): decode
attention with importance accumulation (Eq. 5), causal prefill attention that
seeds the importance (Eq. 2 over the prompt's queries), per-layer Hoyer sparsity
(Eq. 1 on the head-summed score of Eq. 2), the layer budget split, RASR
retention (per KV head, or shared by the heads of a layer), Algorithm 1's
segmented shrinking with its size trigger, and order-preserving compaction.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP path and
imports nothing from it.  Arithmetic is fp64 (see ``lethe_oracle.c``); inputs
are numpy arrays of the values the device holds (bf16 widened exactly).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        lib = ctypes.CDLL(path)
        i64, i32, dbl = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        vp = ctypes.c_void_p
        lib.lethe_oracle_attend.argtypes = [i64, ctypes.c_int, ctypes.c_int, vp, vp, vp, dbl, dbl, vp, vp, vp]
        lib.lethe_oracle_attend.restype = ctypes.c_int
        lib.lethe_oracle_hoyer.argtypes = [i64, vp]
        lib.lethe_oracle_hoyer.restype = dbl
        lib.lethe_oracle_layer_sparsity.argtypes = [i64, ctypes.c_int, vp]
        lib.lethe_oracle_layer_sparsity.restype = dbl
        lib.lethe_oracle_budget.argtypes = [ctypes.c_int, vp, vp, i32, i32, i64, vp]
        lib.lethe_oracle_budget.restype = ctypes.c_int
        lib.lethe_oracle_select.argtypes = [i64, vp, i64, i32, i32, vp]
        lib.lethe_oracle_select.restype = ctypes.c_int
        lib.lethe_oracle_head_sum_f32.argtypes = [i64, ctypes.c_int, vp, vp]
        lib.lethe_oracle_head_sum_f32.restype = None
        lib.lethe_oracle_shrink.argtypes = [i64, vp, i32, ctypes.c_float, i32, i32, vp, vp]
        lib.lethe_oracle_shrink.restype = i64
        lib.lethe_oracle_prefill.argtypes = [i64, i64, ctypes.c_int, ctypes.c_int, vp, vp, vp, dbl, vp, vp, vp]
        lib.lethe_oracle_prefill.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def attend(q, K, V, s_in, gamma, scale):
    """Softmax decode attention of G query heads over one KV segment, plus the
    Eq. 5 importance update summed over the G heads.

    q: (G, D); K, V: (n, D); s_in: (n,) or None.  Returns (out (G, D) float64,
    s_out (n,) float64)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    K = np.ascontiguousarray(K, dtype=np.float32)
    V = np.ascontiguousarray(V, dtype=np.float32)
    G, D = q.shape
    n = K.shape[0]
    assert K.shape == (n, D) and V.shape == (n, D)
    out = np.zeros((G, D), dtype=np.float64)
    s_out = np.zeros(n, dtype=np.float64)
    sp = None
    if s_in is not None:
        s_in = np.ascontiguousarray(s_in, dtype=np.float64)
        assert s_in.shape == (n,)
        sp = _ptr(s_in)
    rc = _load().lethe_oracle_attend(n, D, G, _ptr(q), _ptr(K), _ptr(V), float(scale), float(gamma),
                                     sp, _ptr(s_out), _ptr(out))
    if rc != 0:
        raise MemoryError("oracle attend failed")
    return out, s_out


def prefill(q, K, V, s_in, scale):
    """Causal prefill attention of the qlen newest rows of one KV segment for
    the G query heads of its group, plus Eq. 2's importance (attention summed
    over the heads and the queries) added to s_in.

    q: (qlen, G, D); K, V: (n, D); s_in: (n,) or None.  Returns (out (qlen, G,
    D) float64, s_out (n,) float64)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    K = np.ascontiguousarray(K, dtype=np.float32)
    V = np.ascontiguousarray(V, dtype=np.float32)
    qlen, G, D = q.shape
    n = K.shape[0]
    assert K.shape == (n, D) and V.shape == (n, D)
    out = np.zeros((max(qlen, 1), G, D), dtype=np.float64)
    s_out = np.zeros(max(n, 1), dtype=np.float64)
    sp = None
    if s_in is not None:
        s_in = np.ascontiguousarray(s_in, dtype=np.float64)
        assert s_in.shape == (n,)
        sp = _ptr(s_in)
    rc = _load().lethe_oracle_prefill(n, qlen, D, G, _ptr(q), _ptr(K), _ptr(V), float(scale), sp,
                                      _ptr(s_out), _ptr(out))
    if rc != 0:
        raise ValueError("oracle prefill failed (%d)" % rc)
    return out[:qlen], s_out[:n]


def hoyer(a):
    """Hoyer sparsity of a non-negative vector (Eq. 1); 0 when n <= 1 or a == 0."""
    a = np.ascontiguousarray(a, dtype=np.float64)
    return float(_load().lethe_oracle_hoyer(a.shape[0], _ptr(a)))


def layer_sparsity(s_heads):
    """Hoyer sparsity of the head-summed score (Eq. 2 then Eq. 1).
    s_heads: (H, n) scores of the H KV heads of one (layer, sequence)."""
    s = np.ascontiguousarray(s_heads, dtype=np.float64)
    H, n = s.shape
    return float(_load().lethe_oracle_layer_sparsity(n, H, _ptr(s)))


def budget_split(n, S, recent, sink, global_budget):
    """Per-layer budgets of one sequence from its layer sparsities.
    Returns (budget int32 (L,), infeasible bool)."""
    n = np.ascontiguousarray(n, dtype=np.int32)
    S = np.ascontiguousarray(S, dtype=np.float32)
    L = n.shape[0]
    out = np.zeros(L, dtype=np.int32)
    rc = _load().lethe_oracle_budget(L, _ptr(n), _ptr(S), int(recent), int(sink), int(global_budget), _ptr(out))
    if rc < 0:
        raise ValueError("oracle budget: too many layers")
    return out, bool(rc == 1)


def rasr_select(s, k, recent, sink):
    """RASR keep mask of one segment: sinks, recent window and the top of the
    remaining candidates by (score desc, index asc).  Returns bool (n,)."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    n = s.shape[0]
    keep = np.zeros(max(n, 1), dtype=np.uint8)
    rc = _load().lethe_oracle_select(n, _ptr(s), int(k), int(recent), int(sink), _ptr(keep))
    if rc != 0:
        raise MemoryError("oracle select failed")
    return keep[:n].astype(bool)


def head_sum_f32(s_heads):
    """Selection score of a kept set shared by every KV head of one (layer,
    sequence): the fp32 sum of the H head scores, h ascending, rounded after
    each addition (Eq. 2's sum over heads).  s_heads: (H, n).  Returns fp32 (n,)."""
    s = np.ascontiguousarray(s_heads, dtype=np.float32)
    H, n = s.shape
    a = np.zeros(max(n, 1), dtype=np.float32)
    _load().lethe_oracle_head_sum_f32(n, H, _ptr(s), _ptr(a))
    return a[:n]


def rasr_select_shared(s_heads, k, recent, sink):
    """RASR keep mask shared by all KV heads of one (layer, sequence): the rule
    of rasr_select applied to the head-summed score.  s_heads: (H, n)."""
    return rasr_select(head_sum_f32(s_heads), k, recent, sink)


SHRINK_NOT_TRIGGERED = -2
SHRINK_NO_BREAKPOINT = -1


def segmented_shrink(a, segments, tau, recent, sink, evict_threshold):
    """Algorithm 1 (segmented token shrinking) with the size trigger on one
    score vector a (fp32, n).  Returns (keep bool (n,), breakpoint, new
    evict threshold); breakpoint is SHRINK_NOT_TRIGGERED when n does not
    exceed the threshold and SHRINK_NO_BREAKPOINT when no cut qualifies."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    n = a.shape[0]
    keep = np.zeros(max(n, 1), dtype=np.uint8)
    lev = ctypes.c_int32(int(evict_threshold))
    bp = _load().lethe_oracle_shrink(n, _ptr(a), int(segments), float(tau), int(recent), int(sink),
                                     ctypes.byref(lev), _ptr(keep))
    if bp == -3:
        raise MemoryError("oracle shrink failed")
    return keep[:n].astype(bool), int(bp), int(lev.value)


def pyramid_budgets(L, total, beta):
    """PyramidKV's per-layer budgets (a baseline the paper compares against):
    an arithmetic progression falling with depth, whose last layer holds
    total / (beta * L) and whose first holds 2 total / L minus that, so the L
    budgets sum to total.  Real-valued (fp64), one per layer."""
    last = total / (beta * L)
    first = 2.0 * total / L - last
    if L == 1:
        return [float(total)]
    return [first - l * (first - last) / (L - 1) for l in range(L)]


def compact(rows, keep):
    """Order-preserving compaction: the kept rows, in their original order."""
    keep = np.asarray(keep, dtype=bool)
    return rows[keep]


class OracleCache:
    """Logical KV cache of one model: for every (layer, sequence, KV head) a
    segment of rows K (n, D), V (n, D) as float32 values and a float64 score
    vector s (n,).  Drives the per-segment functions above in plain loops."""

    def __init__(self, L, B, H_Q, H_KV, D):
        assert H_Q % H_KV == 0
        self.L, self.B, self.H_Q, self.H_KV, self.D = L, B, H_Q, H_KV, D
        self.G = H_Q // H_KV
        self.K = [[[np.zeros((0, D), np.float32) for _ in range(H_KV)] for _ in range(B)] for _ in range(L)]
        self.V = [[[np.zeros((0, D), np.float32) for _ in range(H_KV)] for _ in range(B)] for _ in range(L)]
        self.s = [[[np.zeros(0, np.float64) for _ in range(H_KV)] for _ in range(B)] for _ in range(L)]

    def set_segment(self, l, b, h, K, V, s=None):
        K = np.asarray(K, np.float32)
        self.K[l][b][h] = K.copy()
        self.V[l][b][h] = np.asarray(V, np.float32).copy()
        self.s[l][b][h] = np.zeros(K.shape[0]) if s is None else np.asarray(s, np.float64).copy()

    def length(self, l, b):
        return self.K[l][b][0].shape[0]

    def decode_step(self, l, q, k_new, v_new, gamma, scale, seqs=None):
        """Append (if k_new is given), then attend and update scores.
        q: (B, H_Q, D); k_new, v_new: (B, H_KV, D) or None.
        Returns out (B, H_Q, D) float64 (rows of unvisited sequences are 0)."""
        out = np.zeros((self.B, self.H_Q, self.D))
        for b in (range(self.B) if seqs is None else seqs):
            for h in range(self.H_KV):
                if k_new is not None:
                    self.K[l][b][h] = np.concatenate([self.K[l][b][h], np.asarray(k_new[b, h], np.float32)[None]])
                    self.V[l][b][h] = np.concatenate([self.V[l][b][h], np.asarray(v_new[b, h], np.float32)[None]])
                    self.s[l][b][h] = np.concatenate([self.s[l][b][h], [0.0]])
                G = self.G
                o, s_new = attend(q[b, h * G:(h + 1) * G], self.K[l][b][h], self.V[l][b][h],
                                  self.s[l][b][h], gamma, scale)
                out[b, h * G:(h + 1) * G] = o
                self.s[l][b][h] = s_new
        return out

    def sparsity(self, l, b):
        return layer_sparsity(np.stack([self.s[l][b][h] for h in range(self.H_KV)]))

    def prune_round(self, global_budget, recent, sink, sparsity_in=None):
        """Sparsity (unless given) -> budgets -> RASR select -> compaction, all
        layers and sequences.  Scores are ranked as the fp32 values a device
        stores.  Returns (S (B, L) float64, budget (B, L) int32, infeasible (B,))."""
        L, B = self.L, self.B
        S = np.zeros((B, L))
        budget = np.zeros((B, L), np.int32)
        infeasible = np.zeros(B, bool)
        for b in range(B):
            for l in range(L):
                S[b, l] = self.sparsity(l, b) if sparsity_in is None else sparsity_in[b][l]
            n = np.array([self.length(l, b) for l in range(L)], np.int32)
            budget[b], infeasible[b] = budget_split(n, S[b].astype(np.float32), recent, sink, global_budget[b])
        for l in range(L):
            for b in range(B):
                for h in range(self.H_KV):
                    keep = rasr_select(self.s[l][b][h].astype(np.float32), budget[b, l], recent, sink)
                    self.K[l][b][h] = compact(self.K[l][b][h], keep)
                    self.V[l][b][h] = compact(self.V[l][b][h], keep)
                    self.s[l][b][h] = compact(self.s[l][b][h], keep)
        return S, budget, infeasible
