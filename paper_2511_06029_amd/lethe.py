"""Thin Python binding of liblethe.so (include/lethe.h): argument marshalling
only.  Every step of the decode/prune path runs in the library's HIP kernels;
torch provides device memory and the current HIP stream.

There is no fallback: if the library is missing, importing this module's
functions raises.
"""
import ctypes
import math
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblethe.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4
BF16, F32 = 0, 1
DEV_APPEND_OVERFLOW, DEV_INFEASIBLE, DEV_BAD_LAYOUT, DEV_HEAD_MISMATCH, DEV_WAIT_TIMEOUT = 1, 2, 4, 8, 16
OP_DECODE, OP_SPARSITY, OP_SELECT, OP_COMPACT, OP_DECODE_FINAL, OP_COMPACT_PLAN = 0, 1, 2, 3, 4, 5

SHRINK_NO_BREAKPOINT, SHRINK_NOT_TRIGGERED = -1, -2

EXPORTED = ("lethe_workspace_bytes", "lethe_state_bytes", "lethe_decode_attn_score", "lethe_decode_attn_score_final",
            "lethe_decode_attn_score_noalloc", "lethe_kv_compact_plan", "lethe_decode_attn_score_compact",
            "lethe_layer_sparsity", "lethe_rasr_select", "lethe_rasr_select_shared",
            "lethe_segmented_shrink", "lethe_kv_compact", "lethe_kv_compact_layers", "lethe_score_flush",
            "lethe_prefill_attn_score", "lethe_prefill_workspace_bytes", "lethe_status_string")


class CCache(ctypes.Structure):
    """Mirror of ``lethe_cache``."""
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("score", ctypes.c_void_p),
        ("len", ctypes.c_void_p), ("seq_base", ctypes.c_void_p), ("cap", ctypes.c_void_p),
        ("rows_per_layer", ctypes.c_int64), ("num_layers", ctypes.c_int32),
        ("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("dev_status", ctypes.c_void_p), ("state", ctypes.c_void_p),
    ]


class LetheError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s: %s (%d)" % (fn, status_string(status), status))
        self.status = status


_lib = None


def load():
    """Load liblethe.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("liblethe.so is not built; run `python -m paper_2511_06029_amd.build` "
                              "(the HIP library is required: there is no CPU fallback)")
        lib = ctypes.CDLL(LIB_PATH)
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
        pc = ctypes.POINTER(CCache)
        lib.lethe_workspace_bytes.argtypes = [pc, ctypes.c_int]
        lib.lethe_workspace_bytes.restype = sz
        lib.lethe_state_bytes.argtypes = [pc]
        lib.lethe_state_bytes.restype = sz
        lib.lethe_score_flush.argtypes = [pc, vp]
        lib.lethe_score_flush.restype = ctypes.c_int
        lib.lethe_decode_attn_score.argtypes = [pc, i32, vp, vp, vp, ctypes.c_float, ctypes.c_float, vp, vp, sz, vp]
        lib.lethe_decode_attn_score.restype = ctypes.c_int
        lib.lethe_decode_attn_score_final.argtypes = lib.lethe_decode_attn_score.argtypes
        lib.lethe_decode_attn_score_final.restype = ctypes.c_int
        lib.lethe_decode_attn_score_noalloc.argtypes = [pc, i32, vp, vp, vp, ctypes.c_float, ctypes.c_float, vp, vp]
        lib.lethe_decode_attn_score_noalloc.restype = ctypes.c_int
        lib.lethe_layer_sparsity.argtypes = [pc, vp, i32, i32, vp, vp, vp, vp, sz, vp]
        lib.lethe_layer_sparsity.restype = ctypes.c_int
        lib.lethe_rasr_select.argtypes = [pc, vp, i32, i32, vp, vp, sz, vp]
        lib.lethe_rasr_select.restype = ctypes.c_int
        lib.lethe_rasr_select_shared.argtypes = [pc, vp, i32, i32, vp, vp, sz, vp]
        lib.lethe_rasr_select_shared.restype = ctypes.c_int
        lib.lethe_segmented_shrink.argtypes = [pc, i32, ctypes.c_float, i32, i32, vp, vp, vp, vp, sz, vp]
        lib.lethe_segmented_shrink.restype = ctypes.c_int
        lib.lethe_prefill_attn_score.argtypes = [pc, i32, vp, vp, vp, ctypes.c_int64, i32, i32, ctypes.c_float,
                                                 vp, vp, sz, vp]
        lib.lethe_prefill_attn_score.restype = ctypes.c_int
        lib.lethe_prefill_workspace_bytes.argtypes = [pc, ctypes.c_int64]
        lib.lethe_prefill_workspace_bytes.restype = sz
        lib.lethe_kv_compact.argtypes = [pc, vp, vp, sz, vp]
        lib.lethe_kv_compact.restype = ctypes.c_int
        lib.lethe_kv_compact_layers.argtypes = [pc, i32, i32, vp, vp, sz, vp]
        lib.lethe_kv_compact_layers.restype = ctypes.c_int
        lib.lethe_kv_compact_plan.argtypes = [pc, vp, vp, sz, vp]
        lib.lethe_kv_compact_plan.restype = ctypes.c_int
        lib.lethe_decode_attn_score_compact.argtypes = [pc, i32, vp, vp, vp, ctypes.c_float, ctypes.c_float, vp,
                                                        vp, sz, vp, sz, vp]
        lib.lethe_decode_attn_score_compact.restype = ctypes.c_int
        lib.lethe_status_string.argtypes = [ctypes.c_int]
        lib.lethe_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def status_string(status):
    return load().lethe_status_string(int(status)).decode()


DEV_STATUS_NAMES = ((DEV_APPEND_OVERFLOW, "append overflow"), (DEV_INFEASIBLE, "infeasible budget"),
                    (DEV_BAD_LAYOUT, "bad layout"), (DEV_HEAD_MISMATCH, "head mismatch"),
                    (DEV_WAIT_TIMEOUT, "wait timeout (results of that call unspecified)"))


def dev_status_names(bits):
    """The names of the device status bits set in `bits` (include/lethe.h)."""
    names = [name for bit, name in DEV_STATUS_NAMES if int(bits) & bit]
    rest = int(bits) & ~sum(bit for bit, _ in DEV_STATUS_NAMES)
    if rest:
        names.append("unknown bits %#x" % rest)
    return names


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _check(fn, st):
    if st != OK:
        raise LetheError(fn, st)


def workspace_bytes(cache, op):
    return int(load().lethe_workspace_bytes(ctypes.byref(cache.c_struct()), int(op)))


def state_bytes(cache):
    return int(load().lethe_state_bytes(ctypes.byref(cache.c_struct())))


def score_flush(cache, stream=None):
    """lethe_score_flush: apply the pending decode step of every (layer, sequence)."""
    _check("lethe_score_flush", load().lethe_score_flush(ctypes.byref(cache.c_struct()), _stream(stream)))


def decode_attn_score(cache, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, stream=None):
    """lethe_decode_attn_score: append (k_new/v_new may be None), attend; the
    score update of this step stays pending until the next call on the layer,
    score_flush or a prune call."""
    st = load().lethe_decode_attn_score(ctypes.byref(cache.c_struct()), int(layer), _p(q), _p(k_new),
                                        _p(v_new), float(gamma), float(softmax_scale), _p(out), _p(ws),
                                        ws.numel() * ws.element_size(), _stream(stream))
    _check("lethe_decode_attn_score", st)


def decode_attn_score_final(cache, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, stream=None):
    """lethe_decode_attn_score_final: the same step with its own score update
    applied within the call (nothing left pending); ws sized for
    OP_DECODE_FINAL."""
    st = load().lethe_decode_attn_score_final(ctypes.byref(cache.c_struct()), int(layer), _p(q), _p(k_new),
                                              _p(v_new), float(gamma), float(softmax_scale), _p(out), _p(ws),
                                              ws.numel() * ws.element_size(), _stream(stream))
    _check("lethe_decode_attn_score_final", st)


def decode_attn_score_noalloc(cache, layer, q, k_new, v_new, gamma, softmax_scale, out, stream=None):
    """lethe_decode_attn_score_noalloc: the decode step without a workspace
    (the chunk partials use the library's static device scratch)."""
    st = load().lethe_decode_attn_score_noalloc(ctypes.byref(cache.c_struct()), int(layer), _p(q), _p(k_new),
                                                _p(v_new), float(gamma), float(softmax_scale), _p(out),
                                                _stream(stream))
    _check("lethe_decode_attn_score_noalloc", st)


def layer_sparsity(cache, global_budget, recent, sink, sparsity_in, sparsity_out, budget_out,
                   ws=None, stream=None):
    """lethe_layer_sparsity: Hoyer sparsity per (sequence, layer) and budgets."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().lethe_layer_sparsity(ctypes.byref(cache.c_struct()), _p(global_budget), int(recent), int(sink),
                                     _p(sparsity_in), _p(sparsity_out), _p(budget_out), _p(ws), nbytes,
                                     _stream(stream))
    _check("lethe_layer_sparsity", st)


def rasr_select(cache, budget, recent, sink, keep, ws=None, stream=None):
    """lethe_rasr_select: keep mask of every segment."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().lethe_rasr_select(ctypes.byref(cache.c_struct()), _p(budget), int(recent), int(sink), _p(keep),
                                  _p(ws), nbytes, _stream(stream))
    _check("lethe_rasr_select", st)


def prefill_attn_score(cache, layer, q, q_start, q_len, max_q_len, max_kv_len, softmax_scale, out, ws,
                       stream=None):
    """lethe_prefill_attn_score: causal prefill attention over the q_len newest
    rows of every sequence, seeding their scores (Eq. 2).  q: bf16 [rows][H_Q][D];
    q_start int64 [B], q_len int32 [B] (device); out fp32 like q."""
    rows = q.shape[0]
    st = load().lethe_prefill_attn_score(ctypes.byref(cache.c_struct()), int(layer), _p(q), _p(q_start), _p(q_len),
                                         int(rows), int(max_q_len), int(max_kv_len), float(softmax_scale), _p(out),
                                         _p(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                         _stream(stream))
    _check("lethe_prefill_attn_score", st)


def rasr_select_shared(cache, budget, recent, sink, keep, ws=None, stream=None):
    """lethe_rasr_select_shared: one keep mask per (layer, sequence) from the
    head-summed score, written for every KV head."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().lethe_rasr_select_shared(ctypes.byref(cache.c_struct()), _p(budget), int(recent), int(sink),
                                         _p(keep), _p(ws), nbytes, _stream(stream))
    _check("lethe_rasr_select_shared", st)


def segmented_shrink(cache, segments, tau, recent, sink, evict_threshold, breakpoint, keep, ws=None,
                     stream=None):
    """lethe_segmented_shrink: Algorithm 1 with the size trigger; updates
    evict_threshold (int32 [L][B]) in place, fills breakpoint (or None)."""
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load().lethe_segmented_shrink(ctypes.byref(cache.c_struct()), int(segments), float(tau), int(recent),
                                       int(sink), _p(evict_threshold), _p(breakpoint), _p(keep), _p(ws), nbytes,
                                       _stream(stream))
    _check("lethe_segmented_shrink", st)


def kv_compact(cache, keep, ws, stream=None):
    """lethe_kv_compact: in-place order-preserving compaction; updates len."""
    st = load().lethe_kv_compact(ctypes.byref(cache.c_struct()), _p(keep), _p(ws),
                                 ws.numel() * ws.element_size(), _stream(stream))
    _check("lethe_kv_compact", st)


def kv_compact_layers(cache, layer_begin, layer_count, keep, ws, stream=None):
    """lethe_kv_compact_layers: the compaction of layers layer_begin ..
    layer_begin + layer_count - 1 only."""
    st = load().lethe_kv_compact_layers(ctypes.byref(cache.c_struct()), int(layer_begin), int(layer_count), _p(keep),
                                        _p(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check("lethe_kv_compact_layers", st)


def kv_compact_plan(cache, keep, plan, stream=None):
    """lethe_kv_compact_plan: record the compaction the next decode step of
    each layer carries out (nothing in the cache changes)."""
    st = load().lethe_kv_compact_plan(ctypes.byref(cache.c_struct()), _p(keep), _p(plan),
                                      plan.numel() * plan.element_size(), _stream(stream))
    _check("lethe_kv_compact_plan", st)


def decode_attn_score_compact(cache, layer, q, k_new, v_new, gamma, softmax_scale, out, plan, ws, stream=None):
    """lethe_decode_attn_score_compact: the layer's planned compaction, then
    its decode step, in one call."""
    st = load().lethe_decode_attn_score_compact(ctypes.byref(cache.c_struct()), int(layer), _p(q), _p(k_new),
                                                _p(v_new), float(gamma), float(softmax_scale), _p(out), _p(plan),
                                                plan.numel() * plan.element_size(), _p(ws),
                                                ws.numel() * ws.element_size(), _stream(stream))
    _check("lethe_decode_attn_score_compact", st)


class LetheCache:
    """A ragged KV cache in the layout of include/lethe.h, allocated with torch.

    ``caps[b]`` rows per (layer, sequence, KV head) segment; segment (l, b, h)
    starts at row ``l * rows_per_layer + seq_base[b] + h * caps[b]``."""

    def __init__(self, num_layers, caps, num_q_heads, num_kv_heads, head_dim, dtype="bf16", device="cuda"):
        import torch
        self.torch = torch
        self.L = int(num_layers)
        self.caps = [int(c) for c in caps]
        self.B = len(self.caps)
        self.HQ, self.HK, self.D = int(num_q_heads), int(num_kv_heads), int(head_dim)
        self.G = self.HQ // self.HK
        self.dtype_code = BF16 if dtype == "bf16" else F32
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        bases, acc = [], 0
        for c in self.caps:
            bases.append(acc)
            acc += self.HK * c
        self.seq_base_host = bases
        self.rows_per_layer = max(acc, 1)
        R = self.rows_per_layer
        self.k = torch.zeros((self.L, R, self.D), dtype=self.tdtype, device=device)
        self.v = torch.zeros((self.L, R, self.D), dtype=self.tdtype, device=device)
        self.score = torch.zeros((self.L, R), dtype=torch.float32, device=device)
        self.len = torch.zeros((self.L, self.B), dtype=torch.int32, device=device)
        self.seq_base = torch.tensor(bases, dtype=torch.int64, device=device)
        self.cap = torch.tensor(self.caps, dtype=torch.int32, device=device)
        self.dev_status = torch.zeros(1, dtype=torch.int32, device=device)
        self._c = None
        desc = self._struct(0)
        nstate = int(load().lethe_state_bytes(ctypes.byref(desc)))
        if nstate == 0:
            raise LetheError("lethe_state_bytes", ERR_UNSUPPORTED)
        self.state = torch.zeros(nstate, dtype=torch.uint8, device=device)

    def _struct(self, state_ptr):
        return CCache(self.k.data_ptr(), self.v.data_ptr(), self.score.data_ptr(), self.len.data_ptr(),
                      self.seq_base.data_ptr(), self.cap.data_ptr(), self.rows_per_layer, self.L, self.B,
                      self.HQ, self.HK, self.D, self.dtype_code, self.dev_status.data_ptr(), state_ptr)

    def c_struct(self):
        if self._c is None:
            self._c = self._struct(self.state.data_ptr())
        return self._c

    def flush(self, stream=None):
        """Make ``score`` current (apply the pending decode step)."""
        score_flush(self, stream)

    def reset_state(self):
        """Drop any pending decode step (after editing len / scores directly)."""
        self.state.zero_()

    def seg_rows(self, b, h):
        """Row range of segment (., b, h) within a layer."""
        start = self.seq_base_host[b] + h * self.caps[b]
        return start, start + self.caps[b]

    def workspace(self, op):
        n = workspace_bytes(self, op)
        return self.torch.zeros(max(n, 1), dtype=self.torch.uint8, device=self.k.device)

    def prefill_workspace(self, q_rows):
        n = int(load().lethe_prefill_workspace_bytes(ctypes.byref(self.c_struct()), int(q_rows)))
        return self.torch.zeros(max(n, 1), dtype=self.torch.uint8, device=self.k.device)

    def default_scale(self):
        return 1.0 / math.sqrt(self.D)
