"""C-ABI checks that need no GPU: the library loads, exports every entry point
include/lethe.h declares, and rejects invalid arguments on the host before
any HIP call (no call here reaches a kernel launch)."""
import ctypes
import math
import os
import re

import pytest

from paper_2511_06029_amd import lethe as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # never dereferenced: every call below fails validation first


def header_functions():
    text = open(os.path.join(ROOT, "include", "lethe.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lethe_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_entry_point():
    lib = L.load()
    declared = header_functions()
    assert set(declared) == set(L.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def make(**kw):
    c = L.CCache(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4096, 2, 4, 32, 8, 128, L.BF16, FAKE, FAKE)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def decode(c, layer=0, q=FAKE, kn=FAKE, vn=FAKE, gamma=0.9, scale=0.0, out=FAKE, ws=FAKE, wsb=None, final=False):
    lib = L.load()
    if wsb is None:
        wsb = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE_FINAL if final else L.OP_DECODE)
    fn = lib.lethe_decode_attn_score_final if final else lib.lethe_decode_attn_score
    return fn(ctypes.byref(c), layer, q, kn, vn, gamma, scale, out, ws, wsb, None)


def test_status_strings():
    for s in (L.OK, L.ERR_INVALID, L.ERR_UNSUPPORTED, L.ERR_WORKSPACE, L.ERR_HIP):
        assert L.status_string(s)
    assert L.status_string(L.ERR_WORKSPACE) == "workspace too small"


def test_workspace_sizes():
    lib = L.load()
    c = make()
    w = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE)
    # chunk partials: up to 64 chunks per segment, G heads * (m, l, o[D]) floats
    G, D, B, HK = 4, 128, 4, 8
    assert w >= B * HK * 64 * G * (D + 2) * 4
    assert w % 256 == 0
    # device pointers are not looked at
    assert lib.lethe_workspace_bytes(ctypes.byref(make(k=None, state=None)), L.OP_DECODE) == w
    # settling call: the partials, B row counts and 8 floats per row of a layer
    wf = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE_FINAL)
    assert wf >= w + B * 4 + 4096 * 8 * 4 and wf % 256 == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(make(rows_per_layer=8192)), L.OP_DECODE_FINAL) == wf + 4096 * 8 * 4
    assert lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_COMPACT) >= 2 * B * HK * 4
    assert lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_SELECT) == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(c), 99) == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(make(head_dim=96)), L.OP_DECODE) == 0
    assert lib.lethe_workspace_bytes(None, L.OP_DECODE) == 0


@pytest.mark.parametrize("field,value,want", [
    ("k", None, L.ERR_INVALID), ("v", None, L.ERR_INVALID), ("score", None, L.ERR_INVALID),
    ("len", None, L.ERR_INVALID), ("seq_base", None, L.ERR_INVALID), ("cap", None, L.ERR_INVALID),
    ("dev_status", None, L.ERR_INVALID), ("state", None, L.ERR_INVALID),
    ("num_layers", 0, L.ERR_INVALID), ("num_seqs", 0, L.ERR_INVALID),
    ("num_q_heads", 30, L.ERR_INVALID), ("num_kv_heads", 0, L.ERR_INVALID),
    ("rows_per_layer", 0, L.ERR_INVALID), ("dtype", 7, L.ERR_INVALID),
    ("head_dim", 96, L.ERR_UNSUPPORTED), ("head_dim", 256, L.ERR_UNSUPPORTED),
    ("num_q_heads", 72, L.ERR_UNSUPPORTED), ("num_seqs", 1025, L.ERR_UNSUPPORTED),
    ("num_layers", 257, L.ERR_UNSUPPORTED),
])
def test_cache_validation(field, value, want):
    c = make(**{field: value})
    assert decode(c, wsb=1 << 40) == want
    assert decode(c, wsb=1 << 40, final=True) == want
    lib = L.load()
    assert lib.lethe_rasr_select(ctypes.byref(c), FAKE, 8, 0, FAKE, None, 0, None) == want
    assert lib.lethe_rasr_select_shared(ctypes.byref(c), FAKE, 8, 0, FAKE, None, 0, None) == want
    assert lib.lethe_segmented_shrink(ctypes.byref(c), 10, 400.0, 8, 0, FAKE, None, FAKE, None, 0, None) == want
    assert lib.lethe_kv_compact(ctypes.byref(c), FAKE, FAKE, 1 << 40, None) == want
    assert lib.lethe_layer_sparsity(ctypes.byref(c), FAKE, 8, 0, None, FAKE, FAKE, None, 0, None) == want


@pytest.mark.parametrize("final", [False, True])
def test_decode_argument_validation(final):
    c = make()
    assert decode(c, layer=-1, final=final) == L.ERR_INVALID
    assert decode(c, layer=2, final=final) == L.ERR_INVALID
    assert decode(c, q=None, final=final) == L.ERR_INVALID
    assert decode(c, out=None, final=final) == L.ERR_INVALID
    assert decode(c, ws=None, final=final) == L.ERR_INVALID
    assert decode(c, kn=None, final=final) == L.ERR_INVALID          # v_new without k_new
    assert decode(c, vn=None, final=final) == L.ERR_INVALID
    for g in (0.0, -0.5, 1.0001, math.nan, math.inf):
        assert decode(c, gamma=g, final=final) == L.ERR_INVALID
    for s in (math.nan, math.inf, -math.inf):
        assert decode(c, scale=s, final=final) == L.ERR_INVALID
    lib = L.load()
    need = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE_FINAL if final else L.OP_DECODE)
    assert decode(c, wsb=need - 1, final=final) == L.ERR_WORKSPACE
    assert decode(c, wsb=0, final=final) == L.ERR_WORKSPACE
    if final:
        # the deferred call's workspace is too small for the settling one
        assert decode(c, wsb=lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE), final=True) == L.ERR_WORKSPACE


def test_prune_argument_validation():
    c = make()
    lib = L.load()
    cc = ctypes.byref(c)
    assert lib.lethe_layer_sparsity(cc, None, 8, 0, None, FAKE, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_layer_sparsity(cc, FAKE, 8, 0, None, None, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_layer_sparsity(cc, FAKE, 8, 0, None, FAKE, None, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_layer_sparsity(cc, FAKE, -1, 0, None, FAKE, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_layer_sparsity(cc, FAKE, 8, -2, None, FAKE, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select(cc, None, 8, 0, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select(cc, FAKE, 8, 0, None, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select(cc, FAKE, -8, 0, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select(cc, FAKE, 8, -1, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select_shared(cc, None, 8, 0, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select_shared(cc, FAKE, 8, 0, None, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select_shared(cc, FAKE, -1, 0, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_rasr_select_shared(cc, FAKE, 8, -1, FAKE, None, 0, None) == L.ERR_INVALID
    shrink = lib.lethe_segmented_shrink
    assert shrink(cc, 10, 400.0, 8, 0, None, None, FAKE, None, 0, None) == L.ERR_INVALID   # thresholds
    assert shrink(cc, 10, 400.0, 8, 0, FAKE, None, None, None, 0, None) == L.ERR_INVALID   # keep
    for seg in (0, -3):
        assert shrink(cc, seg, 400.0, 8, 0, FAKE, None, FAKE, None, 0, None) == L.ERR_INVALID
    for tau in (1.0, 0.5, -2.0, math.nan, math.inf):
        assert shrink(cc, 10, tau, 8, 0, FAKE, None, FAKE, None, 0, None) == L.ERR_INVALID
    assert shrink(cc, 10, 400.0, -1, 0, FAKE, None, FAKE, None, 0, None) == L.ERR_INVALID
    assert shrink(cc, 10, 400.0, 8, -1, FAKE, None, FAKE, None, 0, None) == L.ERR_INVALID
    assert lib.lethe_kv_compact(cc, None, FAKE, 1 << 20, None) == L.ERR_INVALID
    assert lib.lethe_kv_compact(cc, FAKE, None, 1 << 20, None) == L.ERR_INVALID
    need = lib.lethe_workspace_bytes(cc, L.OP_COMPACT)
    assert lib.lethe_kv_compact(cc, FAKE, FAKE, need - 1, None) == L.ERR_WORKSPACE


def test_prefill_validation_and_workspace():
    lib = L.load()
    c = make()
    cc = ctypes.byref(c)
    rows = 100
    need = lib.lethe_prefill_workspace_bytes(cc, rows)
    assert need >= rows * 32 * 2 * 4 and need % 256 == 0
    assert lib.lethe_prefill_workspace_bytes(cc, 0) == 0
    assert lib.lethe_prefill_workspace_bytes(cc, -1) == 0
    assert lib.lethe_prefill_workspace_bytes(None, 5) == 0
    pf = lib.lethe_prefill_attn_score

    def call(layer=0, q=FAKE, qs=FAKE, ql=FAKE, rows=rows, mq=64, mkv=64, scale=0.0, out=FAKE, ws=FAKE, wsb=need,
             cache=cc):
        return pf(cache, layer, q, qs, ql, rows, mq, mkv, scale, out, ws, wsb, None)

    assert call(layer=-1) == L.ERR_INVALID
    assert call(layer=2) == L.ERR_INVALID
    assert call(qs=None) == L.ERR_INVALID
    assert call(ql=None) == L.ERR_INVALID
    assert call(q=None) == L.ERR_INVALID
    assert call(out=None) == L.ERR_INVALID
    assert call(rows=-1) == L.ERR_INVALID
    assert call(mq=-1) == L.ERR_INVALID
    assert call(mkv=-1) == L.ERR_INVALID
    for sc in (math.nan, math.inf):
        assert call(scale=sc) == L.ERR_INVALID
    assert call(ws=None) == L.ERR_WORKSPACE
    assert call(wsb=need - 1) == L.ERR_WORKSPACE
    assert call(cache=ctypes.byref(make(dtype=L.F32))) == L.ERR_UNSUPPORTED
    assert call(cache=ctypes.byref(make(head_dim=96))) == L.ERR_UNSUPPORTED
    assert call(cache=ctypes.byref(make(state=None))) == L.ERR_INVALID


def test_state_sizes():
    lib = L.load()
    G, B, HQ, HK, D, Ly = 4, 4, 32, 8, 128, 2
    n = lib.lethe_state_bytes(ctypes.byref(make()))
    # double-buffered bf16 queries of the pending step, plus (M, 1/L) per
    # segment and head, plus small per-sequence arrays
    core = Ly * 2 * B * HQ * D * 2 + Ly * B * HK * 2 * G * 4
    assert core <= n < core + (1 << 14)
    assert n % 256 == 0
    assert lib.lethe_state_bytes(ctypes.byref(make(state=None, k=None))) == n
    assert lib.lethe_state_bytes(ctypes.byref(make(rows_per_layer=1 << 20))) == n
    assert lib.lethe_state_bytes(ctypes.byref(make(dtype=L.F32))) > n
    assert lib.lethe_state_bytes(ctypes.byref(make(head_dim=96))) == 0
    assert lib.lethe_state_bytes(None) == 0


def test_flush_validation():
    lib = L.load()
    assert lib.lethe_score_flush(None, None) == L.ERR_INVALID
    assert lib.lethe_score_flush(ctypes.byref(make(state=None)), None) == L.ERR_INVALID
    assert lib.lethe_score_flush(ctypes.byref(make(len=None)), None) == L.ERR_INVALID
    assert lib.lethe_score_flush(ctypes.byref(make(head_dim=96)), None) == L.ERR_UNSUPPORTED


def test_struct_layout_matches_header():
    # Offsets of the C struct on x86-64 / gfx950 (LP64): six pointers, one
    # int64, six 32-bit fields, two pointers.
    assert L.CCache.rows_per_layer.offset == 48
    assert L.CCache.num_layers.offset == 56
    assert L.CCache.dtype.offset == 76
    assert L.CCache.dev_status.offset == 80
    assert L.CCache.state.offset == 88
    assert ctypes.sizeof(L.CCache) == 96


def test_device_status_bits_match_the_header():
    """The binding's device status bits and their names against the
    LETHE_DEV_* values include/lethe.h defines."""
    import re
    from paper_2511_06029_amd import lethe as Lb
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    text = open(os.path.join(root, "include", "lethe.h")).read()
    defs = {m.group(1): int(m.group(2)) for m in re.finditer(r"#define LETHE_DEV_(\w+)\s+(\d+)", text)}
    assert defs == {"APPEND_OVERFLOW": Lb.DEV_APPEND_OVERFLOW, "INFEASIBLE": Lb.DEV_INFEASIBLE,
                    "BAD_LAYOUT": Lb.DEV_BAD_LAYOUT, "HEAD_MISMATCH": Lb.DEV_HEAD_MISMATCH,
                    "WAIT_TIMEOUT": Lb.DEV_WAIT_TIMEOUT}
    assert sorted(bit for bit, _ in Lb.DEV_STATUS_NAMES) == sorted(defs.values())
    assert Lb.dev_status_names(0) == []
    assert Lb.dev_status_names(Lb.DEV_WAIT_TIMEOUT | Lb.DEV_BAD_LAYOUT)[0] == "bad layout"
    assert Lb.dev_status_names(1 << 12) == ["unknown bits 0x1000"]
