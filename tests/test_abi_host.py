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
    c = L.CCache(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4096, 2, 4, 32, 8, 128, L.BF16, FAKE)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def decode(c, layer=0, q=FAKE, kn=FAKE, vn=FAKE, gamma=0.9, scale=0.0, out=FAKE, ws=FAKE, wsb=None):
    lib = L.load()
    if wsb is None:
        wsb = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE) if L.load() else 0
    return lib.lethe_decode_attn_score(ctypes.byref(c), layer, q, kn, vn, gamma, scale, out, ws, wsb, None)


def test_status_strings():
    for s in (L.OK, L.ERR_INVALID, L.ERR_UNSUPPORTED, L.ERR_WORKSPACE, L.ERR_HIP):
        assert L.status_string(s)
    assert L.status_string(L.ERR_WORKSPACE) == "workspace too small"


def test_workspace_sizes():
    lib = L.load()
    c = make()
    w = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE)
    # plan + partials for (4096 + B*H_KV) chunks * G heads * (D + 2) floats
    # + one fp32 logit per row and head
    G, D, B, HK, R = 4, 128, 4, 8, 4096
    assert w >= (4096 + B * HK) * G * (D + 2) * 4 + R * G * 4
    assert w % 256 == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_COMPACT) >= 2 * B * HK * 4
    assert lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_SELECT) == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(c), 99) == 0
    assert lib.lethe_workspace_bytes(ctypes.byref(make(head_dim=96)), L.OP_DECODE) == 0
    assert lib.lethe_workspace_bytes(None, L.OP_DECODE) == 0


@pytest.mark.parametrize("field,value,want", [
    ("k", None, L.ERR_INVALID), ("v", None, L.ERR_INVALID), ("score", None, L.ERR_INVALID),
    ("len", None, L.ERR_INVALID), ("seq_base", None, L.ERR_INVALID), ("cap", None, L.ERR_INVALID),
    ("dev_status", None, L.ERR_INVALID), ("num_layers", 0, L.ERR_INVALID), ("num_seqs", 0, L.ERR_INVALID),
    ("num_q_heads", 30, L.ERR_INVALID), ("num_kv_heads", 0, L.ERR_INVALID),
    ("rows_per_layer", 0, L.ERR_INVALID), ("dtype", 7, L.ERR_INVALID),
    ("head_dim", 96, L.ERR_UNSUPPORTED), ("head_dim", 256, L.ERR_UNSUPPORTED),
    ("num_q_heads", 72, L.ERR_UNSUPPORTED), ("num_seqs", 1025, L.ERR_UNSUPPORTED),
    ("num_layers", 257, L.ERR_UNSUPPORTED),
])
def test_cache_validation(field, value, want):
    c = make(**{field: value})
    assert decode(c, wsb=1 << 40) == want
    lib = L.load()
    assert lib.lethe_rasr_select(ctypes.byref(c), FAKE, 8, 0, FAKE, None, 0, None) == want
    assert lib.lethe_kv_compact(ctypes.byref(c), FAKE, FAKE, 1 << 40, None) == want
    assert lib.lethe_layer_sparsity(ctypes.byref(c), FAKE, 8, 0, None, FAKE, FAKE, None, 0, None) == want


def test_decode_argument_validation():
    c = make()
    assert decode(c, layer=-1) == L.ERR_INVALID
    assert decode(c, layer=2) == L.ERR_INVALID
    assert decode(c, q=None) == L.ERR_INVALID
    assert decode(c, out=None) == L.ERR_INVALID
    assert decode(c, ws=None) == L.ERR_INVALID
    assert decode(c, kn=None) == L.ERR_INVALID          # v_new without k_new
    assert decode(c, vn=None) == L.ERR_INVALID
    for g in (0.0, -0.5, 1.0001, math.nan, math.inf):
        assert decode(c, gamma=g) == L.ERR_INVALID
    for s in (math.nan, math.inf, -math.inf):
        assert decode(c, scale=s) == L.ERR_INVALID
    lib = L.load()
    need = lib.lethe_workspace_bytes(ctypes.byref(c), L.OP_DECODE)
    assert decode(c, wsb=need - 1) == L.ERR_WORKSPACE
    assert decode(c, wsb=0) == L.ERR_WORKSPACE


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
    assert lib.lethe_kv_compact(cc, None, FAKE, 1 << 20, None) == L.ERR_INVALID
    assert lib.lethe_kv_compact(cc, FAKE, None, 1 << 20, None) == L.ERR_INVALID
    need = lib.lethe_workspace_bytes(cc, L.OP_COMPACT)
    assert lib.lethe_kv_compact(cc, FAKE, FAKE, need - 1, None) == L.ERR_WORKSPACE


def test_struct_layout_matches_header():
    # Offsets of the C struct on x86-64 / gfx950 (LP64): six pointers, one
    # int64, six 32-bit fields, one pointer.
    assert L.CCache.rows_per_layer.offset == 48
    assert L.CCache.num_layers.offset == 56
    assert L.CCache.dtype.offset == 76
    assert L.CCache.dev_status.offset == 80
    assert ctypes.sizeof(L.CCache) == 88
