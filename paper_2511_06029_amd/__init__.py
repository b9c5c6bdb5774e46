"""MI355X (gfx950) implementation of Lethe's decode/prune hot path.

The C ABI is declared in ``include/lethe.h`` and implemented by
``liblethe.so`` (HIP kernels in ``csrc/``); ``lethe`` is its ctypes binding.
"""
from .lethe import (  # noqa: F401
    LetheCache, LetheError, decode_attn_score, kv_compact, layer_sparsity, load, rasr_select,
    status_string, workspace_bytes,
)
