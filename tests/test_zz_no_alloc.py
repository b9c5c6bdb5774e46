"""lethe_decode_attn_score_noalloc, the decode step for callers that cannot
allocate: its chunk partials live in the library's static device scratch
instead of a caller workspace.

On an MI355X it must give what lethe_decode_attn_score gives on a twin cache
(the same kernels): with the fixed step schedule bit for bit (out, len and
the scores after a flush), with the default schedule within the decode
tolerance (|x - y| <= 1e-3 + 2e-3 |y|).  Each case makes two calls in a row,
the second on a smaller cache, so the scratch still holds the first call's
partials when the second starts.  The size limit is checked on the host.
"""
import ctypes
import math
import sys

import numpy as np
import pytest
import torch

from paper_2511_06029_amd import lethe as L
from workloads import synth

from test_gpu_final_decode import assert_same, live_scores, twin
from test_gpu_parity import DEV, Harness, close, host

FAKE = 0x10000  # never dereferenced: the host check fails first


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def filled(dtype, D, G, HK, lengths, rng):
    """Harness (two layers) with random K, V and Zipf scores, lengths set."""
    H = Harness(2, [n + 4 for n in lengths], G * HK, HK, D, dtype)
    for l in range(2):
        for b, n in enumerate(lengths):
            for h in range(HK):
                K = (rng.standard_normal((n, D)) * (1 + 2 * rng.random((n, 1)))).astype(np.float32)
                H.fill(l, b, h, K, rng.standard_normal((n, D)).astype(np.float32), synth.score_vector(rng, n, "zipf"))
            H.set_len(l, b, n)
    return H


def compare(H, steps, rng, exact):
    """`steps` decode steps over both layers on the harness cache through the
    workspace entry point and on its twin through the scratch entry point."""
    A = H.c
    T = twin(A)
    B, HQ, D, HK = A.B, A.HQ, A.D, A.HK
    ws = A.workspace(L.OP_DECODE)
    scale = 1 / math.sqrt(D)
    for step in range(steps):
        for l in range(2):
            q = H.store(2 * rng.standard_normal((B, HQ, D)))
            kn = H.store(rng.standard_normal((B, HK, D)))
            vn = H.store(rng.standard_normal((B, HK, D)))
            out_a = torch.empty((B, HQ, D), dtype=torch.float32, device=DEV)
            out_t = torch.full_like(out_a, float("nan"))
            L.decode_attn_score(A, l, q, kn, vn, 0.95, scale, out_a, ws)
            L.decode_attn_score_noalloc(T, l, q, kn, vn, 0.95, scale, out_t)
            torch.cuda.synchronize()
            if exact:
                np.testing.assert_array_equal(host(out_t), host(out_a), err_msg="out step %d layer %d" % (step, l))
            else:
                close(host(out_t), host(out_a), "out step %d layer %d" % (step, l))
    A.flush()
    T.flush()
    torch.cuda.synchronize()
    assert A.len.cpu().tolist() == T.len.cpu().tolist()
    if exact:
        assert_same(live_scores(T), live_scores(A), "scores")
    else:
        for x, y in zip(live_scores(T), live_scores(A)):
            close(x, y, "scores")
    assert int(A.dev_status[0]) == 0 and int(T.dev_status[0]) == 0


CASES = [
    # (dtype, D, G, HK, lengths) of the first call, then of the second (smaller) one
    (("bf16", 128, 4, 8, [3000, 17, 2500, 1, 640, 0]), ("bf16", 128, 4, 2, [200, 33])),
    (("bf16", 128, 7, 4, [4100, 900, 5]), ("bf16", 64, 2, 3, [1, 65])),
    (("f32", 64, 2, 2, [512, 3, 1200]), ("f32", 64, 2, 1, [100])),
]


@pytest.mark.gpu
@pytest.mark.parametrize("exact", [True, False], ids=["fixed-schedule", "default-schedule"])
@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_workspace_call(first, second, exact, monkeypatch):
    if exact:
        monkeypatch.setenv("LETHE_DECODE_DETERMINISTIC", "1")
    rng = np.random.default_rng(sum(first[4]) + 7 * first[2] + exact)
    for shape in (first, second):
        note("noalloc decode %s D=%d G=%d HK=%d lengths=%s exact=%s" % (shape + (exact,)))
        H = filled(*shape, rng)
        compare(H, 2, rng, exact)
        del H
        torch.cuda.synchronize()


@pytest.mark.gpu
def test_noalloc_against_oracle():
    """Two calls in a row on the tiny fp32 case against the oracle directly."""
    note("noalloc decode, tiny case against the oracle")
    d = synth.tiny_case(seed=1)
    HQ, HK, D = 4, 2, 64
    H = Harness(1, [528], HQ, HK, D, "f32")
    for h in range(HK):
        H.fill(0, 0, h, d["K0"][0, h], d["V0"][0, h])
    H.set_len(0, 0, 512)
    scale = 1 / math.sqrt(D)
    for t in range(2):
        out = torch.empty((1, HQ, D), dtype=torch.float32, device=DEV)
        L.decode_attn_score_noalloc(H.c, 0, torch.from_numpy(d["q"][t]).to(DEV), torch.from_numpy(d["k_new"][t]).to(DEV),
                                    torch.from_numpy(d["v_new"][t]).to(DEV), 0.99, scale, out)
        ref = H.orc.decode_step(0, d["q"][t], d["k_new"][t], d["v_new"][t], 0.99, scale)
        torch.cuda.synchronize()
        close(host(out), ref, "out step %d" % t)
    H.check_scores(0)


def test_noalloc_size_limit_on_host():
    """One partial per (sequence, KV head) must fit the 32 MiB scratch: 1024
    sequences x 8 KV heads x G = 8 (4224-byte partials) do not, G = 4 does
    (it then fails later, on the fake pointers' null q)."""
    lib = L.load()
    fn = lib.lethe_decode_attn_score_noalloc
    big = L.CCache(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, 1, 1024, 64, 8, 128, L.BF16, FAKE, FAKE)
    assert fn(ctypes.byref(big), 0, FAKE, FAKE, FAKE, 0.9, 0.0, FAKE, None) == L.ERR_UNSUPPORTED
    ok = L.CCache(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, 1, 1024, 32, 8, 128, L.BF16, FAKE, FAKE)
    assert fn(ctypes.byref(ok), 0, None, FAKE, FAKE, 0.9, 0.0, FAKE, None) == L.ERR_INVALID
    # Argument checks come first, as in lethe_decode_attn_score.
    assert fn(ctypes.byref(ok), 0, FAKE, FAKE, None, 0.9, 0.0, FAKE, None) == L.ERR_INVALID
    assert fn(ctypes.byref(ok), 0, FAKE, FAKE, FAKE, 1.5, 0.0, FAKE, None) == L.ERR_INVALID
    assert fn(ctypes.byref(ok), 1, FAKE, FAKE, FAKE, 0.9, 0.0, FAKE, None) == L.ERR_INVALID
