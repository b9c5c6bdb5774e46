"""The compaction's bounded wait between blocks, forced from the host to give up.

With LETHE_COMPACT_TEST_WAIT=1 every queue entry of lethe_kv_compact also waits
for a flag that nothing sets, and LETHE_COMPACT_SPIN_LIMIT bounds the polls, so
the call must end with LETHE_DEV_WAIT_TIMEOUT set instead of hanging; every
block still exits.  The library reads both variables once per process, so the
call runs in a child process.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent("""
    import sys
    import torch
    from paper_2511_06029_amd import lethe as L

    lengths = (700, 3000)
    c = L.LetheCache(2, list(lengths), 8, 2, 128, dtype="bf16", device="cuda")
    keep = torch.zeros((2, c.rows_per_layer), dtype=torch.uint8, device="cuda")
    for b, n in enumerate(lengths):
        c.len[:, b] = n
        for h in range(2):
            s0, _ = c.seg_rows(b, h)
            keep[:, s0:s0 + n:2] = 1  # every other row: every tile moves
    print("kv_compact with a flag nothing sets", flush=True)
    L.kv_compact(c, keep, c.workspace(L.OP_COMPACT))
    torch.cuda.synchronize()
    st = int(c.dev_status[0])
    print("dev_status", st, flush=True)
    sys.exit(0 if st & L.DEV_WAIT_TIMEOUT else 3)
""")


@pytest.mark.gpu
def test_compact_wait_gives_up_with_status_bit():
    env = dict(os.environ, LETHE_COMPACT_TEST_WAIT="1", LETHE_COMPACT_SPIN_LIMIT="64")
    print("child process: compaction with the never-set flag", flush=True)
    r = subprocess.run([sys.executable, "-c", CHILD], env=env, cwd=ROOT, timeout=120,
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
