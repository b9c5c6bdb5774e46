"""Host logic of bench.py (CPU): the prune-round accounting, the traffic figure
read from a committed counter summary, the host description and the
one-GPU guard."""
import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def synthetic_run(windows, rows_per_step, interval, start, kept, a_ms, b_ms, prune_ms):
    """Intervals whose decode step costs exactly a + b * (rows at the
    interval's middle); kept[w]: rows the round after interval w keeps."""
    start_rows = [start] + list(kept[:-1])
    mid = np.array(start_rows, np.float64) + rows_per_step * (interval + 2) / 2.0
    dec = a_ms + b_ms * mid
    return dec, np.array(prune_ms, np.float64), start_rows, kept[-1]


def test_prune_against_saved_exact_on_a_linear_cost():
    rows_per_step, interval = 10 * 4, 100
    # A full-length start cut to its budget, then rounds that each drop a
    # different number of rows.
    kept = [60000, 61000, 62500, 62000, 63800]
    dec, prune, start_rows, last = synthetic_run(5, rows_per_step, interval, 200000, kept, 0.02, 3e-7,
                                                 [0.5, 0.1, 0.2, 0.15, 0.3])
    r = bench.prune_against_saved(dec, prune, start_rows, last, rows_per_step, interval, [0.0] * 5)
    assert r is not None
    assert r["decode_ms_per_token_step"] == pytest.approx(3e-7, rel=1e-9)
    assert r["decode_step_fixed_ms"] == pytest.approx(0.02, rel=1e-9)
    want = []
    prev = 200000
    for w in range(5):
        evicted = prev + rows_per_step * interval - kept[w]
        want.append(prune[w] / (interval * 3e-7 * evicted))
        prev = kept[w]
    np.testing.assert_allclose(r["per_round"], want, rtol=1e-9)
    assert r["round1"] == pytest.approx(want[0], rel=1e-9)
    assert r["steady_median"] == pytest.approx(float(np.median(want[1:])), rel=1e-9)
    assert r["prune_round_ms"] == list(prune)


def test_prune_against_saved_round_without_eviction():
    """A round that evicts nothing saves nothing: no ratio for it, and the
    steady median skips it."""
    rows_per_step, interval = 8, 50
    kept = [3000, 3400, 3300, 3600]    # the second round keeps everything
    dec, prune, start_rows, last = synthetic_run(4, rows_per_step, interval, 10000, kept, 0.01, 1e-6,
                                                 [0.2, 0.05, 0.07, 0.06])
    r = bench.prune_against_saved(dec, prune, start_rows, last, rows_per_step, interval, [0.0] * 4)
    assert r["per_round"][1] is None
    assert all(x is not None for i, x in enumerate(r["per_round"]) if i != 1)
    assert r["steady_median"] == pytest.approx(float(np.median([r["per_round"][2], r["per_round"][3]])))


def test_prune_against_saved_needs_different_sizes():
    """A run that starts at the steady state has intervals of one size: no fit."""
    dec = np.full(6, 5.0)
    r = bench.prune_against_saved(dec, np.full(6, 9.0), [100000] * 6, 100000, 4096, 128, [0.0] * 6)
    assert r is None
    assert bench.prune_against_saved(dec[:1], np.full(1, 9.0), [100000], 50000, 4096, 128, [0.0]) is None


def write_summary(path, sha, measured, algorithmic):
    path.write_text("# summary\n\n- source_sha256: `%s`\n- hbm_bytes_per_launch: %d\n"
                    "- algorithmic_bytes_per_launch: %d\n" % (sha, measured, algorithmic))


def test_traffic_scaled_while_sources_match(tmp_path, monkeypatch):
    p = tmp_path / "t.md"
    write_summary(p, bench.kernel_source_hash(), 1030, 1000)
    monkeypatch.setattr(bench, "TRAFFIC_PROFILES", {5: str(p)})
    t = bench.load_traffic(5, 2.0e9)
    assert t["bytes"] == pytest.approx(2.06e9)
    assert "1.0300" in t["source"]
    # Another workload, a changed source, a missing file: no figure.
    assert bench.load_traffic(3, 2.0e9) is None
    write_summary(p, hashlib.sha256(b"other").hexdigest(), 1030, 1000)
    assert bench.load_traffic(5, 2.0e9) is None
    p.unlink()
    assert bench.load_traffic(5, 2.0e9) is None


def test_committed_traffic_summary_matches_the_kernel_sources():
    """The headline workload's counter summary was taken on the current
    decode kernel sources, and its HBM bytes are close to the algorithmic
    ones (K and V read once)."""
    t = bench.load_traffic(5, 1.0e9)
    assert t is not None, "profiles/decode_bf16_kernel_llama8b_b128_traffic.md is stale or unreadable"
    assert 1.0e9 <= t["bytes"] <= 1.1e9


def test_host_cpu_description():
    model, threads = bench.host_cpu()
    assert threads >= 1
    assert model is None or isinstance(model, str)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)
