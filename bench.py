#!/usr/bin/env python3
"""Benchmark of the Lethe hot path on one MI355X.

Default workload: the largest model-scale configuration, Llama-3-8B-shaped
decoding (32 layers, 32 query / 8 KV heads, head_dim 128, bf16 cache) of 128
sequences whose logical lengths are log-uniform in [1k, 64k]; a 10% global
budget split over the layers by fixed shares of 2% to 40% (through the
budget split's sparsity_in argument); a prune round every 128 decode steps
with a recent window of 64.  The full caches of this batch (about 260 GB) do
not fit one GPU with headroom, so the run starts from the steady state: every
layer holds its budget share of each sequence.

One benchmark step is one prune interval: 128 decode steps over all 32 layers
(append + fused attention and Eq. 5 score update: lethe_decode_attn_score),
then one prune round over all layers (lethe_layer_sparsity,
lethe_rasr_select, lethe_kv_compact).  Inputs are resident in HBM before the
timed region starts.  After the CPU baseline the default run frees that cache
and runs a short leg of the Qwen-7B-shaped batch-16 workload (28 layers, 28
query / 4 KV heads, 16k cached tokens, 30% budget, prune every 256, recent
256; --config3-rounds intervals) and reports under "config3" what each of its
prune rounds costs against the decode time it saves over the next interval.

--config 2|3|4 run one of the other model-scale workloads instead (Llama-3-8B
batch 8 with a 2k prompt and 40% budget every 512; the Qwen-7B batch-16
workload; Llama-3-8B batch 64 of U[8k, 32k] cached tokens, 25% every 256).
Every line reports what each prune round costs against the decode time it
saves over the next interval (prune_vs_saved) when the run's intervals differ
enough in size to fit the per-token decode cost.

Prune rounds (--policy):
  lethe         lethe_layer_sparsity, lethe_rasr_select (a kept set per KV
                head), lethe_kv_compact -- the default, the headline line;
  lethe-shared  the same with lethe_rasr_select_shared (one kept set per
                layer and sequence, ranked by the head-summed score);
  shrink        lethe_segmented_shrink (Algorithm 1 with the size trigger:
                --segments cut points, ratio --tau, first threshold the
                prompt length) and lethe_kv_compact;
  h2o, streaming, pyramid
                the baselines as parameterisations of the same calls
                (paper_2511_06029_amd/policies.py): cumulative scores and
                uniform layer budgets; sinks plus a window filling the
                budget; PyramidKV's static layer budgets.

With --prefill the line instead measures lethe_prefill_attn_score on the
Llama-3-8B shapes: one step is the causal prefill attention with score
seeding (Eq. 2) of a 2048-token prompt for 8 sequences, over all 32 layers;
the roofline is the matrix-core bf16 peak.

The JSON line reports KV tokens scanned per second (one token = one cached
(layer, sequence, position) row, all KV heads) over the whole timed run, the
per-step decode latency, the prune-round latency, the HBM roofline of the
decode call and the CPU oracle's throughput (decode step and prune round) on
a bounded sample.
"""
import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# rocprofv3 counter summaries of the decode kernel per workload (FETCH_SIZE
# and WRITE_SIZE runs); used for roofline.traffic while the kernel sources
# still hash to the value recorded there.
TRAFFIC_PROFILES = {
    2: os.path.join(ROOT, "profiles", "decode_bf16_kernel_llama8b_b8_traffic.md"),
    5: os.path.join(ROOT, "profiles", "decode_bf16_kernel_llama8b_b128_traffic.md"),
}
KERNEL_SOURCES = ("paper_2511_06029_amd/csrc/decode_attn.hip", "paper_2511_06029_amd/csrc/lethe_internal.h",
                  "paper_2511_06029_amd/csrc/device_common.h")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", type=int, choices=(2, 3, 4, 5), default=5,
                    help="5: Llama-3-8B shapes batch 128, lengths logU[1k, 64k], fixed layer shares, from the "
                         "steady state (default); 2: Llama-3-8B batch 8, 2k prompt; 3: Qwen-7B shapes batch 16, "
                         "16k cached; 4: Llama-3-8B batch 64, lengths U[8k, 32k]")
    ap.add_argument("--steps", type=int, default=None,
                    help="timed prune intervals (default: the workload's generated tokens minus warm-up)")
    ap.add_argument("--warmup", type=int, default=1, help="untimed prune intervals")
    ap.add_argument("--interval", type=int, default=None, help="decode steps per prune interval (the workload's)")
    ap.add_argument("--config3-rounds", type=int, default=16,
                    help="prune intervals of the Qwen-7B batch-16 leg after the default line's run (0: none)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU-baseline time budget of each timed part")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--policy", choices=("lethe", "lethe-shared", "shrink", "h2o", "streaming", "pyramid"),
                    default="lethe")
    ap.add_argument("--segments", type=int, default=10, help="Algorithm 1 segments D (shrink)")
    ap.add_argument("--tau", type=float, default=400.0, help="Algorithm 1 ratio threshold (shrink)")
    ap.add_argument("--prefill", action="store_true", help="time the prompt prefill with score seeding instead")
    ap.add_argument("--no-settle", action="store_true",
                    help="last step of an interval deferred like the others (the prune round then applies it)")
    ap.add_argument("--compaction", choices=("fused", "eager", "overlap"), default="eager",
                    help="fused: the round plans the compaction and the next decode step of each layer carries it "
                         "out (lethe_kv_compact_plan + lethe_decode_attn_score_compact); eager: lethe_kv_compact "
                         "in the round; overlap: lethe_kv_compact_layers layer by layer on a second stream, each "
                         "decode call of the next step waiting for its own layer's compaction")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="first copy MIB MiB device-to-device 3 times (counter calibration runs)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.prefill:
        run_prefill(args)
        return

    import torch

    def log(msg):
        print("[bench] " + msg, file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    result, held = run_decode(args, args.config, args.steps, args.warmup, args.interval, args.policy, log,
                              copy_probe=args.copy_probe)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(held, args.cpu_seconds, log)
    del held
    torch.cuda.empty_cache()
    if args.config == 5 and args.policy == "lethe" and args.config3_rounds > 0:
        # The prune-round target is stated at the Qwen-7B batch-16 workload: a
        # short leg of it, after the batch-128 buffers are freed.
        c3, held3 = run_decode(args, 3, args.config3_rounds - 1, 1, None, "lethe", log)
        del held3
        torch.cuda.empty_cache()
        result["config3"] = {k: c3[k] for k in ("config", "decode_call_us", "decode_step_ms", "prune_round_us",
                                                "prune_kernels_us", "select_us", "compaction", "prune_vs_saved",
                                                "steps", "warmup")}
        result["config3"]["roofline_frac"] = c3["roofline"]["frac"]
        result["config3"]["value"] = c3["value"]
    print(json.dumps(result), flush=True)


WORKLOADS = {
    2: "llama3-8b-shapes batch 8, 2k prompt + generated tokens, 40% budget, prune every 512, recent 128",
    3: "qwen7b-shapes batch 16, 16k cached + generated tokens, 30% budget, prune every 256, recent 256",
    4: "llama3-8b-shapes batch 64, cached lengths U[8k, 32k] + generated tokens, drifting heavy hitters, "
       "25% budget, prune every 256, recent 128",
    5: "llama3-8b-shapes batch 128, lengths logU[1k, 64k], fixed layer shares 2%-40% (10% budget), "
       "steady-state start, prune every 128, recent 64",
}


def run_decode(args, cfg_id, steps, warmup, interval, policy_name, log, copy_probe=0):
    """Decode intervals and prune rounds of one workload.  Returns the JSON
    fields of its line and what the CPU baseline reads (the end-state cache)."""
    import numpy as np
    import torch

    from paper_2511_06029_amd import lethe as L
    from paper_2511_06029_amd import policies
    from workloads import CONFIGS
    from workloads.synth import ZipfCache

    cfg = CONFIGS[cfg_id]
    dev = "cuda"
    Lyr, B, HQ, HK, D = cfg.num_layers, cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    interval = interval or cfg.prune_every
    if steps is None:
        steps = max(1, cfg.decode_steps // interval - warmup)
    windows = warmup + steps
    recent, sink = cfg.recent, cfg.sink
    policy = None if policy_name == "shrink" else policies.get(policy_name, gamma=cfg.gamma, sink=sink)
    gamma = policy.gamma if policy else cfg.gamma
    log("workload %d: %s" % (cfg_id, WORKLOADS[cfg_id]))

    gen = ZipfCache(cfg_id, device=dev)
    T = gen.lengths().astype(np.int64)          # logical length of every sequence at the start
    T0 = int(T.max())
    static_s = None
    if cfg.zipf == "fixed_weights":
        # Fixed layer shares (2%..40%, mean 10%) through sparsity_in; the full
        # cache of this workload does not fit one GPU with headroom, so the run
        # starts from the steady state: every layer holds its budget share.
        shares, static_s = gen.layer_weights()
        floor_rows = recent + sink
        n_init = np.zeros((Lyr, B), np.int64)
        for b in range(B):
            G_b = int(math.floor(cfg.budget_frac * T[b])) * Lyr
            n_init[:, b] = np.clip(np.floor(floor_rows + (G_b - floor_rows * Lyr) * shares / shares.sum()),
                                   min(T[b], floor_rows), T[b])
    else:
        n_init = np.tile(T, (Lyr, 1))
    caps = [int(n_init[:, b].max()) + interval * windows + 3 for b in range(B)]
    log("allocating cache: %d layers x %d seqs x %d kv heads, %d rows per layer (%.1f GB)"
        % (Lyr, B, HK, HK * sum(caps), Lyr * HK * sum(caps) * (4 * D + 4) / 1e9))
    cache = L.LetheCache(Lyr, caps, HQ, HK, D, dtype="bf16", device=dev)
    for l in range(Lyr):
        for b in range(B):
            n = int(n_init[l, b])
            K, V = gen.segment(l, b, n, T=int(T[b]))
            for h in range(HK):
                s0, _ = cache.seg_rows(b, h)
                cache.k[l, s0:s0 + n] = K[h]
                cache.v[l, s0:s0 + n] = V[h]
            del K, V
    cache.len.copy_(torch.from_numpy(n_init.astype(np.int32)).to(dev))
    # Decode-step inputs: 32 sets per epoch of the query direction (one epoch
    # unless the heavy hitters drift), reused cyclically within an epoch.
    P = 32
    epoch = cfg.epoch if (cfg.zipf == "drift" and cfg.epoch > 0) else 0
    E = max(1, -(-(interval * windows) // epoch)) if epoch else 1
    log("generating %d x %d decode-step input sets" % (E, P))
    qp = torch.empty((E * P, Lyr, B, HQ, D), dtype=torch.bfloat16, device=dev)
    kp = torch.empty((E * P, Lyr, B, HK, D), dtype=torch.bfloat16, device=dev)
    vp = torch.empty((E * P, Lyr, B, HK, D), dtype=torch.bfloat16, device=dev)
    for e in range(E):
        for t in range(P):
            for l in range(Lyr):
                q, k, v = gen.step(e * epoch + t, l, T=T)
                qp[e * P + t, l], kp[e * P + t, l], vp[e * P + t, l] = q, k, v
    out = torch.empty((B, HQ, D), dtype=torch.float32, device=dev)
    # One workspace for both decode calls: the settling call's layout starts
    # with the deferred call's.
    ws = cache.workspace(L.OP_DECODE if args.no_settle else L.OP_DECODE_FINAL)
    fused = args.compaction == "fused"
    overlap = args.compaction == "overlap"
    deferred = fused or overlap  # the round's compaction lands in the next step
    ws_c = cache.workspace(L.OP_COMPACT_PLAN if fused else L.OP_COMPACT)
    # overlap: the round compacts the layers on a side stream in groups of 1,
    # 2, 4, ... layers; the next step's decode call of layer l waits for the
    # group holding l only, so every group after the first runs beside the
    # decode calls of the layers before it.
    side = torch.cuda.Stream(device=dev) if overlap else None
    sel_done = torch.cuda.Event() if overlap else None
    groups = []
    while sum(n for _, n in groups) < Lyr:
        l0 = sum(n for _, n in groups)
        groups.append((l0, min(1 << len(groups), Lyr - l0)))
    group_done = [torch.cuda.Event() for _ in groups] if overlap else None
    layer_done = [group_done[gi] for gi, (_, n) in enumerate(groups) for _ in range(n)] if overlap else None
    keep = torch.empty((Lyr, cache.rows_per_layer), dtype=torch.uint8, device=dev)
    prune = policies.PruneRound(cache, policy) if policy else None
    if prune is not None and static_s is not None and policy.layer_budget == "sparsity":
        prune.s_in = torch.from_numpy(np.tile(static_s, (B, 1))).to(dev)
    evict = torch.from_numpy(n_init.astype(np.int32)).to(dev)
    # Per-layer budget of every sequence at every round, on the device ahead
    # of the timed loop: floor(rho * T_b) at the round's logical length.
    per_layer_all = np.array([[policies.per_layer_budget(cfg.budget_frac, int(T[b] + (w + 1) * interval))
                               for b in range(B)] for w in range(windows)], np.int64)
    per_layer_dev = torch.from_numpy(per_layer_all).to(dev)
    torch.cuda.synchronize()
    if copy_probe > 0:
        # A plain copy of known size: its FETCH_SIZE / WRITE_SIZE readings
        # calibrate the counters for the decode kernel in the same run.
        src = torch.ones(copy_probe << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy probe: 3 x %d MiB device-to-device" % copy_probe)

    lib = L.load()
    cref = ctypes.byref(cache.c_struct())
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    fn = lib.lethe_decode_attn_score
    # The step before each prune round settles its own score update, so the
    # round reads no K row to apply it.
    fn_last = fn if args.no_settle else lib.lethe_decode_attn_score_final
    fn_compact = lib.lethe_decode_attn_score_compact
    out_p, ws_p, wsb = ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel()
    plan_p, planb = ctypes.c_void_p(ws_c.data_ptr()), ws_c.numel()
    q_ptr = [[ctypes.c_void_p(qp[t, l].data_ptr()) for l in range(Lyr)] for t in range(E * P)]
    k_ptr = [[ctypes.c_void_p(kp[t, l].data_ptr()) for l in range(Lyr)] for t in range(E * P)]
    v_ptr = [[ctypes.c_void_p(vp[t, l].data_ptr()) for l in range(Lyr)] for t in range(E * P)]

    # Lengths once each interval's first step is done (with fused compaction
    # that step drops the evicted rows), and at the end.
    len_snap = [torch.empty((Lyr, B), dtype=torch.int32, pin_memory=True) for _ in range(windows + 1)]
    # Events: interval start, after its first and second steps, end of its
    # decode steps, after the budgets, after the selection, end of the round.
    win_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(windows + 1)]
    planned = [False]  # a compaction plan waits for the next step

    def decode_step(t, f, compact):
        for l in range(Lyr):
            if compact and overlap:
                stream.wait_event(layer_done[l])
            if compact and fused:
                rc = fn_compact(cref, l, q_ptr[t][l], k_ptr[t][l], v_ptr[t][l], gamma, 0.0, out_p, plan_p, planb,
                                ws_p, wsb, sp)
            else:
                rc = f(cref, l, q_ptr[t][l], k_ptr[t][l], v_ptr[t][l], gamma, 0.0, out_p, ws_p, wsb, sp)
            if rc != 0:
                raise RuntimeError("decode call: %s" % L.status_string(rc))

    def compact_on_side(keep_t):
        sel_done.record(stream)
        side.wait_event(sel_done)
        for gi, (l0, n) in enumerate(groups):
            L.kv_compact_layers(cache, l0, n, keep_t, ws_c, stream=side)
            group_done[gi].record(side)

    def run_window(w):
        ev = win_ev[w]
        ev[0].record(stream)
        for i in range(interval):
            tg = w * interval + i
            t = (min(tg // epoch, E - 1) * P if epoch else 0) + tg % P
            decode_step(t, fn_last if i == interval - 1 else fn, i == 0 and planned[0])
            if i == 0:
                planned[0] = False
                ev[1].record(stream)
                len_snap[w].copy_(cache.len, non_blocking=True)
            elif i == 1:
                ev[2].record(stream)
        ev[3].record(stream)
        if policy_name == "shrink":
            L.score_flush(cache)
            ev[4].record(stream)
            L.segmented_shrink(cache, args.segments, args.tau, recent, sink, evict, None, keep)
            ev[5].record(stream)
            if fused:
                L.kv_compact_plan(cache, keep, ws_c)
            elif overlap:
                compact_on_side(keep)
            else:
                L.kv_compact(cache, keep, ws_c)
        else:
            if policy.window_fills:
                r, sk = prune.budgets(int(per_layer_all[w].min()), recent)
            else:
                r, sk = prune.budgets(per_layer_dev[w], recent)
            ev[4].record(stream)
            prune.select(r, sk)
            ev[5].record(stream)
            if fused:
                prune.plan(ws_c)
            elif overlap:
                compact_on_side(prune.keep)
            else:
                prune.compact()
        planned[0] = deferred
        ev[6].record(stream)

    log("warm-up: %d interval(s) of %d decode steps" % (warmup, interval))
    # With overlapped compaction only the launch stream is waited for here:
    # the side stream's work of the last round runs into the next interval
    # and is charged to it, as a fused compaction is.
    sync = stream.synchronize if overlap else torch.cuda.synchronize
    for w in range(warmup):
        run_window(w)
    sync()
    log("timed: %d interval(s)" % steps)
    t0 = time.perf_counter()
    for w in range(warmup, windows):
        run_window(w)
        log("interval %d enqueued" % w)
    sync()
    t1 = time.perf_counter()
    if not deferred:
        len_snap[windows].copy_(cache.len)
    if deferred:
        # The last round's compaction happens in the next step: two more
        # steps (outside the timed run) give its cost.
        ev = win_ev[windows]
        ev[0].record(stream)
        decode_step(0, fn, True)
        ev[1].record(stream)
        decode_step(1, fn, False)
        ev[2].record(stream)
        torch.cuda.synchronize()
        # Rows the last round kept: the lengths after those two steps, less them.
        len_snap[windows].copy_(cache.len - 2)
        last_kept = int(len_snap[windows].numpy().astype(np.int64).sum())
    else:
        last_kept = int(len_snap[windows].numpy().astype(np.int64).sum())
    status = int(cache.dev_status[0])
    if status != 0:
        raise RuntimeError("device status bits set: %d (%s)" % (status, ", ".join(L.dev_status_names(status))))
    log("timed intervals done")

    # Work accounting from the length snapshots (lengths after each
    # interval's first step, which appended one row to the rows kept).
    elem = 2
    row_bytes = HK * (2 * D * elem + 8)               # K + V + score read/write, all KV heads
    fixed_bytes = B * HQ * D * (elem + 4) + 2 * B * HK * D * elem
    kept0 = [len_snap[w].numpy().astype(np.int64) - 1 for w in range(windows)]  # rows before step 0
    tokens = 0
    tokens_rest = 0  # steps 1 .. interval-1 only
    for w in range(warmup, windows):
        n0 = kept0[w]
        tokens += interval * int(n0.sum()) + Lyr * B * interval * (interval + 1) // 2
        tokens_rest += (interval - 1) * int(n0.sum()) + Lyr * B * ((interval * (interval + 1)) // 2 - 1)
    elapsed = t1 - t0
    ms = lambda w, i, j: win_ev[w][i].elapsed_time(win_ev[w][j])
    decode_ms = [ms(w, 0, 3) for w in range(warmup, windows)]
    round_ms = [ms(w, 3, 6) for w in range(warmup, windows)]
    select_ms = [ms(w, 4, 5) for w in range(warmup, windows)]
    # What a fused or overlapped compaction adds to the step that carries it
    # out (or runs beside it): that step's time less the next step's (one row
    # longer, no compaction).
    extra = [max(ms(w + 1, 0, 1) - ms(w + 1, 1, 2), 0.0) if deferred else 0.0 for w in range(windows)]
    prune_ms = [round_ms[i] + extra[warmup + i] for i in range(steps)]
    # Roofline of lethe_decode_attn_score: one kernel launch per call, back to
    # back on the launch stream; the events bracket every decode call of the
    # timed intervals after each interval's first step (which carries a fused
    # compaction), so their span / calls is the average launch duration (the
    # settling calls' second, small kernel included: one step in an interval).
    n_calls = steps * (interval - 1) * Lyr
    avg_call_s = float(np.sum([ms(w, 1, 3) for w in range(warmup, windows)])) / 1e3 / n_calls
    avg_call_bytes = (tokens_rest * row_bytes + n_calls * fixed_bytes) / n_calls
    achieved = avg_call_bytes / avg_call_s / 1e9
    traffic = load_traffic(cfg_id, avg_call_bytes) if policy_name == "lethe" else None

    # Selection reads every live score once per KV head and writes a mask
    # byte per row and head (lengths at the end of each interval).
    sel_rows = 0
    for w in range(warmup, windows):
        sel_rows += int(kept0[w].sum()) + Lyr * B * interval
    select_gbs = sel_rows * HK * 5 / (float(np.sum(select_ms)) / 1e3) / 1e9

    value = tokens / elapsed
    all_dec = np.array([ms(w, 1, 3) for w in range(windows)]) / (interval - 1)
    all_prune = np.array([ms(w, 3, 6) + extra[w] for w in range(windows)])
    start_rows = np.array([int(kept0[w].sum()) for w in range(windows)])
    prune_vs_saved = prune_against_saved(all_dec, all_prune, start_rows, last_kept, Lyr * B, interval, extra)
    workload = WORKLOADS[cfg_id]
    if policy_name == "lethe-shared":
        workload += ", one kept set per layer and sequence"
    elif policy_name in ("h2o", "streaming", "pyramid"):
        workload += ", %s rule" % policy_name
    elif policy_name == "shrink":
        workload = ("%s-shapes batch %d, %d cached + generated tokens, Algorithm 1 shrinking every %d "
                    "(D=%d, tau=%g, recent %d, first threshold %d)" % (
                        "qwen7b" if cfg_id == 3 else "llama3-8b", B, T0, interval, args.segments, args.tau,
                        recent, T0))
    result = {
        "metric": "KV tokens scanned/s (fused decode-attn+score, prune rounds included)",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": elapsed * 1e3 / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Zipf key-bias caches, random queries)",
        "config": {
            "workload": workload,
            "layers": Lyr, "q_heads": HQ, "kv_heads": HK, "head_dim": D, "batch": B, "storage": "bf16",
            "accumulation": "fp32",
            "prompt": T0 if cfg.length_dist == "fixed" else "%s%s" % (cfg.length_dist, list(cfg.length_range)),
            "generated": interval * windows, "interval": interval, "gamma": gamma,
        },
        "decode_step_ms": float(np.mean(decode_ms)) / interval,
        "prune_round_us": float(np.mean(prune_ms)) * 1e3,
        "prune_kernels_us": float(np.mean(round_ms)) * 1e3,
        "compaction": args.compaction,
        "policy": policy_name,
        "settled_last_step": not args.no_settle,
        "select_us": float(np.mean(select_ms)) * 1e3,
        "select_hbm_gbs": select_gbs,
        "decode_call_us": avg_call_s * 1e6,
        "decode_hbm_gbs": achieved,
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic and traffic["bytes"],
            "kernel": "decode_bf16_kernel<%d, %d> (lethe_decode_attn_score, one launch per layer call)" % (D, HQ // HK),
            "bytes_per_launch": avg_call_bytes, "launches": n_calls,
            "traffic_source": traffic and traffic["source"],
        },
        "final_lengths_mean": float(len_snap[windows].numpy().mean()),
        "prune_vs_saved": prune_vs_saved,
    }
    held = {"cache": cache, "gamma": gamma, "recent": recent, "sink": sink,
            "per_layer": per_layer_all[-1], "s_in": static_s if (policy and policy.layer_budget == "sparsity") else None}
    del qp, kp, vp, ws, ws_c, keep, prune, evict, per_layer_dev, out
    return result, held


MFMA_BF16_PEAK_TFLOPS = 2500.0


def prune_against_saved(dec_step_ms, prune_ms, start_rows, last_kept, rows_per_step, interval, extra_ms):
    """What each prune round costs against the decode time it saves over the
    next interval.  dec_step_ms[w]: average decode step of interval w (ms);
    prune_ms[w]: the round after it; start_rows[w]: cached rows (all layers,
    sequences) when interval w starts; last_kept: rows after the last round;
    rows_per_step: rows one decode step appends (layers x sequences).

    The per-step decode time is fit as a + b * (cached rows at the interval's
    middle) over every interval, and the round after interval w saves
    interval * b * (rows it evicted): the rows at the interval's end less the
    rows the next interval starts from.  Returns None when the intervals do
    not differ enough in size for the fit (a run that starts at the steady
    state)."""
    import numpy as np
    windows = len(dec_step_ms)
    start_rows = np.asarray(start_rows, np.float64)
    mid_rows = start_rows + rows_per_step * (interval + 2) / 2.0
    if windows < 2 or np.ptp(mid_rows) < 0.1 * mid_rows.mean():
        return None
    slope, icpt = np.polyfit(mid_rows, np.asarray(dec_step_ms, np.float64), 1)
    ratios = []
    for w in range(windows):
        end_rows = start_rows[w] + rows_per_step * interval
        nxt = start_rows[w + 1] if w + 1 < windows else last_kept
        saved_ms = interval * slope * (end_rows - nxt)
        ratios.append(float(prune_ms[w] / saved_ms) if saved_ms > 0 else None)
    steady = [r for r in ratios[1:] if r is not None]
    return {
        "round1": ratios[0], "steady_median": float(np.median(steady)) if steady else None,
        "per_round": ratios, "decode_ms_per_token_step": float(slope), "decode_step_fixed_ms": float(icpt),
        "prune_round_ms": [float(x) for x in prune_ms],
        "fused_step_extra_ms": [float(x) for x in extra_ms],
    }


def run_prefill(args):
    """Prompt prefill with score seeding on the Llama-3-8B shapes, batch 8,
    2048-token prompts, all 32 layers per step."""
    import numpy as np
    import torch

    from paper_2511_06029_amd import lethe as L
    from workloads import CONFIGS
    from workloads.synth import ZipfCache

    def log(msg):
        print("[bench] " + msg, file=sys.stderr, flush=True)

    cfg = CONFIGS[2]
    dev = "cuda"
    torch.cuda.set_device(0)
    if args.steps is None:
        args.steps = 10  # prefills of all 32 layers
    Lyr, B, HQ, HK, D, T = cfg.num_layers, cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.prompt
    log("allocating cache: %d layers x %d seqs x %d kv heads x %d rows" % (Lyr, B, HK, T))
    cache = L.LetheCache(Lyr, [T] * B, HQ, HK, D, dtype="bf16", device=dev)
    gen = ZipfCache(2, device=dev)
    for l in range(Lyr):
        for b in range(B):
            K, V = gen.segment(l, b, T, T=T)
            for h in range(HK):
                s0, _ = cache.seg_rows(b, h)
                cache.k[l, s0:s0 + T] = K[h]
                cache.v[l, s0:s0 + T] = V[h]
    cache.len.fill_(T)
    rows = B * T
    g = torch.Generator(device=dev)
    g.manual_seed(2)
    q = (torch.randn((Lyr, rows, HQ, D), generator=g, device=dev) * 1.0).to(torch.bfloat16)
    q_start = torch.arange(B, dtype=torch.int64, device=dev) * T
    q_len = torch.full((B,), T, dtype=torch.int32, device=dev)
    out = torch.empty((rows, HQ, D), dtype=torch.float32, device=dev)
    ws = cache.prefill_workspace(rows)
    lib = L.load()
    cref = ctypes.byref(cache.c_struct())
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    qp = [ctypes.c_void_p(q[l].data_ptr()) for l in range(Lyr)]
    out_p, ws_p, wsb = ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel()
    qs_p, ql_p = ctypes.c_void_p(q_start.data_ptr()), ctypes.c_void_p(q_len.data_ptr())
    fn = lib.lethe_prefill_attn_score
    torch.cuda.synchronize()

    def step():
        cache.score.zero_()
        for l in range(Lyr):
            rc = fn(cref, l, qp[l], qs_p, ql_p, rows, T, T, 0.0, out_p, ws_p, wsb, sp)
            if rc != 0:
                raise RuntimeError("lethe_prefill_attn_score: %s" % L.status_string(rc))

    log("warm-up: %d step(s)" % args.warmup)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    log("timed: %d step(s)" % args.steps)
    t0 = time.perf_counter()
    for k in range(args.steps):
        cache.score.zero_()
        ev[k][0].record(stream)
        for l in range(Lyr):
            rc = fn(cref, l, qp[l], qs_p, ql_p, rows, T, T, 0.0, out_p, ws_p, wsb, sp)
            if rc != 0:
                raise RuntimeError("lethe_prefill_attn_score: %s" % L.status_string(rc))
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    status = int(cache.dev_status[0])
    if status != 0:
        raise RuntimeError("device status bits set: %d (%s)" % (status, ", ".join(L.dev_status_names(status))))
    elapsed = t1 - t0
    call_ms = float(np.sum([e[0].elapsed_time(e[1]) for e in ev])) / (args.steps * Lyr)
    # Algorithmic work of one call: causal Q K^T and P V once per query head,
    # 4 D flops per (query, attended row) pair.
    pairs = T * (T + 1) // 2
    flops = 4.0 * D * pairs * B * HQ
    achieved = flops / (call_ms / 1e3) / 1e12
    tokens = B * T * args.steps
    result = {
        "metric": "prompt tokens/s (prefill attention + Eq. 2 score seeding, all layers)",
        "value": tokens / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Zipf key-bias caches, random queries)",
        "config": {
            "workload": "llama3-8b-shapes batch 8, 2048-token prompts, prefill with score seeding",
            "layers": Lyr, "q_heads": HQ, "kv_heads": HK, "head_dim": D, "batch": B, "storage": "bf16",
            "prompt": T,
        },
        "prefill_call_ms": call_ms,
        "roofline": {
            "bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
            "kernel": "prefill_fwd_kernel<128, 4> + prefill_score_kernel<128, 4> (lethe_prefill_attn_score, "
                      "one call per layer)",
            "flops_per_launch": flops, "launches": args.steps * Lyr,
        },
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = prefill_cpu_baseline(cache, q, args.cpu_seconds, log)
    print(json.dumps(result), flush=True)


def prefill_cpu_baseline(cache, q, budget_s, log):
    """The oracle's prefill on whole (layer 0, sequence, KV head) segments for
    about budget_s seconds of one host thread; a token is one prompt position
    through one layer with all its heads."""
    import numpy as np

    import oracle

    log("cpu baseline: oracle prefill on full-prompt segments (%.0f s budget)" % budget_s)
    T = int(cache.len[0, 0])
    G, D = cache.G, cache.D
    qh = q[0].float().cpu().numpy()
    segs, t_cpu = 0, 0.0
    for b in range(cache.B):
        for h in range(cache.HK):
            s0, _ = cache.seg_rows(b, h)
            K = cache.k[0, s0:s0 + T].float().cpu().numpy()
            V = cache.v[0, s0:s0 + T].float().cpu().numpy()
            t = time.perf_counter()
            oracle.prefill(qh[b * T:(b + 1) * T, h * G:(h + 1) * G], K, V, None, 1 / math.sqrt(D))
            t_cpu += time.perf_counter() - t
            segs += 1
            if t_cpu >= budget_s:
                break
        if t_cpu >= budget_s:
            break
    tokens = segs * T / cache.HK
    return {"value": tokens / t_cpu, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": "oracle prefill attention + score seeding of %d (layer 0, seq, kv-head) segments of %d "
                      "prompt tokens (%.1f s on one host thread)" % (segs, T, t_cpu)}


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def load_traffic(cfg_id, bytes_per_launch):
    """HBM bytes per launch from the workload's committed counter summary,
    scaled from its run's algorithmic bytes per launch to this run's; None
    when there is no summary or the kernel sources changed since it was
    taken."""
    path = TRAFFIC_PROFILES.get(cfg_id)
    try:
        text = open(path).read()
    except (OSError, TypeError):
        return None
    vals = {}
    for line in text.splitlines():
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    try:
        if vals["source_sha256"] != kernel_source_hash():
            return None
        measured = float(vals["hbm_bytes_per_launch"])
        algorithmic = float(vals["algorithmic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None
    return {"bytes": measured / algorithmic * bytes_per_launch,
            "source": "%s (ratio %.4f of algorithmic bytes)" % (os.path.relpath(path, ROOT), measured / algorithmic)}


# Host threads of the parallel oracle runs: the host share one GPU has on the
# measurement box (its nproc can show more).
POOL_THREADS = 16


def host_cpu():
    """CPU model name and the number of host threads visible to this process."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        threads = len(os.sched_getaffinity(0))
    except AttributeError:
        threads = os.cpu_count()
    return model, threads


def cpu_baseline(held, budget_s, log):
    """The oracle on the end-state cache, in the same units: its decode step
    (attention + Eq. 5) on one host thread for about budget_s seconds, then
    over POOL_THREADS threads; and its prune round (Hoyer sparsity of the
    head-summed scores, the budget split, RASR selection and compaction of K,
    V and scores) on whole sequences, likewise."""
    model, threads = host_cpu()
    dec = cpu_baseline_decode(held["cache"], budget_s, held["gamma"], log)
    prune = cpu_baseline_prune(held, budget_s, log)
    dec["cpu_model"] = model
    dec["host_threads"] = threads
    dec["prune_round"] = prune
    return dec


def cpu_baseline_decode(cache, budget_s, gamma, log):
    """The oracle's decode step on segments of the final cache, for about
    `budget_s` seconds of one host thread, in the same unit (a token is a
    (layer, sequence, position) row across all KV heads)."""
    import numpy as np

    import oracle

    log("cpu baseline: oracle decode on end-state segments (%.0f s budget)" % budget_s)
    rng = np.random.default_rng(0)
    lens = cache.len.cpu().numpy()
    reps = 4  # steps per segment copy: the host copies are not what is timed
    scale = 1 / math.sqrt(cache.D)
    rows = 0
    segs = 0
    t_cpu = 0.0
    l = 0
    kept = []  # the first segments, for the multi-thread run
    while t_cpu < budget_s and l < cache.L:
        for b in range(cache.B):
            n = int(lens[l, b])
            for h in range(cache.HK):
                s0, _ = cache.seg_rows(b, h)
                K = cache.k[l, s0:s0 + n].float().cpu().numpy()
                V = cache.v[l, s0:s0 + n].float().cpu().numpy()
                s = cache.score[l, s0:s0 + n].double().cpu().numpy()
                if len(kept) < 64:
                    kept.append((K, V, s.copy()))
                for _ in range(reps):
                    q = rng.standard_normal((cache.G, cache.D)).astype(np.float32)
                    t = time.perf_counter()
                    _, s = oracle.attend(q, K, V, s, gamma, scale)
                    t_cpu += time.perf_counter() - t
                    rows += n
                segs += 1
            if t_cpu >= budget_s:
                break
        l += 1
    tokens = rows / cache.HK
    result = {"value": tokens / t_cpu, "unit": "tokens/s", "cores": 1, "kind": "oracle",
              "sample": "oracle decode attention + score update, %d steps on each of %d (layer, seq, kv-head) "
                        "segments of the end-state cache (%d rows, %.1f s on one host thread)"
                        % (reps, segs, rows, t_cpu)}
    result["parallel"] = cpu_baseline_parallel(kept, reps, gamma, scale, cache.G, cache.D, cache.HK, log)
    return result


def cpu_baseline_parallel(segments, reps, gamma, scale, G, D, HK, log, min_seconds=3.0):
    """The same oracle steps on up to 64 of those segments, one segment per task
    on a pool of host threads (the oracle's C code runs without the GIL), for at
    least min_seconds of wall time."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle

    threads = POOL_THREADS
    log("cpu baseline: the same oracle steps on %d segments over %d threads" % (len(segments), threads))
    qs = [np.random.default_rng(1 + i).standard_normal((reps, G, D)).astype(np.float32) for i in range(len(segments))]

    def run(i):
        K, V, s = segments[i]
        for r in range(reps):
            _, s = oracle.attend(qs[i][r], K, V, s, gamma, scale)
        return reps * K.shape[0]

    rows, passes = 0, 0
    t = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as pool:
        while passes == 0 or time.perf_counter() - t < min_seconds:
            rows += sum(pool.map(run, range(len(segments))))
            passes += 1
    dt = time.perf_counter() - t
    return {"value": rows / HK / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "%d passes of %d steps on each of %d segments (%d rows) over %d host threads, %.1f s wall"
                      % (passes, reps, len(segments), rows, threads, dt)}


def _prune_sequence(seq, recent, sink):
    """One sequence's prune round on the oracle: layer sparsity (or the fixed
    layer values), the budget split, RASR selection per KV head and the
    compaction of K, V and scores.  Returns the rows (all KV heads counted
    once per position) it went through."""
    import numpy as np

    import oracle

    layers, s_in, G_b = seq
    L = len(layers)
    n = np.array([lay[0].shape[1] for lay in layers], np.int32)
    if s_in is None:
        S = np.array([oracle.layer_sparsity(lay[0]) for lay in layers], np.float32)
    else:
        S = np.asarray(s_in, np.float32)
    budget, _ = oracle.budget_split(n, S, recent, sink, G_b)
    for l in range(L):
        s_h, K_h, V_h = layers[l]
        for h in range(s_h.shape[0]):
            keep = oracle.rasr_select(s_h[h].astype(np.float32), int(budget[l]), recent, sink)
            oracle.compact(K_h[h], keep)
            oracle.compact(V_h[h], keep)
            oracle.compact(s_h[h], keep)
    return int(n.sum())


def cpu_baseline_prune(held, budget_s, log, keep_for_parallel=16, min_seconds=3.0):
    """The oracle's prune round on whole sequences of the end-state cache (all
    layers and KV heads of a sequence: the budget split couples its layers),
    one host thread for about budget_s seconds, then the first sequences over
    POOL_THREADS threads.  The rate is in (layer, sequence, position) rows per
    second; full_round_s scales it to every row of the cache."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    cache = held["cache"]
    recent, sink = held["recent"], held["sink"]
    per_layer = held["per_layer"]
    s_in = held["s_in"]
    lens = cache.len.cpu().numpy()
    total_rows = int(lens.sum())
    log("cpu baseline: oracle prune round on whole sequences (%.0f s budget)" % budget_s)

    def fetch(b):
        layers = []
        for l in range(cache.L):
            n = int(lens[l, b])
            idx = [cache.seg_rows(b, h)[0] for h in range(cache.HK)]
            s_h = np.stack([cache.score[l, i:i + n].double().cpu().numpy() for i in idx])
            K_h = np.stack([cache.k[l, i:i + n].float().cpu().numpy() for i in idx])
            V_h = np.stack([cache.v[l, i:i + n].float().cpu().numpy() for i in idx])
            layers.append((s_h, K_h, V_h))
        return (layers, s_in, int(per_layer[b]) * cache.L)

    rows, seqs, t_cpu = 0, 0, 0.0
    kept = []
    for b in range(cache.B):
        seq = fetch(b)
        t = time.perf_counter()
        rows += _prune_sequence(seq, recent, sink)
        t_cpu += time.perf_counter() - t
        seqs += 1
        if len(kept) < keep_for_parallel:
            kept.append(seq)
        if t_cpu >= budget_s:
            break
    rate = rows / t_cpu
    result = {"value": rate, "unit": "rows/s", "cores": 1, "kind": "oracle",
              "full_round_s": total_rows / rate,
              "sample": "oracle prune round (sparsity, budget split, RASR select, compaction of K, V and scores) "
                        "of %d whole sequences of the end-state cache (%d (layer, seq, position) rows, %.1f s on "
                        "one host thread); full_round_s scales it to the cache's %d rows"
                        % (seqs, rows, t_cpu, total_rows)}
    threads = POOL_THREADS
    log("cpu baseline: the same prune rounds on %d sequences over %d threads" % (len(kept), threads))
    prow, passes = 0, 0
    t = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as pool:
        while passes == 0 or time.perf_counter() - t < min_seconds:
            prow += sum(pool.map(lambda sq: _prune_sequence(sq, recent, sink), kept))
            passes += 1
    dt = time.perf_counter() - t
    result["parallel"] = {"value": prow / dt, "unit": "rows/s", "cores": threads, "kind": "oracle",
                          "full_round_s": total_rows / (prow / dt),
                          "sample": "%d passes over %d sequences (%d rows) over %d host threads, %.1f s wall"
                                    % (passes, len(kept), prow, threads, dt)}
    return result


if __name__ == "__main__":
    main()
