"""Benchmark of the phrase-memory lookup + inject path on one MI355X.

Default workload (batch-64 decode against the 2^20-phrase bf16 table):
a step is one tfe_lookup_inject call over R = 256 independent batch-64 decode
steps stacked into one launch (16384 rows, each with its own 3-token window
and hidden row), i.e. one pass of key formation, probe, gather and gated
injection over one batch of synthetic input.  Eight input sets (tokens,
hidden in, hidden out) rotate so more than 512 MB are touched between reuses
of a set, which keeps the hidden rows out of the 256 MB last-level cache; the
2 GiB value table is larger than that cache by itself.

The JSON line also carries the latency mode (one batch-64 step per call), the
roofline of the kernel (algorithmic bytes per launch over the average launch
duration, measured with HIP events on the launch stream) and the CPU oracle
timed on a bounded sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--stack R] [--sets N]

Tiered workload (2^25 phrases, 64 GiB of bf16 values in pinned host memory;
the full 2^26-phrase, 128 GiB size needs a host that can pin 128 GiB), a
4M-row HBM cache pre-filled with the most frequent rows, batch-64 decode over
per-row token streams, 8 predicted candidates per row and step with the true
next token among them with probability 0.7):

  python bench.py --workload tiered [--tier-steps N] [--t-hide-us 0,20,100,500]

Offline phrase-table construction (n-gram counting + top-N on the GPU):

  python bench.py --workload build

Multi-match workload (every matched phrase retained and combined with
length weights, Eq. 4 / Eq. 11), same stacked decode launch as the default:

  python bench.py --workload multi

The other two resident table shapes: 8 x 4096 prefill against the
2^22-phrase 2/3/4-gram table (8 GiB of values), and batch-256 decode against
the 2^25-phrase table (64 GiB), per call and with 64 steps stacked per call:

  python bench.py --workload prefill
  python bench.py --workload large

Each configuration (prefetch off / on, emulated compute window T_hide between
a step's lookup and the next) starts from a freshly loaded table.  A step is
one tfe_lookup_inject (plus, with prefetch, one tfe_prefetch for the next
step on a side stream, issued right after the lookup, then T_hide of device
work on the main stream).
"""
import argparse
import json
import os
import sys
import time

# Idle OpenMP workers (torch's CPU thread pool) sleep instead of spinning:
# spinning workers take the CPU from the host threads that stage a tiered
# table's pageable rows (measured: 16384-row miss-path calls 5-6 ms instead
# of 0.6-0.8 ms right after CPU-parallel work).  Set before torch loads.
os.environ.setdefault("OMP_WAIT_POLICY", "PASSIVE")

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "lookup+inject tokens/sec and achieved HBM GB/s, batch-64 decode, 1 MI355X"
HBM_PEAK_GBPS = 8000.0

# HBM bytes per launch of the stacked-decode kernel, from the rocprofv3
# FETCH_SIZE / WRITE_SIZE passes (calibrated on the reference copy kernel) in
# profiles/k_lookup_inject_bf16_d1024_decode_stacked16384.md.  Reported only
# while the kernel sources still hash to the profiled version.
PROFILED_TRAFFIC = {
    "sources_sha256": "4fece8a7d469ff90d4cf9bddfb427eed004d59f96cac15bc45f4826f406b2d78",
    "bytes_per_launch": 93801562,
}
KERNEL_SOURCES = ("paper_2607_07388_amd/csrc/tfe_lookup.hip",
                  "paper_2607_07388_amd/csrc/tfe_device.h",
                  "paper_2607_07388_amd/csrc/tfe_index.h")


# The same for the multi-match kernel in the same 16384-row launch, from the
# passes in profiles/k_lookup_inject_multi_bf16_d1024_decode_stacked16384.md.
PROFILED_TRAFFIC_MULTI = {
    "sources_sha256": "ced797b78d255db95b6544bf97d341421fb20e2f6f63030710ecac13e1354c45",
    "bytes_per_launch": 98836857,
}
MULTI_SOURCES = ("paper_2607_07388_amd/csrc/tfe_multi.hip",
                 "paper_2607_07388_amd/csrc/tfe_device.h",
                 "paper_2607_07388_amd/csrc/tfe_index.h")

# The same for one call of the early-exit head (W 151936 x 1024 bf16, 64 rows,
# K = 128): the one-launch k_head_fused, from the passes in
# profiles/k_head_fused_v151936_d1024_b64_k128.md.
PROFILED_TRAFFIC_HEAD = {
    "sources_sha256": "7b4673180138ac6e265fddd9bbf2936a9155dbb45a0f719f9ae1d65f7bc524c0",
    "bytes_per_launch": 318459155,
}
HEAD_SOURCES = ("paper_2607_07388_amd/csrc/tfe_head.hip",
                "paper_2607_07388_amd/csrc/tfe_head.h",
                "paper_2607_07388_amd/csrc/tfe_head_api.cpp")


# The same for one construction of the 2^26-token stream's top 2^19 2-grams
# (every kernel of the call summed), from the passes in
# profiles/tfe_ngram_top_zipf_streams.md.
PROFILED_TRAFFIC_BUILD = {
    "sources_sha256": "ba8919c86fed4482f21188001dc87ab38f975b0d5aebc860104d69bb78c6eea6",
    "bytes_per_call": 8271581751,
}
BUILD_SOURCES = ("paper_2607_07388_amd/csrc/tfe_build.hip",)


def kernel_sources_sha256(files=KERNEL_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()
D = 1024
ESZ = 2  # bf16


def host_cpu():
    """The host processor the CPU baseline ran on: model name and the
    threads the operating system exposes."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"host_cpu": model, "host_threads": os.cpu_count()}


def algorithmic_bytes(T, hits, keys, window):
    """Bytes the method must move for T positions (bf16, out of place):
    hidden row in and out, one value row and one row id per hit, one 8-byte
    key slot per formed key, the token window, and hit/slot/len outputs."""
    return (T * 2 * D * ESZ + hits * (D * ESZ + 4) + keys * 8 + T * window * 4 + T * (1 + 4 + 1))


def counts_after_run(n_sets, run, sync, count):
    """Per-set counts read from outputs that the set's own call wrote: one
    untimed call of every rotating set (the warmup may have covered fewer
    sets than there are), a synchronisation, then count(k) for each set.
    Output buffers start filled with a sentinel, so counting a set that never
    ran would read the sentinel, not hits."""
    for k in range(n_sets):
        run(k)
    sync()
    return [count(k) for k in range(n_sets)]


def settle(call, sync, seconds=0.03):
    """Untimed calls for about `seconds` of wall time right before a timed
    region, on top of the W warmup steps: a short timed region (20 stacked
    decode calls take under 0.4 ms) otherwise starts while the GPU is still
    raising its clocks after the idle gaps of set-up and hit counting.
    Synchronises every 64 calls so the queue stays short."""
    t0, k = time.perf_counter(), 0
    while time.perf_counter() - t0 < seconds:
        call(k)
        k += 1
        if k % 64 == 0:
            sync()
    sync()
    return k


def check_line(result):
    """Refuses to print a line whose rates cannot be measurements: every hit
    rate in [0, 1] and every roofline fraction in [0, 1]."""
    def walk(x, path):
        if isinstance(x, dict):
            for k, v in x.items():
                if k in ("hit_rate", "frac", "frac_of_8tbs") and v is not None:
                    if not (0.0 <= float(v) <= 1.0):
                        raise AssertionError("%s.%s = %r is outside [0, 1]" % (path, k, v))
                walk(v, path + "." + k)
        elif isinstance(x, list):
            for i, v in enumerate(x):
                walk(v, "%s[%d]" % (path, i))
    walk(result, "line")
    return result


def algorithmic_bytes_multi(T, rows, keys, window, L):
    """Multi-match variant: one value row and row id per retained phrase, a
    match mask and L row ids per position."""
    return (T * 2 * D * ESZ + rows * (D * ESZ + 4) + keys * 8 + T * window * 4 + T * (1 + 4 * L))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--stack", type=int, default=256, help="batch-64 steps per call")
    ap.add_argument("--sets", type=int, default=8, help="rotating input sets")
    ap.add_argument("--latency-steps", type=int, default=2000)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload",
                    choices=("decode", "multi", "tiered", "head", "build", "prefill", "large"),
                    default="decode")
    ap.add_argument("--head-k", type=int, default=128)
    ap.add_argument("--build-reps", type=int, default=3)
    ap.add_argument("--tier-steps", type=int, default=2000)
    ap.add_argument("--tier-warmup", type=int, default=100)
    ap.add_argument("--t-hide-us", default="0,100")
    ap.add_argument("--tier-log2-phrases", type=int, default=26,
                    help="tiered table size (2^26: 128 GiB of values)")
    ap.add_argument("--tier-pinned-log2", type=int, default=25,
                    help="rows kept in pinned host memory (2^25: 64 GiB, this box's pin limit)")
    ap.add_argument("--prefetch-budget", type=int, default=64)
    ap.add_argument("--tier-fill", default="inline,side",
                    help="miss fill modes of the tiered table to run (inline, side)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2607_07388_amd import tfe
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.workload == "tiered":
        return run_tiered(args)
    if args.workload == "head":
        return run_head(args)
    if args.workload == "build":
        return run_build(args)
    if args.workload in ("prefill", "large"):
        return run_resident_config(args)
    t0 = time.time()
    table = synth.config2_table()
    gt = H.GpuTable(table)
    print("# table loaded (%d phrases) in %.1f s" % (table.n_phrases, time.time() - t0),
          file=sys.stderr, flush=True)

    B = 64 * args.stack
    window, ctx, S = 3, 2, 1
    stream = torch.cuda.current_stream()
    sets = []
    for k in range(args.sets):
        batch = synth.decode_batch(1, B, set_index=100 + k)
        tok = torch.from_numpy(batch.tokens).cuda()
        hid = torch.empty((B, D), dtype=torch.bfloat16, device="cuda")
        synth.normal_fill_device(hid.data_ptr(), 0, B, D, batch.seed, batch.hidden_tag, 1.0,
                                 synth.BF16, stream.cuda_stream)
        sets.append((batch, tok, hid, H.Outputs(B, D, synth.BF16)))
    torch.cuda.synchronize()

    multi = args.workload == "multi"
    L = table.n_max - table.n_min + 1
    if multi:
        mslots = [torch.full((B, L), -7, dtype=torch.int32, device="cuda") for _ in sets]

    def call(k):
        _, tok, hid, outs = sets[k % len(sets)]
        if multi:
            tfe.tfe_lookup_inject_multi(gt.handle, tok, B, ctx, S, hid, outs.out, outs.hit,
                                        mslots[k % len(sets)], tfe.TFE_WEIGHT_LENGTH,
                                        tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)
        else:
            tfe.tfe_lookup_inject(gt.handle, tok, B, ctx, S, hid, outs.out, outs.hit, outs.slot,
                                  outs.len, tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)

    for k in range(args.warmup):
        call(k)
    if multi:
        # Retained rows per set: the population count of the match masks.
        hits = counts_after_run(
            len(sets), call, torch.cuda.synchronize,
            lambda k: int(sum(((sets[k][3].hit >> j) & 1).sum().item() for j in range(L))))
        positions_hit = [int((s[3].hit > 0).sum().item()) for s in sets]
    else:
        hits = counts_after_run(len(sets), call, torch.cuda.synchronize,
                                lambda k: int(sets[k][3].hit.sum().item()))
        positions_hit = hits
    keys = B * L
    settle(call, torch.cuda.synchronize)

    # Timed region: K back-to-back calls bracketed by HIP events on the launch
    # stream; their elapsed time over K is the kernel's average launch duration.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    for k in range(args.steps):
        call(k)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    avg_launch = e0.elapsed_time(e1) * 1e-3 / args.steps  # seconds
    if multi:
        bytes_per_call = [algorithmic_bytes_multi(B, h, keys, window, L) for h in hits]
    else:
        bytes_per_call = [algorithmic_bytes(B, h, keys, window) for h in hits]
    avg_bytes = float(np.mean([bytes_per_call[k % len(sets)] for k in range(args.steps)]))
    achieved = avg_bytes / avg_launch / 1e9
    tokens_per_s = B * args.steps / wall

    # Practical copy ceiling: a plain 16-byte-per-lane device copy of 64 MiB
    # (read + write) over four rotating buffer pairs.
    nb = 64 << 20
    cbufs = [(torch.empty(nb, dtype=torch.uint8, device="cuda"),
              torch.empty(nb, dtype=torch.uint8, device="cuda")) for _ in range(4)]
    for k in range(8):
        synth.copy_device(cbufs[k % 4][1].data_ptr(), cbufs[k % 4][0].data_ptr(), nb, 1024,
                          stream.cuda_stream)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for k in range(200):
        synth.copy_device(cbufs[k % 4][1].data_ptr(), cbufs[k % 4][0].data_ptr(), nb, 1024,
                          stream.cuda_stream)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * nb * 200 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del cbufs

    if multi:
        return finish_multi(args, table, gt, sets, mslots, B, ctx, S, window, L, tokens_per_s,
                            wall, achieved, avg_bytes, avg_launch, copy_gbps, hits,
                            positions_hit)

    # Latency mode: one batch-64 decode step per call.
    lat_sets = []
    for k in range(args.sets):
        batch = synth.decode_batch(1, 64, set_index=200 + k)
        tok = torch.from_numpy(batch.tokens).cuda()
        hid = H.to_device(batch.hidden(), synth.BF16)
        lat_sets.append((tok, hid, H.Outputs(64, D, synth.BF16)))
    torch.cuda.synchronize()
    # Per-call event pairs: each call's own duration, as a decode step sees it.
    lev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.latency_steps)]
    torch.cuda.synchronize()
    for k in range(args.latency_steps):
        tok, hid, outs = lat_sets[k % len(lat_sets)]
        lev[k][0].record(stream)
        tfe.tfe_lookup_inject(gt.handle, tok, 64, ctx, S, hid, outs.out, outs.hit, outs.slot,
                              outs.len, tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)
        lev[k][1].record(stream)
    torch.cuda.synchronize()
    ldur = np.array([a.elapsed_time(b) for a, b in lev]) * 1e-3
    # Back-to-back: the sustained decode-step rate of one stream.
    l0 = time.perf_counter()
    for k in range(args.latency_steps):
        tok, hid, outs = lat_sets[k % len(lat_sets)]
        tfe.tfe_lookup_inject(gt.handle, tok, 64, ctx, S, hid, outs.out, outs.hit, outs.slot,
                              outs.len, tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)
    torch.cuda.synchronize()
    lwall = time.perf_counter() - l0
    def lat_call(k):
        tok, hid, outs = lat_sets[k]
        tfe.tfe_lookup_inject(gt.handle, tok, 64, ctx, S, hid, outs.out, outs.hit, outs.slot,
                              outs.len, tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)

    lhits = float(np.mean(counts_after_run(len(lat_sets), lat_call, torch.cuda.synchronize,
                                           lambda k: lat_sets[k][2].hit.float().mean().item())))
    # Graph-replayed: 64 decode steps (rotating over the sets) captured once
    # and replayed, as a decode loop without per-call launch overhead.
    graph_us = None
    try:
        gsteps = 64

        def gloop():
            cs = torch.cuda.current_stream().cuda_stream
            for k in range(gsteps):
                tok, hid, outs = lat_sets[k % len(lat_sets)]
                tfe.tfe_lookup_inject(gt.handle, tok, 64, ctx, S, hid, outs.out, outs.hit,
                                      outs.slot, outs.len, tfe.TFE_GATE_SIGMOID, 1.0, cs)

        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            gloop()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            gloop()
        graph.replay()
        torch.cuda.synchronize()
        reps = max(1, args.latency_steps // gsteps)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(reps):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) * 1e3 / (reps * gsteps)
        del graph
    except RuntimeError as e:  # graphs unavailable: report without them
        print("# graph replay skipped: %s" % e, file=sys.stderr)

    traffic = None
    if (kernel_sources_sha256() == PROFILED_TRAFFIC["sources_sha256"] and args.stack == 256):
        traffic = PROFILED_TRAFFIC["bytes_per_launch"]

    result = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "batch-64 decode, stacked throughput mode: %d batch-64 steps per call "
                        "(%d rows, 3-token windows, Zipf(1.1) ids), 2^20-phrase 2/3-gram table, "
                        "1024-wide bf16 values (2 GiB), sigmoid gate, out of place" % (args.stack, B),
            "table_phrases": table.n_phrases,
            "rows_per_call": B,
            "rotating_sets": args.sets,
            "hit_rate": float(np.mean(hits) / B),
        },
        "hbm_gbps_algorithmic": achieved,
        "roofline": {
            "bound": "hbm",
            "kernel": "k_lookup_inject<bf16, D=1024>",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "bytes_per_launch": avg_bytes,
            "avg_launch_us": avg_launch * 1e6,
            "copy_reference_gbps": copy_gbps,
            "frac_of_copy_reference": achieved / copy_gbps,
        },
        "latency_mode": {
            "rows_per_call": 64,
            "median_us_per_step": float(np.median(ldur) * 1e6),
            "mean_us_per_step": float(ldur.mean() * 1e6),
            "back_to_back_us_per_step": lwall / args.latency_steps * 1e6,
            "tokens_per_s_back_to_back": 64 * args.latency_steps / lwall,
            "graph_replay_us_per_step": graph_us,
            "tokens_per_s_graph_replay": (64e6 / graph_us) if graph_us else None,
            "hit_rate": lhits,
            "algorithmic_gbps_median": algorithmic_bytes(64, lhits * 64, 128, 3) /
                                       float(np.median(ldur)) / 1e9,
        },
    }

    if not args.no_cpu_baseline:
        import oracle
        ot = H.oracle_table(table)
        batch = sets[0][0]
        hidden = synth.normal_range(batch.seed, batch.hidden_tag, 0, B, D, 1.0, synth.BF16)
        hit, row, _ = ot.lookup(batch.tokens, ctx, S)
        uniq, inv = np.unique(row[row >= 0].astype(np.int64), return_inverse=True)
        vals = table.value_rows(uniq)
        idx = np.full(B, -1, np.int64)
        idx[row >= 0] = inv
        rows_done, c0 = 0, time.perf_counter()
        while time.perf_counter() - c0 < args.cpu_seconds:
            ot.lookup(batch.tokens, ctx, S)
            oracle.inject(hidden, vals, idx, synth.BF16)
            rows_done += B
        csec = time.perf_counter() - c0
        result["cpu_baseline"] = {
            "value": rows_done / csec,
            "unit": "tokens/s",
            "cores": 1,
            "kind": "oracle", **host_cpu(),
            "sample": "%d passes of std::map lookup + double-precision gate/inject over one "
                      "%d-row stacked decode set (%.1f s, single thread)"
                      % (rows_done // B, B, csec),
        }
        # The same oracle calls on every host core: the rows of the set split
        # over threads (the oracle's table is read-only, and its C calls
        # release the interpreter lock).
        import threading
        nthr = max(1, min(16, os.cpu_count() or 1))
        bounds = [B * t // nthr for t in range(nthr + 1)]
        parts = []
        for t in range(nthr):
            lo, hi = bounds[t], bounds[t + 1]
            parts.append((np.ascontiguousarray(batch.tokens[lo:hi]), hidden[lo:hi].copy(),
                          idx[lo:hi].copy()))
        counts = [0] * nthr
        stop = time.perf_counter() + args.cpu_seconds

        def work(t):
            tk, hd, ix = parts[t]
            while time.perf_counter() < stop:
                ot.lookup(tk, ctx, S)
                oracle.inject(hd, vals, ix, synth.BF16)
                counts[t] += tk.shape[0]

        threads = [threading.Thread(target=work, args=(t,)) for t in range(nthr)]
        c0 = time.perf_counter()
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        psec = time.perf_counter() - c0
        result["cpu_baseline_threads"] = {
            "value": sum(counts) / psec, "unit": "tokens/s", "cores": nthr, "kind": "oracle",
            **host_cpu(),
            "sample": "the same passes with the set's rows split over %d threads (%.1f s)"
                      % (nthr, psec)}
    gt.close()
    print(json.dumps(check_line(result)))


def finish_multi(args, table, gt, sets, mslots, B, ctx, S, window, L, tokens_per_s, wall,
                 achieved, avg_bytes, avg_launch, copy_gbps, hits, positions_hit):
    """JSON line of the multi-match workload (Eq. 4, Eq. 11): the stacked
    decode launch with every matched phrase retained, length weights."""
    result = {
        "metric": "multi-match lookup+inject tokens/sec and achieved HBM GB/s, batch-64 decode, "
                  "1 MI355X",
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "batch-64 decode, stacked throughput mode: %d batch-64 steps per call "
                        "(%d rows, 3-token windows, Zipf(1.1) ids), 2^20-phrase 2/3-gram table, "
                        "every matched phrase retained, length weights, sigmoid gate, out of "
                        "place" % (args.stack, B),
            "table_phrases": table.n_phrases,
            "rows_per_call": B,
            "rotating_sets": args.sets,
            "hit_rate": float(np.mean(positions_hit) / B),
            "retained_rows_per_position": float(np.mean(hits) / B),
        },
        "hbm_gbps_algorithmic": achieved,
        "roofline": {
            "bound": "hbm",
            "kernel": "k_lookup_inject_multi<bf16, D=1024>",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": (PROFILED_TRAFFIC_MULTI["bytes_per_launch"]
                        if kernel_sources_sha256(MULTI_SOURCES) ==
                        PROFILED_TRAFFIC_MULTI["sources_sha256"] and args.stack == 256 else None),
            "bytes_per_launch": avg_bytes,
            "avg_launch_us": avg_launch * 1e6,
            "copy_reference_gbps": copy_gbps,
            "frac_of_copy_reference": achieved / copy_gbps,
        },
    }
    if not args.no_cpu_baseline:
        import oracle
        from tests import harness as H
        ot = H.oracle_table(table)
        batch = sets[0][0]
        hidden = synth_hidden(batch, B)
        _, rows = ot.lookup_all(batch.tokens, ctx, S)
        uniq, inv = np.unique(rows[rows >= 0].astype(np.int64), return_inverse=True)
        vals = table.value_rows(uniq)
        idx = np.full(rows.shape, -1, np.int64)
        idx[rows >= 0] = inv
        done, c0 = 0, time.perf_counter()
        while time.perf_counter() - c0 < args.cpu_seconds:
            ot.lookup_all(batch.tokens, ctx, S)
            oracle.inject_multi(hidden, vals, idx, table.n_min, table.dtype)
            done += B
        csec = time.perf_counter() - c0
        result["cpu_baseline"] = {
            "value": done / csec,
            "unit": "tokens/s",
            "cores": 1,
            "kind": "oracle", **host_cpu(),
            "sample": "%d passes of the all-matches std::map lookup + double-precision weighted "
                      "inject over one %d-row stacked decode set (%.1f s, single thread)"
                      % (done // B, B, csec),
        }
    gt.close()
    print(json.dumps(check_line(result)))


def keys_formed(B, ctx, S, n_min, n_max):
    """Keys the lookup forms for B rows of ctx + S tokens (every token valid):
    position s has ctx + s + 1 tokens up to it, so lengths n <= ctx + s + 1."""
    per_row = sum(sum(1 for n in range(n_min, n_max + 1) if n <= ctx + s + 1) for s in range(S))
    return B * per_row


def run_resident_config(args):
    """Throughput of the resident lookup + inject on the two other table
    shapes: 8 x 4096 prefill against the 2^22-phrase 2/3/4-gram table (8 GiB
    of values), and batch-256 decode against the 2^25-phrase table (64 GiB),
    per call and stacked (64 batch-256 steps per call).  The prefill and
    stacked shapes rotate input sets that together exceed the 256 MB
    last-level cache; the per-call batch-256 shape is bound by launch time
    (its 8 input sets stay cached, the value rows do not)."""
    import torch

    import synth
    from paper_2607_07388_amd import tfe
    from tests import harness as H

    stream = torch.cuda.current_stream()
    t0 = time.time()
    if args.workload == "prefill":
        table = synth.config3_table()
        shapes = [("prefill 8 x 4096", 4, lambda k: synth.prefill_batch(2, 8, 4096, set_index=k))]
    else:
        table = synth.config4_table()
        shapes = [("batch-256 decode", 8,
                   lambda k: synth.decode_batch(3, 256, s=1.05, set_index=k)),
                  ("batch-256 decode, 64 steps stacked per call", 8,
                   lambda k: synth.decode_batch(3, 256 * 64, s=1.05, set_index=40 + k))]
    gt = H.GpuTable(table)
    print("# table loaded (%d phrases) in %.1f s" % (table.n_phrases, time.time() - t0),
          file=sys.stderr, flush=True)
    runs = []
    for name, nsets, make in shapes:
        sets = []
        for k in range(nsets):
            batch = make(k)
            B, ctx, S = batch.tokens.shape[0], batch.ctx, batch.S
            T = B * S
            tok = torch.from_numpy(batch.tokens).cuda()
            hid = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
            synth.normal_fill_device(hid.data_ptr(), 0, T, D, batch.seed, batch.hidden_tag, 1.0,
                                     synth.BF16, stream.cuda_stream)
            sets.append((tok, hid, H.Outputs(T, D, synth.BF16), B, ctx, S))
        torch.cuda.synchronize()

        def call(k):
            tok, hid, outs, B, ctx, S = sets[k % nsets]
            tfe.tfe_lookup_inject(gt.handle, tok, B, ctx, S, hid, outs.out, outs.hit, outs.slot,
                                  outs.len, tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)

        for k in range(args.warmup):
            call(k)
        hits = counts_after_run(nsets, call, torch.cuda.synchronize,
                                lambda k: int(sets[k][2].hit.sum().item()))
        settle(call, torch.cuda.synchronize)
        _, _, _, B, ctx, S = sets[0]
        T = B * S
        keys = keys_formed(B, ctx, S, table.n_min, table.n_max)
        window = (ctx + S) / S
        steps = args.steps
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        e0.record(stream)
        for k in range(steps):
            call(k)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        avg_launch = e0.elapsed_time(e1) * 1e-3 / steps
        avg_bytes = float(np.mean([algorithmic_bytes(T, hits[k % nsets], keys, window)
                                   for k in range(steps)]))
        runs.append({
            "shape": name, "positions_per_call": T, "sets": nsets,
            "hit_rate": float(np.mean(hits)) / T,
            "us_per_call": avg_launch * 1e6,
            "tokens_per_s": T * steps / wall,
            "bytes_per_call": avg_bytes,
            "hbm_gbps_algorithmic": avg_bytes / avg_launch / 1e9,
            "frac_of_8tbs": avg_bytes / avg_launch / 8e12,
        })
        print("# %s: %.2f us per call" % (name, avg_launch * 1e6), file=sys.stderr, flush=True)
        del sets
    head = runs[-1]
    result = {
        "metric": "lookup+inject tokens/sec, %s, 1 MI355X" % head["shape"],
        "value": head["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head["us_per_call"] * 1e-3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": ("8 x 4096 prefill (ctx 0), 2^21 2-grams + 2^20 3-grams + "
                                "2^20 4-grams of a 200M-token Zipf(1.1) stream (8 GiB bf16 "
                                "values), sigmoid gate, out of place"
                                if args.workload == "prefill" else
                                "batch-256 decode (3-token windows, Zipf(1.05) ids), 2^25-phrase "
                                "2/3-gram table (64 GiB bf16 values), sigmoid gate, out of place"),
                   "table_phrases": table.n_phrases},
        "roofline": {"bound": "hbm", "kernel": "k_lookup_inject<bf16, D=1024>",
                     "achieved": head["hbm_gbps_algorithmic"], "peak": 8000.0, "unit": "GB/s",
                     "frac": head["frac_of_8tbs"], "traffic": None},
        "runs": runs,
    }
    gt.close()
    print(json.dumps(check_line(result)))


def synth_hidden(batch, B):
    import synth
    return synth.normal_range(batch.seed, batch.hidden_tag, 0, B, D, 1.0, synth.BF16)


def run_head(args):
    """Early-exit prefetch head (Eq. 13, Eq. 14): softmax(W h) and its top K
    for one batch-64 decode step, W = 151936 x 1024 bf16 (311 MB)."""
    import torch

    import synth
    from paper_2607_07388_amd import tfe

    V, Dh, B, K = synth.V, 1024, 64, args.head_k
    stream = torch.cuda.current_stream()
    w = torch.empty((V, Dh), dtype=torch.bfloat16, device="cuda")
    synth.normal_fill_device(w.data_ptr(), 0, V, Dh, 5, 42, 0.1, synth.BF16, stream.cuda_stream)
    sets = []
    for k in range(args.sets):
        h = torch.empty((B, Dh), dtype=torch.bfloat16, device="cuda")
        synth.normal_fill_device(h.data_ptr(), 0, B, Dh, 5, 43 + 16 * k, 1.0, synth.BF16,
                                 stream.cuda_stream)
        sets.append((h, torch.empty((B, K), dtype=torch.int32, device="cuda"),
                     torch.empty((B, K), dtype=torch.float32, device="cuda")))
    head = tfe.tfe_head_create(w, V, Dh, B, K)
    torch.cuda.synchronize()

    def call(k):
        h, ids, prob = sets[k % len(sets)]
        tfe.tfe_head_topk(head, h, B, K, ids, prob, stream.cuda_stream)

    for k in range(args.warmup):
        call(k)
    settle(call, torch.cuda.synchronize)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    for k in range(args.steps):
        call(k)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    avg = e0.elapsed_time(e1) * 1e-3 / args.steps
    # The same calls captured in a HIP graph (16 per graph, as a model step
    # that captures its head would run them), timed after the timed region.
    graph_us = None
    try:
        gcalls = 16

        def gloop():
            cs = torch.cuda.current_stream().cuda_stream
            for k in range(gcalls):
                h, ids, prob = sets[k % len(sets)]
                tfe.tfe_head_topk(head, h, B, K, ids, prob, cs)

        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            gloop()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            gloop()
        graph.replay()
        torch.cuda.synchronize()
        reps = max(1, args.steps // gcalls)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(reps):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) * 1e3 / (reps * gcalls)
        del graph
    except RuntimeError as e:  # graphs unavailable: report without them
        print("# graph replay skipped: %s" % e, file=sys.stderr)
    # Algorithmic bytes of one call: W once, the hidden rows, the outputs.
    nbytes = V * Dh * 2 + B * Dh * 2 + B * K * 8
    flops = 2.0 * V * Dh * B
    result = {
        "metric": "early-exit prefetch head calls/sec (softmax(W h) + top-K), batch-64 decode, "
                  "1 MI355X",
        "value": args.steps / wall,
        "unit": "calls/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "early-exit head: W 151936 x 1024 bf16 ~N(0, 0.1), 64 hidden "
                               "rows ~N(0, 1), top %d" % K, "vocab": V, "dim": Dh, "batch": B,
                   "k": K},
        "roofline": {
            "bound": "hbm",
            "kernel": "tfe_head_topk (k_head_fused: one launch)",
            "achieved": nbytes / avg / 1e9,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": nbytes / avg / 1e9 / HBM_PEAK_GBPS,
            "traffic": (PROFILED_TRAFFIC_HEAD["bytes_per_launch"]
                        if kernel_sources_sha256(HEAD_SOURCES) ==
                        PROFILED_TRAFFIC_HEAD["sources_sha256"] and (V, Dh, B, K) ==
                        (151936, 1024, 64, 128) else None),
            "bytes_per_launch": nbytes,
            "avg_launch_us": avg * 1e6,
            "mfma_tflops": flops / avg / 1e12,
        },
        "graph_replay_us_per_call": graph_us,
        "graph_replay_frac_of_8tbs": (nbytes / (graph_us * 1e-6) / 1e9 / HBM_PEAK_GBPS
                                      if graph_us else None),
    }
    if not args.no_cpu_baseline:
        import oracle
        wh = synth.normal_range(5, 42, 0, V, Dh, 0.1, synth.BF16)
        hh = synth.normal_range(5, 43, 0, B, Dh, 1.0, synth.BF16)
        done, c0 = 0, time.perf_counter()
        while time.perf_counter() - c0 < args.cpu_seconds:
            oracle.head_topk(wh, hh[done % B:done % B + 1], K, synth.BF16)
            done += 1
        csec = time.perf_counter() - c0
        result["cpu_baseline"] = {
            "value": done / B / csec,
            "unit": "calls/s",
            "cores": 1,
            "kind": "oracle", **host_cpu(),
            "sample": "%d of the 64 rows of one call (double-precision logits over the full "
                      "vocabulary + partial sort), %.1f s, single thread, scaled to calls"
                      % (done, csec),
        }
    tfe.tfe_head_free(head)
    print(json.dumps(check_line(result)))


def build_bytes_per_window(n, vocab):
    """Data the construction pipeline moves per window of the stream.  A key
    holds 18 n bits (one more when vocab = 2^18, whose invalid-window mark
    needs a bit above the token fields); the radix passes take 9 bits each.
    n <= 3: the first pass forms the keys from the tokens (4 B read by its
    histogram, 4 B read and the 8 B key written by its scatter), every later
    pass reads the keys for its histogram (8 B) and reads and writes them in
    its scatter (16 B); the run count reads the sorted keys twice (16 B).
    n = 4: the low word's first pass writes key and 32-bit payload (the
    oldest token: 4 + 4 + 12 B), its five later passes move the payload too
    (8 + 24 B each), the passes over the high word's 18 (19) bits carry the
    low word (4 + 24 B each), and the run count reads both words twice
    (24 B).
    The selection and ranking work on far fewer items."""
    extra = 1 if vocab >= (1 << 18) else 0
    if n <= 3:
        passes = (18 * n + extra + 8) // 9
        return 16 + 24 * (passes - 1) + 16
    hi_passes = (18 + extra + 8) // 9
    return 20 + 5 * 32 + hi_passes * 28 + 24


def run_build(args):
    """Offline phrase-table construction (Sec. 4.2): the most frequent 2-, 3-
    and 4-grams of the workload streams, as the decode and prefill tables are
    built (2^26 tokens -> top 2^19 2- and 3-grams; 200M tokens -> 2^21
    2-grams, 2^20 3-grams and 2^20 4-grams after skipping the 80000 most
    frequent of each)."""
    import torch

    import synth
    from paper_2607_07388_amd import tfe

    stream = torch.cuda.current_stream()
    runs = []
    cases = [("2^26-token Zipf(1.1) stream", synth.workload2_stream(), [(2, 0, 1 << 19),
                                                                          (3, 0, 1 << 19)]),
             ("200M-token Zipf(1.1) stream", synth.workload3_stream(),
              [(2, synth.CONFIG3_STOP[0], 1 << 21), (3, synth.CONFIG3_STOP[1], 1 << 20),
               (4, synth.CONFIG3_STOP[2], 1 << 20)])]
    cpu_sample = None
    for name, toks, jobs in cases:
        tok_d = torch.from_numpy(toks).cuda()
        N = toks.size
        if cpu_sample is None:
            cpu_sample = toks[: 1 << 20].copy()
        del toks
        for n, skip, top in jobs:
            tup = torch.empty((top, n), dtype=torch.int32, device="cuda")
            cnt = torch.empty(top, dtype=torch.int64, device="cuda")
            tfe.tfe_ngram_top(tok_d, N, synth.V, n, skip, top, tup, cnt, stream.cuda_stream)
            reps = max(1, args.build_reps)
            t0 = time.perf_counter()
            for _ in range(reps):
                m = tfe.tfe_ngram_top(tok_d, N, synth.V, n, skip, top, tup, cnt,
                                      stream.cuda_stream)
            sec = (time.perf_counter() - t0) / reps
            moved = N * build_bytes_per_window(n, synth.V)
            runs.append({"stream": name, "n": n, "skip": skip, "top": top, "written": m,
                         "ms": sec * 1e3, "tokens_per_s": N / sec,
                         "pipeline_gbps": moved / sec / 1e9})
            print(json.dumps(runs[-1]), file=sys.stderr, flush=True)
        del tok_d
    main_run = runs[0]
    result = {
        "metric": "phrase-table construction tokens/sec (n-gram count + top-N), 1 MI355X",
        "value": main_run["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": max(1, args.build_reps),
        "warmup": 1,
        "ms_per_step": main_run["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": "top 2^19 2-grams of the 2^26-token Zipf(1.1) stream; other "
                               "lengths and the 200M-token stream under 'runs'"},
        "roofline": {
            "bound": "hbm",
            "kernel": "tfe_ngram_top pipeline (key formation, radix passes, run count)",
            "achieved": main_run["pipeline_gbps"],
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": main_run["pipeline_gbps"] / HBM_PEAK_GBPS,
            "traffic": (PROFILED_TRAFFIC_BUILD["bytes_per_call"]
                        if kernel_sources_sha256(BUILD_SOURCES) ==
                        PROFILED_TRAFFIC_BUILD["sources_sha256"] else None),
        },
        "runs": runs,
    }
    if not args.no_cpu_baseline:
        import oracle
        done, c0 = 0, time.perf_counter()
        while time.perf_counter() - c0 < args.cpu_seconds:
            oracle.ngram_top(cpu_sample, synth.V, 2, 0, 1 << 19)
            done += cpu_sample.size
        csec = time.perf_counter() - c0
        result["cpu_baseline"] = {
            "value": done / csec, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            **host_cpu(),
            "sample": "2-gram top-2^19 of the first 2^20 tokens of the stream, repeated "
                      "(%.1f s, single thread)" % csec}
    print(json.dumps(check_line(result)))


def run_tiered(args):
    import torch

    import synth
    from paper_2607_07388_amd import tfe
    from tests import harness as H

    B, K, C = 64, 8, 4 << 20
    t0 = time.time()
    log = lambda m: print("# %s (%.1f s)" % (m, time.time() - t0), file=sys.stderr, flush=True)
    table = synth.config5_table(args.tier_log2_phrases)
    P = table.n_phrases
    log("table of %d phrases generated" % P)
    # The most frequent rows (the table is ordered by count) in pinned host
    # memory, the rest, if any, in pageable host memory behind the table's
    # staging queue: one process pins at most 64 GiB here.
    Pp = min(P, 1 << args.tier_pinned_log2)
    vals = torch.empty((Pp, D), dtype=torch.bfloat16, pin_memory=True)
    log("pinned %.1f GiB" % (vals.numel() * 2 / 2**30))
    stream = torch.cuda.current_stream()
    synth.normal_fill_device(synth.host_device_ptr(vals.data_ptr()), 0, Pp, D, table.seed,
                             synth.TAG_VALUES, table.sigma, synth.BF16, stream.cuda_stream)
    torch.cuda.synchronize()
    pageable = None
    if Pp < P:
        pageable = H.pageable_values(table, Pp, stream)
        log("pageable %.1f GiB" % (pageable.nbytes / 2**30))
    log("values drawn into host memory")
    split = dict(pinned_rows=Pp if Pp < P else 0, pageable_values=pageable)

    # Host -> device copy ceiling of this machine (pinned, 1 GiB).
    hb = vals[: (1 << 29) // D]
    db = torch.empty_like(hb, device="cuda")
    db.copy_(hb, non_blocking=True)
    torch.cuda.synchronize()
    c0 = time.perf_counter()
    for _ in range(5):
        db.copy_(hb, non_blocking=True)
    torch.cuda.synchronize()
    h2d_gbps = 5 * hb.numel() * 2 / (time.perf_counter() - c0) / 1e9
    del db

    n_steps = args.tier_warmup + args.tier_steps
    seqs = synth.zipf_tokens(4, synth.TAG_QUERY, B * (n_steps + 3), 1.1).reshape(B, n_steps + 3)
    seqs_d = torch.from_numpy(seqs).cuda()
    cands = np.stack([synth.workloads.candidates(4, B, K, seqs[:, s + 3], step=s)
                      for s in range(n_steps)])
    cands_d = torch.from_numpy(cands).cuda()
    # Candidate probabilities for the scored prefetch: falling geometrically
    # with the candidate's rank (0.5^k, normalised), as a softmax's top-K
    # list does.
    pk = np.float32(0.5) ** np.arange(K, dtype=np.float32)
    probs_d = torch.from_numpy(np.tile(pk / pk.sum(), (B, 1)).astype(np.float32)).cuda()
    tails_d = [seqs_d[:, s + 1:s + 3].contiguous() for s in range(n_steps)]
    wins_d = [seqs_d[:, s:s + 3].contiguous() for s in range(n_steps)]
    hid = [torch.empty((B, D), dtype=torch.bfloat16, device="cuda") for _ in range(8)]
    for k, hdn in enumerate(hid):
        synth.normal_fill_device(hdn.data_ptr(), 0, B, D, 4, 900 + k, 1.0, synth.BF16,
                                 stream.cuda_stream)
    outs = H.Outputs(B, D, synth.BF16)
    side = torch.cuda.Stream()
    log("inputs ready")

    fills = {"inline": tfe.TFE_FILL_INLINE, "side": tfe.TFE_FILL_SIDE_STREAM}
    fill_names = [f for f in args.tier_fill.split(",") if f]
    results = []
    for t_hide, fill, prefetch in [(float(x), f, p) for x in args.t_hide_us.split(",")
                                   for f in fill_names for p in ("off", "all", "scored")]:
        desc = tfe.make_desc(table.tokens, table.lens, 2, 3, synth.V, vals, D, synth.BF16, 0,
                             0.5, hbm_cache_rows=C, adopt_host_values=1, prefill_rows=C,
                             miss_fill=fills[fill], **split)
        handle = tfe.tfe_table_load(desc, stream.cuda_stream)
        log("tiered table loaded (T_hide %g us, fill %s, prefetch %s)" % (t_hide, fill,
                                                                        prefetch))

        def step(s):
            tfe.tfe_lookup_inject(handle, wins_d[s], B, 2, 1, hid[s % 8], outs.out, outs.hit,
                                  outs.slot, outs.len, tfe.TFE_GATE_SIGMOID, 1.0,
                                  stream.cuda_stream)
            if prefetch == "all":
                tfe.tfe_prefetch(handle, tails_d[s], 2, cands_d[s], B, K, side)
            elif prefetch == "scored":
                tfe.tfe_prefetch_scored(handle, tails_d[s], 2, cands_d[s], probs_d, B, K,
                                        args.prefetch_budget, side)
            if t_hide > 0:
                synth.spin_device(t_hide, stream.cuda_stream)

        for s in range(args.tier_warmup):
            step(s)
        torch.cuda.synchronize()
        tfe.tfe_reset_stats(handle)
        w0 = time.perf_counter()
        for s in range(args.tier_warmup, n_steps):
            step(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        st = tfe.tfe_get_stats(handle)
        tfe.tfe_table_free(handle)
        n = args.tier_steps
        results.append({
            "t_hide_us": t_hide,
            "fill": fill,
            "prefetch": prefetch,
            "us_per_step": wall / n * 1e6,
            "tokens_per_s": B * n / wall,
            "table_hit_rate": st["hits"] / max(1, st["positions"]),
            "hbm_cache_hit_rate": st["cache_hits"] / max(1, st["hits"]),
            "prefetch_precision": st["prefetch_used"] / max(1, st["prefetch_filled"]),
            "prefetch_filled_per_step": st["prefetch_filled"] / n,
            "prefetch_dropped_per_step": st["prefetch_dropped"] / n,
            "host_bytes_per_step": st["host_bytes"] / n,
            "host_link_gbps": st["host_bytes"] / wall / 1e9,
        })
        print(json.dumps(results[-1]), file=sys.stderr, flush=True)
    # Miss path against the host link: a cold cache (nothing prefilled) and
    # stacked calls of 16384 decode rows, so that most matched rows are read
    # from pinned host memory and copied into the cache.
    RB = 16384
    cold = []
    for fill, k in [(f, k) for f in fill_names for k in range(4)]:
        if k == 0:
            desc = tfe.make_desc(table.tokens, table.lens, 2, 3, synth.V, vals, D, synth.BF16, 0,
                                 0.5, hbm_cache_rows=C, adopt_host_values=1, prefill_rows=0,
                                 miss_fill=fills[fill], **split)
            handle = tfe.tfe_table_load(desc, stream.cuda_stream)
            # Untimed call whose windows match nothing (every token -1): it
            # sizes the table's per-call scratch for RB positions and leaves
            # the cold cache untouched, so no timed call includes allocation.
            ntok = torch.full((RB, 3), -1, dtype=torch.int32, device="cuda")
            nh = torch.zeros((RB, D), dtype=torch.bfloat16, device="cuda")
            nb = H.Outputs(RB, D, synth.BF16)
            tfe.tfe_lookup_inject(handle, ntok, RB, 2, 1, nh, nb.out, nb.hit, nb.slot, nb.len,
                                  tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)
            torch.cuda.synchronize()
            del ntok, nh, nb
        bt = synth.decode_batch(6, RB, set_index=500 + k)
        tok = torch.from_numpy(bt.tokens).cuda()
        hd = torch.empty((RB, D), dtype=torch.bfloat16, device="cuda")
        synth.normal_fill_device(hd.data_ptr(), 0, RB, D, bt.seed, bt.hidden_tag, 1.0,
                                 synth.BF16, stream.cuda_stream)
        ob = H.Outputs(RB, D, synth.BF16)
        torch.cuda.synchronize()
        tfe.tfe_reset_stats(handle)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        tfe.tfe_lookup_inject(handle, tok, RB, 2, 1, hd, ob.out, ob.hit, ob.slot, ob.len,
                              tfe.TFE_GATE_SIGMOID, 1.0, stream.cuda_stream)
        e1.record(stream)
        torch.cuda.synchronize()
        st = tfe.tfe_get_stats(handle)
        sec = e0.elapsed_time(e1) * 1e-3
        rows = ob.slot.cpu().numpy()
        cold.append({"fill": fill, "call": k, "us": sec * 1e6, "hits": st["hits"],
                     "cache_misses": st["cache_misses"], "host_bytes": st["host_bytes"],
                     "pageable_rows_matched": int((rows >= Pp).sum()),
                     "host_link_gbps": st["host_bytes"] / sec / 1e9})
        print(json.dumps(cold[-1]), file=sys.stderr, flush=True)
        if k == 3:
            tfe.tfe_table_free(handle)
    first = cold[0]
    best = max((r for r in results if r["t_hide_us"] == 0.0), key=lambda r: r["tokens_per_s"],
               default=results[0])
    print(json.dumps(check_line({
        "metric": "tiered lookup+inject tokens/sec, batch-64 decode, 1 MI355X",
        "value": best["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.tier_steps,
        "warmup": args.tier_warmup,
        "ms_per_step": best["us_per_step"] / 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "tiered: 2^%d-phrase 2/3-gram table, %d GiB bf16 values in host memory "
                        "(%d GiB pinned, the rest pageable behind the staging queue), 4M-row "
                        "HBM cache (LRU), batch-64 decode, 8 candidates per row"
                        % (args.tier_log2_phrases, P * D * 2 >> 30, Pp * D * 2 >> 30),
            "h2d_copy_gbps": h2d_gbps,
            "prefetch_budget_scored": args.prefetch_budget,
            "miss_fill": "headline: %s (best no-prefetch, T_hide 0); all modes under 'runs'"
                         % best["fill"],
        },
        "miss_path": {
            "rows_per_call": RB,
            "calls": cold,
            "roofline": {"bound": "host-link", "achieved": first["host_link_gbps"],
                         "peak": h2d_gbps, "unit": "GB/s",
                         "frac": first["host_link_gbps"] / h2d_gbps,
                         "note": "first cold call of fill mode %s; peak = pinned "
                                 "host-to-device copy measured in the same run" % first["fill"]},
        },
        "runs": results,
    })))


if __name__ == "__main__":
    main()
