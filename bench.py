#!/usr/bin/env python3
"""Benchmark of the GDN tail-replay hot path on one MI355X.

One step = the whole hot path over one batch of resident synthetic input:
Independent Tail-Replay of every value head's state from zero over the last
r tokens of the matched prefix (paper Section 3, Eq. 2), then the chunked
forward over the new suffix from the rebuilt state, emitting its outputs.

Default workload: a stack of 36 GDN layers with hybrid-model head shapes
(16 key heads, 32 value heads, d_k = d_v = 128, bf16 q/k/v, fp32 g/beta/state),
each with its own seeded inputs; matched prefix 32768 tokens, replay tail 3277
tokens (10 %), 1024 new suffix tokens.  The step runs the layers one after the
other, as the layers of a group depend on each other (paper Section 3): per
layer one ``gdn_replay_forward`` call (the tail replay, then the suffix forward
from the rebuilt state; the suffix's chunk preparation runs beside the tail's
scan), launched eagerly on one stream.  ``value`` = tokens through the path per
second, 36 x (3277 + 1024) per step.  Beside it: the same step as two calls
per layer (``gdn_tail_replay`` + ``gdn_chunk_forward``, bit for bit the same
results) and replayed from a HIP graph, the 36 layers as one batched call
(layers as sequences), the 36 layers as a hybrid model's 12 groups of 3 GDN
layers (groups replay independently, paper Section 3: one fused call per
depth with that depth's 12 layers as its sequences, the 3 depths in order), the
rebuild latency of the 36 replays (warm, cold, queued), per-stage kernel
durations from HIP events that the library records on the stream its kernels
run on, ``roofline`` for the dominant kernel, the one-layer workload
(tail 819 + suffix 512) and ``cpu_baseline`` (the fp64 oracle on the same
inputs on the host cores).

``--sweep`` times the other workloads (one JSON line each); ``--summarize-pmc
FETCH_DIR WRITE_DIR`` (no GPU) turns two rocprofv3 --pmc runs of ``bench.py
--calib-copy`` (FETCH_SIZE, then WRITE_SIZE) into the traffic summary under
profiles/ that later runs report as ``traffic``.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "GDN tail-replay tokens/sec/GPU + state-rebuild latency; % of MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
CHUNK = 64
CALIB_BYTES = 1 << 30          # plain copy used to calibrate the PMC byte counters (> the 256 MB MALL)
FLUSH_BYTES = 512 << 20        # > 256 MB Infinity Cache: evicts it between cold reps
QUEUE_SPIN_CYCLES = 2_000_000  # spin kernel (~0.8 ms) that outlasts the host's enqueue of one call
GROUP_DEPTH = 3                # GDN layers per hybrid-model group in the grouped form (3 GDN : 1 FA)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic_workload2.json")
KERNEL_SOURCES = ("include/gdn_tail_replay.h", "paper_2608_30310_amd/csrc/gdn_plan.h",
                  "paper_2608_30310_amd/csrc/gdn_plan.cpp", "paper_2608_30310_amd/csrc/gdn_device.h",
                  "paper_2608_30310_amd/csrc/gdn_intra.h", "paper_2608_30310_amd/csrc/gdn_scan.h",
                  "paper_2608_30310_amd/csrc/gdn_decode.h",
                  "paper_2608_30310_amd/csrc/gdn_api.hip", "paper_2608_30310_amd/build.py")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--layers", type=int, default=36,
                    help="layers of the stack (the workload has 36; fewer only for quick checks)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate wall time of each oracle baseline sample (all cores, one thread)")
    ap.add_argument("--procs", type=int, default=0,
                    help="threads drawing the seeded inputs (default: usable cores, at most 16)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches only")
    ap.add_argument("--no-workload1", action="store_true", help="skip the one-layer workload's extra keys")
    ap.add_argument("--no-batched", action="store_true",
                    help="skip the batched form (counter runs: only the per-layer launches)")
    ap.add_argument("--cold-reps", type=int, default=10,
                    help="rebuilds of the stack timed after an Infinity Cache flush")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run plain device copies of a known size (PMC calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--pmc-out", default=None,
                    help="with --summarize-pmc: output .json (default: the default workload's file)")
    ap.add_argument("--pmc-workload", default=None,
                    help="with --summarize-pmc: workload description stored in the summary")
    ap.add_argument("--sweep", action="store_true",
                    help="time the other workloads instead (one JSON line each): small fp32 layer, "
                         "one layer at tail 410, full prefill vs tails with the error bound, 16 varlen hits, "
                         "decode steps, FA-KV transfer overlap, layer-block replay, replay-vs-full at 8K/16K/32K")
    ap.add_argument("--only", default="",
                    help="with --sweep: comma list of sections to run "
                         "(small, layer410, accuracy, hits, decode, h2d, block, full)")
    ap.add_argument("--decode-seqs", default="1,64,256",
                    help="with --sweep: batch sizes of the decode lines")
    return ap.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(rel.encode() + b"\0" + f.read())
    return h.hexdigest()


def per_token_work(hk, hv, dk, dv, elt, outputs):
    """Algorithmic FLOPs and HBM bytes per token per value head (full 64-token tiles).

    FLOPs: K K^T shared by the Hv/Hk value heads of a key head, W = T diag K,
    U = T diag V, W M and K^T Delta; outputs add Q K^T, Q M and P Delta.
    Bytes: k (shared by the group), v, g and beta; outputs add q and o.
    """
    grp = hv // hk
    flops = 2 * CHUNK * dk / grp + 2 * CHUNK * dk + 2 * CHUNK * dv + 4 * dk * dv
    nbytes = elt * dk / grp + elt * dv + 8
    if outputs:
        flops += 2 * CHUNK * dk / grp + 2 * dk * dv + 2 * CHUNK * dv
        nbytes += elt * dk / grp + elt * dv
    return flops, nbytes


def quantiles(xs):
    xs = sorted(xs)
    pick = lambda q: xs[min(len(xs) - 1, int(round(q * (len(xs) - 1))))]
    return {"p10": pick(0.1), "p50": statistics.median(xs), "p90": pick(0.9)}


# ---------------------------------------------------------------- PMC summary
def _counter_rows(d):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no *counter_collection.csv under {d}")
    rows = []
    for fn in files:
        with open(fn) as f:
            rows += list(csv.DictReader(f))
    return rows


def _per_dispatch(rows, counter):
    """{(kernel name, grid size): [counter value per dispatch, KiB]}."""
    per = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        key = (r["Kernel_Name"], int(r.get("Grid_Size") or 0), r.get("Dispatch_Id") or r.get("Correlation_Id"))
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (name, grid, _), v in per.items():
        out.setdefault((name, grid), []).append(v)
    return out


def _per_kernel_mean(rows, counter):
    """Mean over dispatches of the counter, per kernel name (KiB per dispatch)."""
    out = {}
    for (name, _), v in _per_dispatch(rows, counter).items():
        out.setdefault(name, []).extend(v)
    return {name: statistics.fmean(v) for name, v in out.items()}


def _calibration(rows, counter):
    """The calibration copy's mean reading: dispatches of the elementwise `neg`
    kernel with the largest grid (other, smaller `neg` launches of the same
    process do not count)."""
    cands = {k: v for k, v in _per_dispatch(rows, counter).items() if "neg" in k[0] and "gdn" not in k[0]}
    if not cands:
        raise SystemExit(f"no calibration kernel in the {counter} run: rerun bench.py with --calib-copy")
    key = max(cands, key=lambda k: k[1])
    return key[0], statistics.fmean(cands[key])


def summarize_pmc(fetch_dir, write_dir, out_path=None, workload=None):
    frows, wrows = _counter_rows(fetch_dir), _counter_rows(write_dir)
    fetch = _per_kernel_mean(frows, "FETCH_SIZE")
    write = _per_kernel_mean(wrows, "WRITE_SIZE")
    # the calibration kernel reads and writes CALIB_BYTES
    cname, cal_fetch = _calibration(frows, "FETCH_SIZE")
    _, cal_write = _calibration(wrows, "WRITE_SIZE")
    f_fetch = CALIB_BYTES / (cal_fetch * 1024.0)
    f_write = CALIB_BYTES / (cal_write * 1024.0)
    kernels = {}
    for name in fetch:
        if not any(t in name for t in ("k_scan", "k_intra", "k_decode", "k_state_combine", "k_combine_intra")):
            continue
        short = name.split("(")[0].replace("void ", "")
        fb = fetch[name] * 1024.0 * f_fetch
        wb = write.get(name, 0.0) * 1024.0 * f_write
        kernels[short] = {"fetch_kib": fetch[name], "write_kib": write.get(name, 0.0),
                          "fetch_bytes": fb, "write_bytes": wb, "traffic_bytes": fb + wb}
    summary = {"workload": workload or WORKLOAD2_NAME,
               "source_sha256": kernel_source_hash(),
               "calibration": {"kernel": cname.split("(")[0], "bytes_each_way": CALIB_BYTES,
                               "fetch_kib": cal_fetch, "write_kib": cal_write,
                               "fetch_factor": f_fetch, "write_factor": f_write},
               "kernels": kernels,
               "commands": [
                   "cd /tmp && export TMPDIR=/tmp && timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE "
                   "--output-format csv -d $OUT/pmc_fetch -o fetch -- python3 $ROOT/bench.py "
                   "--no-cpu-baseline --no-graph --no-workload1 --steps 5 --warmup 2 --cold-reps 0 --calib-copy --no-batched",
                   "(same with WRITE_SIZE into $OUT/pmc_write)",
                   f"python bench.py --summarize-pmc $OUT/pmc_fetch $OUT/pmc_write"]}
    path = out_path or TRAFFIC_FILE
    with open(path, "w") as f:
        json.dump(summary, f, indent=1)
    print(json.dumps(summary, indent=1))
    return path


def load_traffic(kernel_short):
    """Calibrated HBM bytes per launch of `kernel_short` from the committed PMC
    summary, or None when there is none or the kernels changed since."""
    path = TRAFFIC_FILE
    if not os.path.exists(path):
        return None
    with open(path) as f:
        s = json.load(f)
    if s.get("source_sha256") != kernel_source_hash():
        return None
    k = s["kernels"].get(kernel_short)
    return None if k is None else k["traffic_bytes"]


# ---------------------------------------------------------------- inputs
WORKLOAD2_NAME = ("36-layer stack, one GDN layer each: Hk=16 Hv=32 d_k=d_v=128 bf16 q/k/v; prefix 32768, "
                  "tail replay r=3277 from zero + 1024-token suffix forward with outputs, per layer")


def usable_cores():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


# ---------------------------------------------------------------- main
def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.pmc_out, args.pmc_workload)
        return
    if args.sweep:
        sweep(args)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU and has no multi-GPU path: the (sequence, head) "
              "units are independent, so several GPUs would each take a share of them with "
              "no exchange; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np

    import synth
    from synth import workloads

    # ---- seeded inputs (drawn on a pool of threads)
    t_draw = time.perf_counter()
    shape, hits = workloads.workload2(args.layers)
    drawn = workloads.draw_hits(hits, shape, threads=args.procs)
    tails = synth.pack([t for t, _ in drawn])
    sufs = synth.pack([s for _, s in drawn])
    del drawn
    t_draw = time.perf_counter() - t_draw

    import torch

    import paper_2608_30310_amd as gdn

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    gdn.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def to_dev(p):
        def qkv(a):
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return dict(q=qkv(p.q), k=qkv(p.k), v=qkv(p.v), g=torch.from_numpy(p.g).to(dev),
                    beta=torch.from_numpy(p.beta).to(dev),
                    cu=torch.from_numpy(p.cu_seqlens).to(dev),
                    cu_host=torch.from_numpy(p.cu_seqlens.copy()))

    xt, xs = to_dev(tails), to_dev(sufs)
    L = args.layers
    hk, hv, dk, dv = shape.hk, shape.hv, shape.dk, shape.dv
    r, s = hits[0].r, hits[0].s
    # per-layer views of the packed inputs: each layer is its own one-sequence call
    cu_t1, cu_s1 = [0, r], [0, s]
    cu_t1_d = torch.tensor(cu_t1, dtype=torch.int32, device=dev)
    cu_s1_d = torch.tensor(cu_s1, dtype=torch.int32, device=dev)
    cu_t1_h = torch.tensor(cu_t1, dtype=torch.int32)
    cu_s1_h = torch.tensor(cu_s1, dtype=torch.int32)
    lt = [{n: xt[n][l * r:(l + 1) * r] for n in ("k", "v", "g", "beta")} for l in range(L)]
    ls = [{n: xs[n][l * s:(l + 1) * s] for n in ("q", "k", "v", "g", "beta")} for l in range(L)]
    mid = torch.empty((L, hv, dk, dv), dtype=torch.float32, device=dev)
    fin = torch.empty_like(mid)
    o = torch.empty((L * s, hv, dv), dtype=torch.bfloat16, device=dev)
    ws_t = torch.empty(gdn.workspace_size(1, hk, hv, dk, dv, cu_t1) + 256, dtype=torch.uint8, device=dev)
    ws_f = torch.empty(gdn.workspace_size(1, hk, hv, dk, dv, cu_s1, with_outputs=True) + 256,
                       dtype=torch.uint8, device=dev)
    ws_rf = torch.empty(gdn.replay_forward_workspace_size(1, hk, hv, dk, dv, cu_t1, cu_s1) + 256,
                        dtype=torch.uint8, device=dev)
    names_rf = gdn.replay_forward_stage_names()

    def replay_layer(l, ev=None):
        x = lt[l]
        gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], cu_t1_d, cu_t1_h, state_out=mid[l:l + 1],
                        workspace=ws_t, events=ev)

    def forward_layer(l, ev=None):
        x = ls[l]
        gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], cu_s1_d, cu_s1_h, state_in=mid[l:l + 1],
                          o=o[l * s:(l + 1) * s], state_out=fin[l:l + 1], workspace=ws_f, events=ev)

    def fused_layer(l, ev=None):
        a, b = lt[l], ls[l]
        gdn.replay_forward(a["k"], a["v"], a["g"], a["beta"], cu_t1_d, b["q"], b["k"], b["v"], b["g"], b["beta"],
                           cu_s1_d, cu_tail_host=cu_t1_h, cu_suf_host=cu_s1_h, state_mid=mid[l:l + 1],
                           o=o[l * s:(l + 1) * s], state_out=fin[l:l + 1], workspace=ws_rf, events=ev)

    def step(evs=None):
        for l in range(L):
            fused_layer(l, evs[l] if evs else None)

    def two_calls_step():
        for l in range(L):
            replay_layer(l)
            forward_layer(l)

    def rebuild():
        for l in range(L):
            replay_layer(l)

    # the layers as one batched call each (layers as the sequences of one launch)
    midb, finb = torch.empty_like(mid), torch.empty_like(fin)
    ob = torch.empty_like(o)
    ws_bt = torch.empty(gdn.workspace_size(L, hk, hv, dk, dv, tails.cu_seqlens.tolist()) + 256,
                        dtype=torch.uint8, device=dev)
    ws_bf = torch.empty(gdn.workspace_size(L, hk, hv, dk, dv, sufs.cu_seqlens.tolist(), with_outputs=True)
                        + 256, dtype=torch.uint8, device=dev)

    def batched_replay():
        gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"], state_out=midb,
                        workspace=ws_bt)

    def batched_step():
        batched_replay()
        gdn.chunk_forward(xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"], xs["cu_host"],
                          state_in=midb, o=ob, state_out=finb, workspace=ws_bf)

    # the layers as a hybrid model's groups (paper Section 3: one FA layer and
    # the GDN layers after it; each group replays on its own, from the cached
    # FA output hidden): GROUP_DEPTH GDN layers per group, so the layers of one
    # depth, one per group, run as the sequences of one fused call, and the
    # depths run in sequence (a layer's inputs come from the one before it)
    depth_calls = []
    for dd in range(min(GROUP_DEPTH, L)):
        lays = list(range(dd, L, GROUP_DEPTH))
        n = len(lays)
        tk = {nm: torch.cat([xt[nm][l * r:(l + 1) * r] for l in lays]) for nm in ("k", "v", "g", "beta")}
        sk = {nm: torch.cat([xs[nm][l * s:(l + 1) * s] for l in lays]) for nm in ("q", "k", "v", "g", "beta")}
        cut_l, cus_l = [r * i for i in range(n + 1)], [s * i for i in range(n + 1)]
        depth_calls.append(dict(
            lays=lays, t=tk, s=sk,
            cut=torch.tensor(cut_l, dtype=torch.int32, device=dev), cut_h=torch.tensor(cut_l, dtype=torch.int32),
            cus=torch.tensor(cus_l, dtype=torch.int32, device=dev), cus_h=torch.tensor(cus_l, dtype=torch.int32),
            mid=torch.empty((n, hv, dk, dv), dtype=torch.float32, device=dev),
            fin=torch.empty((n, hv, dk, dv), dtype=torch.float32, device=dev),
            o=torch.empty((n * s, hv, dv), dtype=torch.bfloat16, device=dev),
            ws=torch.empty(gdn.replay_forward_workspace_size(n, hk, hv, dk, dv, cut_l, cus_l) + 256,
                           dtype=torch.uint8, device=dev),
            ws_t=torch.empty(gdn.workspace_size(n, hk, hv, dk, dv, cut_l) + 256, dtype=torch.uint8, device=dev)))

    def grouped_step():
        for c in depth_calls:
            a, b = c["t"], c["s"]
            gdn.replay_forward(a["k"], a["v"], a["g"], a["beta"], c["cut"], b["q"], b["k"], b["v"], b["g"],
                               b["beta"], c["cus"], cu_tail_host=c["cut_h"], cu_suf_host=c["cus_h"],
                               state_mid=c["mid"], o=c["o"], state_out=c["fin"], workspace=c["ws"])

    def grouped_replay():
        for c in depth_calls:
            a = c["t"]
            gdn.tail_replay(a["k"], a["v"], a["g"], a["beta"], c["cut"], c["cut_h"], state_out=c["mid"],
                            workspace=c["ws_t"])

    for _ in range(args.warmup):
        step()
        grouped_step()
        if not args.no_batched:
            batched_step()
    torch.cuda.synchronize()
    K = args.steps

    def timed(fn, reps=K):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for _ in range(reps):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / reps

    # ---- graph of one step, checked bitwise against the eager step on several replays
    graph, graph_note = None, None
    step()
    torch.cuda.synchronize()
    want = (mid.clone(), fin.clone(), o.clone())
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        ok = True
        for _ in range(3):
            for t in (mid, fin, o):
                t.zero_()
            g.replay()
            torch.cuda.synchronize()
            ok = ok and torch.equal(mid, want[0]) and torch.equal(fin, want[1]) and torch.equal(o, want[2])
            step()               # eager work between replays
            torch.cuda.synchronize()
        if ok:
            graph = g
        else:
            graph_note = "graph replay differed from the eager step; graph not timed"
    # the two calls give the fused call's results bit for bit; the batched
    # form the same states up to rounding order
    two_calls_step()
    torch.cuda.synchronize()
    two_calls_equal = bool(torch.equal(mid, want[0]) and torch.equal(fin, want[1]) and torch.equal(o, want[2]))
    bdiff = None
    if not args.no_batched:
        batched_step()
        torch.cuda.synchronize()
        bdiff = [float(((x - w).norm() / w.norm()).item()) for x, w in ((midb, want[0]), (finb, want[1]))]
    grouped_step()
    torch.cuda.synchronize()
    mid_g, fin_g = torch.empty_like(mid), torch.empty_like(fin)
    for c in depth_calls:
        mid_g[c["lays"]] = c["mid"]
        fin_g[c["lays"]] = c["fin"]
    gdiff = [float(((x - w).norm() / w.norm()).item()) for x, w in ((mid_g, want[0]), (fin_g, want[1]))]
    del mid_g, fin_g

    ms_per_step = timed(step)
    ms_graph = timed(graph.replay) if graph is not None else None
    ms_two_calls = timed(two_calls_step)
    ms_batched = None if args.no_batched else timed(batched_step)
    ms_batched_rebuild = None if args.no_batched else timed(batched_replay)
    ms_grouped = timed(grouped_step)
    ms_grouped_rebuild = timed(grouped_replay)

    # ---- per-stage kernel durations: events recorded by the library on its stream
    n_ev = min(K, 20)

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    evs = [[new_events(len(names_rf) + 1) for _ in range(L)] for _ in range(n_ev)]
    torch.cuda.synchronize()
    for i in range(n_ev):
        step(evs[i])
    torch.cuda.synchronize()
    stages = {}
    for j, nm in enumerate(names_rf):
        d = [evs[i][l][j].elapsed_time(evs[i][l][j + 1]) * 1e3 for i in range(n_ev) for l in range(L)]
        stages["replay_forward." + nm] = {"mean_us": statistics.fmean(d), "median_us": statistics.median(d),
                                          "per_step_us": statistics.fmean(d) * L}

    # ---- rebuild latency of the stack (the 36 replays): warm (from an idle
    #      stream), queued (a spin kernel holds the GPU while the host enqueues,
    #      so the interval is the device's alone) and cold (Infinity Cache
    #      flushed before each rep)
    def latency(fn, reps, before=None, spin=False):
        lat = []
        for i in range(reps):
            if before:
                before(i)
            if spin:
                torch.cuda._sleep(QUEUE_SPIN_CYCLES * max(1, L // 4))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            lat.append(a.elapsed_time(b) * 1e3)
        return quantiles(lat)

    warm = latency(rebuild, min(K, 20))
    queued_rebuild = latency(rebuild, min(K, 20), spin=True)
    cold = None
    if args.cold_reps > 0:
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
        cold = latency(rebuild, args.cold_reps, before=lambda i: flush.fill_(float(i)))
        del flush

    if args.calib_copy:
        # a plain elementwise kernel that reads and writes CALIB_BYTES once each
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ---- algorithmic work (SURVEY-style per-token counts, full 64-token tiles)
    elt = 2
    ft, bt = per_token_work(hk, hv, dk, dv, elt, outputs=False)
    ff, bf = per_token_work(hk, hv, dk, dv, elt, outputs=True)
    state_bytes = hv * dk * dv * 4          # one layer's states
    tail_flops, tail_bytes = r * hv * ft, r * hv * bt + state_bytes
    fwd_flops, fwd_bytes = s * hv * ff, s * hv * bf + 2 * state_bytes
    path_flops, path_bytes = L * (tail_flops + fwd_flops), L * (tail_bytes + fwd_bytes)
    t_s = ms_per_step * 1e-3
    path_bound_s = max(path_flops / (BF16_PEAK_TFLOPS * 1e12), path_bytes / (HBM_PEAK_GBS * 1e9))

    # dominant kernel: the stage with the most time per step; its algorithmic
    # bytes are those of the part of the path it runs, per launch (one layer)
    dom = max(stages, key=lambda k: stages[k]["per_step_us"])
    grp = hv // hk
    split = stages["replay_forward.combine (+ suffix intra)"]["mean_us"] > 0.5
    # the suffix's chunk preparation reads q, k (shared by the group), g and
    # beta and forms K K^T and Q K^T per chunk; the combine reads the
    # transition, the second half's state and the first half's, and writes
    # the state
    prep_bytes = s * hv * (2 * elt * dk / grp + 8)
    prep_flops = s * hv * (2 * 2 * CHUNK * dk / grp)
    comb_bytes, comb_flops = 3 * state_bytes + hv * dk * dk * 4, 2 * hv * dk * dk * dv
    kinfo = {
        "replay_forward.tail intra": ("gdn::k_intra<unsigned short, 128, false>",
                                      r * hv * (elt * dk / grp + 8), r * hv * 2 * CHUNK * dk / grp),
        "replay_forward.tail scan (+ suffix intra)":
            ("gdn::k_scan_cols_split<unsigned short, 128>", tail_bytes, tail_flops) if split else
            ("gdn::k_scan_cols_intra<unsigned short, 128>", tail_bytes + prep_bytes, tail_flops + prep_flops),
        "replay_forward.combine (+ suffix intra)": ("gdn::k_combine_intra<unsigned short, 128>",
                                                    comb_bytes + prep_bytes, comb_flops + prep_flops),
        "replay_forward.suffix scan": ("gdn::k_scan_cols<unsigned short, 128, true>", fwd_bytes, fwd_flops),
    }
    kname, kbytes, kflops = kinfo[dom]
    dom_s = stages[dom]["mean_us"] * 1e-6
    achieved = kbytes / dom_s / 1e9
    roofline = {"kernel": kname, "stage": dom, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": load_traffic(kname.split("(")[0]),
                "algorithmic_bytes_per_launch": kbytes, "algorithmic_flops_per_launch": kflops,
                "launch_us": stages[dom]["mean_us"],
                "mfma_frac": kflops / dom_s / (BF16_PEAK_TFLOPS * 1e12)}

    tokens = L * (r + s)
    result = {
        "metric": METRIC,
        "value": tokens / t_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded per 64-token block; see synth/)",
        "config": {"workload": WORKLOAD2_NAME if L == 36 else f"{L}-layer stack (reduced), shapes as the "
                                                              f"36-layer workload",
                   "layers": L, "prefix": hits[0].m, "tail": r, "suffix": s,
                   "global_batch": L, "seq_len": r + s, "parallelism": "single GPU"},
        "launch": "eager; per layer one gdn_replay_forward call (tail replay, then the suffix forward from "
                  "the rebuilt state), layers in sequence",
        "ms_per_step_graph": ms_graph,
        "ms_per_step_two_calls": ms_two_calls,
        "two_calls_bitwise_equal": two_calls_equal,
        "ms_per_step_batched": ms_batched,
        # relative Frobenius differences of the rebuilt (tail) states and the
        # final states: the forms differ in rounding order only (the final
        # states agree once the suffix's decay has erased the difference)
        "batched_vs_sequential_rel_state_diff": None if bdiff is None else {"tail": bdiff[0], "final": bdiff[1]},
        "ms_per_step_grouped": ms_grouped,
        "grouped": f"{len(depth_calls[0]['lays'])} groups of {GROUP_DEPTH} layers: one fused call per depth, "
                   "the depth's layers as its sequences",
        "grouped_vs_sequential_rel_state_diff": {"tail": gdiff[0], "final": gdiff[1]},
        "rebuild_latency_us": warm["p50"],
        "rebuild_latency_warm_us": warm,
        "rebuild_latency_cold_us": cold,
        "rebuild_latency_queued_us": queued_rebuild,
        "rebuild_latency_batched_us": None if ms_batched_rebuild is None else ms_batched_rebuild * 1e3,
        "rebuild_latency_grouped_us": ms_grouped_rebuild * 1e3,
        "replay_tokens_per_s": L * r / (warm["p50"] * 1e-6),
        "replay_tokens_per_s_batched": None if ms_batched_rebuild is None else L * r / (ms_batched_rebuild * 1e-3),
        "stages": stages,
        "path": {"flops": path_flops, "bytes": path_bytes, "roofline_us": path_bound_s * 1e6,
                 "roofline_frac": path_bound_s / t_s,
                 "mfma_frac": path_flops / t_s / (BF16_PEAK_TFLOPS * 1e12)},
        "roofline": roofline,
        "cpu_baseline": None,
        "input_draw_s": t_draw,
        "gpu": torch.cuda.get_device_name(dev),
    }
    if graph_note:
        result["note"] = graph_note
    if not args.no_workload1:
        result["workload1"] = workload1_line(args, gdn, torch, dev)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(tails, sufs, r, s, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def workload1_line(args, gdn, torch, dev):
    """The one-layer workload (tail 819 + suffix 512) as extra keys: the fused
    call, the two calls, and the rebuild latency."""
    import numpy as np

    import synth
    from synth import workloads
    shape, hits = workloads.workload1(819)
    h = hits[0]
    tail, suf = synth.pack([h.tail(shape)]), synth.pack([h.suffix(shape)])

    def to_dev(p):
        qkv = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return dict(q=qkv(p.q), k=qkv(p.k), v=qkv(p.v), g=torch.from_numpy(p.g).to(dev),
                    beta=torch.from_numpy(p.beta).to(dev), cu=torch.from_numpy(p.cu_seqlens).to(dev),
                    cu_host=torch.from_numpy(p.cu_seqlens.copy()))

    xt, xs = to_dev(tail), to_dev(suf)
    hv, dk, dv = shape.hv, shape.dk, shape.dv
    st = torch.empty((1, hv, dk, dv), dtype=torch.float32, device=dev)
    st2 = torch.empty_like(st)
    o = torch.empty((h.s, hv, dv), dtype=torch.bfloat16, device=dev)

    def fused():
        gdn.replay_forward(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xs["q"], xs["k"], xs["v"],
                           xs["g"], xs["beta"], xs["cu"], cu_tail_host=xt["cu_host"],
                           cu_suf_host=xs["cu_host"], state_mid=st, o=o, state_out=st2)

    def replay():
        gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"], state_out=st)

    def two():
        replay()
        gdn.chunk_forward(xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"], xs["cu_host"],
                          state_in=st, o=o, state_out=st2)

    for _ in range(5):
        fused()
        two()
    torch.cuda.synchronize()

    def timed(fn, reps=args.steps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    def lat(fn, reps=20):
        xs_ = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            xs_.append(a.elapsed_time(b) * 1e3)
        return quantiles(xs_)

    ms_fused = timed(fused)
    return {"workload": "one GDN layer Hk=16 Hv=32 d=128 bf16: prefix 8192, tail 819 + suffix 512",
            "ms_per_step_fused": ms_fused, "ms_per_step_two_calls": timed(two),
            "tokens_per_s_fused": (h.r + h.s) / (ms_fused * 1e-3),
            "rebuild_latency_us": lat(replay)}


# ---------------------------------------------------------------- other workloads
def sweep(args):
    """Latency of the other workloads; one JSON line each.  Inputs of the small
    layer and of the varlen hits are the seeded ones the parity tests use; the
    36-layer stack and the replay-vs-full sweep use device-drawn inputs of the
    same distributions (timing only: the kernels' time does not depend on the
    values)."""
    import numpy as np
    import torch

    import paper_2608_30310_amd as gdn
    import synth
    from paper_2608_30310_amd import transfer
    from synth import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    gdn.load_library()
    reps, warm = max(args.steps // 2, 10), 5

    def timed_us(fn, queued=False):
        # queued: the rep's launches wait behind a spin kernel, so the interval
        # is the device's time alone (kernels and the gaps between them), not
        # the host's pacing; otherwise each rep starts from an idle stream and
        # includes the host's launch latency
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            if queued:
                torch.cuda._sleep(QUEUE_SPIN_CYCLES)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        return quantiles(ts)

    def packed_dev(p, shape):
        if shape.dtype == "bf16":
            qkv = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        else:
            qkv = lambda a: torch.from_numpy(a).to(dev)
        return dict(q=qkv(p.q), k=qkv(p.k), v=qkv(p.v), g=torch.from_numpy(p.g).to(dev),
                    beta=torch.from_numpy(p.beta).to(dev), cu=torch.from_numpy(p.cu_seqlens).to(dev),
                    cu_host=torch.from_numpy(p.cu_seqlens.copy()))

    def random_dev(lens, hk, hv, d, gate_scale=0.1, seed=0):
        """Device-drawn inputs with the workload distributions (timing only)."""
        gen = torch.Generator(device=dev).manual_seed(seed)
        T = int(sum(lens))
        nrm = lambda x: (x / x.norm(dim=-1, keepdim=True)).to(torch.bfloat16)
        q = nrm(torch.randn(T, hk, d, device=dev, generator=gen))
        k = nrm(torch.randn(T, hk, d, device=dev, generator=gen))
        v = torch.randn(T, hv, d, device=dev, generator=gen).to(torch.bfloat16)
        beta = torch.sigmoid(torch.randn(T, hv, device=dev, generator=gen))
        g = -torch.nn.functional.softplus(torch.randn(T, hv, device=dev, generator=gen)) * gate_scale
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        return dict(q=q, k=k, v=v, g=g.contiguous(), beta=beta.contiguous(),
                    cu=torch.from_numpy(cu).to(dev), cu_host=torch.from_numpy(cu))

    def replay(x, state, ws):
        gdn.tail_replay(x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"], state_out=state,
                        workspace=ws)

    def forward(x, state_in, o, state_out, ws, write_state=True):
        gdn.chunk_forward(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["cu_host"],
                          state_in=state_in, o=o, state_out=state_out, workspace=ws,
                          write_state=write_state)

    def fused(xt, xs, st, o, st2, ws):
        gdn.replay_forward(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xs["q"], xs["k"], xs["v"],
                           xs["g"], xs["beta"], xs["cu"], cu_tail_host=xt["cu_host"],
                           cu_suf_host=xs["cu_host"], state_mid=st, o=o, state_out=st2, workspace=ws)

    def fused_ws(xt, xs, n, hk, hv, d):
        return torch.empty(gdn.replay_forward_workspace_size(n, hk, hv, d, d, xt["cu_host"].tolist(),
                                                             xs["cu_host"].tolist(), dtype=xt["k"].dtype)
                           + 256, dtype=torch.uint8, device=dev)

    def buffers(x, n, hk, hv, d, outputs):
        cu = x["cu_host"].tolist()
        ws = torch.empty(gdn.workspace_size(n, hk, hv, d, d, cu, dtype=x["k"].dtype,
                                            with_outputs=outputs) + 256,
                         dtype=torch.uint8, device=dev)
        st = torch.empty((n, hv, d, d), dtype=torch.float32, device=dev)
        o = torch.empty((cu[-1], hv, d), dtype=x["v"].dtype, device=dev) if outputs else None
        return ws, st, o

    def emit(rec):
        print(json.dumps(rec), flush=True)

    want = lambda name: not args.only or name in args.only.split(",")

    def oracle_time(tail, suf, seconds=args.cpu_seconds):
        """The fp64 oracle on the host cores on a workload's own inputs: the
        tail replay then the suffix forward from its state, all heads, on every
        usable core; then on one thread over the value heads of the first key
        head only (bounded wall time).  Rates in (token, value head) pairs per
        second, so the two are comparable; the all-core run also as tokens/s."""
        import oracle

        def run(p_t, p_s, threads):
            n, t0 = 0, time.perf_counter()
            while True:
                et, es = p_t.exact(), p_s.exact()
                _, st = oracle.recurrence(et["k"], et["v"], et["g"], et["beta"], et["cu_seqlens"], nthreads=threads)
                if p_s.num_tokens:
                    oracle.recurrence(es["k"], es["v"], es["g"], es["beta"], es["cu_seqlens"], q=es["q"],
                                      state_in=st, nthreads=threads)
                n += 1
                el = time.perf_counter() - t0
                if el >= seconds / 2 or n >= 50:
                    return n, el

        def first_group(p):
            import dataclasses
            grp = p.shape.hv // p.shape.hk
            shp = dataclasses.replace(p.shape, hk=1, hv=grp)
            return synth.Packed(shp, p.q[:, :1].copy(), p.k[:, :1].copy(), p.v[:, :grp].copy(),
                                p.g[:, :grp].copy(), p.beta[:, :grp].copy(), p.cu_seqlens)

        tokens = tail.num_tokens + suf.num_tokens
        cores = min(usable_cores(), oracle.max_threads())
        n_all, el_all = run(tail, suf, cores)
        t1, s1 = first_group(tail), first_group(suf)
        n_one, el_one = run(t1, s1, 1)
        return {"kind": "oracle", "cpu_model": cpu_model(),
                "all_cores": {"cores": cores, "tokens_per_s": n_all * tokens / el_all,
                              "head_tokens_per_s": n_all * tokens * tail.shape.hv / el_all,
                              "sample": f"{n_all} run(s) of every head in {el_all:.2f} s"},
                "one_thread": {"cores": 1, "head_tokens_per_s": n_one * tokens * t1.shape.hv / el_one,
                               "sample": f"{n_one} run(s) of the {t1.shape.hv} value heads of key head 0 "
                                         f"in {el_one:.2f} s"}}

    # ---- small fp32 layer (Hk = Hv = 4, d = 64): tail 205 + suffix 256
    if want("small"):
        shape, hits = workloads.workload0()
        h = hits[0]
        xt, xs = packed_dev(synth.pack([h.tail(shape)]), shape), packed_dev(synth.pack([h.suffix(shape)]), shape)
        wst, st, _ = buffers(xt, 1, 4, 4, 64, False)
        wsf, st2, o = buffers(xs, 1, 4, 4, 64, True)
        wsr = fused_ws(xt, xs, 1, 4, 4, 64)
        rep = timed_us(lambda: replay(xt, st, wst))
        repq = timed_us(lambda: replay(xt, st, wst), queued=True)
        two = timed_us(lambda: (replay(xt, st, wst), forward(xs, st, o, st2, wsf)))
        both = timed_us(lambda: fused(xt, xs, st, o, st2, wsr))
        emit({"workload": "small fp32 layer Hk=Hv=4 d=64: tail 205 + suffix 256",
              "rebuild_latency_us": rep, "rebuild_latency_queued_us": repq,
              "step_us": both, "step_two_calls_us": two,
              "tokens_per_s": (205 + 256) / (both["p50"] * 1e-6),
              "cpu_oracle": oracle_time(synth.pack([h.tail(shape)]), synth.pack([h.suffix(shape)]))})

    # ---- hybrid-model layer, tail 410 (the default bench line covers 819)
    if want("layer410"):
        shape, hits = workloads.workload1(410)
        h = hits[0]
        xt, xs = packed_dev(synth.pack([h.tail(shape)]), shape), packed_dev(synth.pack([h.suffix(shape)]), shape)
        wst, st, _ = buffers(xt, 1, 16, 32, 128, False)
        wsf, st2, o = buffers(xs, 1, 16, 32, 128, True)
        wsr = fused_ws(xt, xs, 1, 16, 32, 128)
        rep = timed_us(lambda: replay(xt, st, wst))
        repq = timed_us(lambda: replay(xt, st, wst), queued=True)
        two = timed_us(lambda: (replay(xt, st, wst), forward(xs, st, o, st2, wsf)))
        both = timed_us(lambda: fused(xt, xs, st, o, st2, wsr))
        emit({"workload": "one GDN layer Hk=16 Hv=32 d=128 bf16: tail 410 + suffix 512",
              "rebuild_latency_us": rep, "rebuild_latency_queued_us": repq,
              "step_us": both, "step_two_calls_us": two,
              "tokens_per_s": (410 + 512) / (both["p50"] * 1e-6)})

    # ---- full prefill against tail replay, one layer, m = 32768 (seeded
    #      inputs of that workload): for every replay length r and gate scale,
    #      the tail state's relative distance from the full-prefill state next
    #      to the bound ||S_head||_F prod(alpha) / ||S_full||_F (S_head = the
    #      full-prefill state at m - r; prod(alpha) = exp(sum of g over the
    #      tail)), maxima over the 32 value heads, log10 of the bound, and the
    #      time ratio of the full forward (with outputs) to the tail replay; plus
    #      the fp64 oracle's time on the full prefix (all cores; one thread over
    #      the two value heads of key head 0)
    if want("accuracy"):
        for gs in workloads.WORKLOAD4_GATE_SCALES:
            shape, hit = workloads.workload4(3277, gs)
            full = synth.pack([hit.prefix(shape)])
            xf = packed_dev(full, shape)
            wsF, stF, oF = buffers(xf, 1, 16, 32, 128, True)
            t_full = timed_us(lambda: forward(xf, None, oF, stF, wsF), queued=True)
            s_full = stF.double().cpu().numpy()[0]
            g_all = full.g.astype(np.float64)
            cells = []
            for r in workloads.WORKLOAD4_TAILS:
                m = hit.m
                # the tail's inputs are rows [m - r, m) of the full prefix
                xt = {n: xf[n][m - r:] for n in ("k", "v", "g", "beta")}
                xt["cu"] = torch.tensor([0, r], dtype=torch.int32, device=dev)
                xt["cu_host"] = torch.tensor([0, r], dtype=torch.int32)
                xh = {n: xf[n][:m - r] for n in ("k", "v", "g", "beta")}
                xh["cu"] = torch.tensor([0, m - r], dtype=torch.int32, device=dev)
                xh["cu_host"] = torch.tensor([0, m - r], dtype=torch.int32)
                wst, st, _ = buffers(xt, 1, 16, 32, 128, False)
                wsh, sth, _ = buffers(xh, 1, 16, 32, 128, False)
                t_rep = timed_us(lambda: replay(xt, st, wst), queued=True)
                replay(xh, sth, wsh)
                torch.cuda.synchronize()
                s_tail = st.double().cpu().numpy()[0]
                s_head = sth.double().cpu().numpy()[0]
                log_prod = g_all[m - r:].sum(axis=0) / np.log(10.0)       # per head, log10 prod(alpha)
                n_full = np.linalg.norm(s_full.reshape(32, -1), axis=1)
                rel = np.linalg.norm((s_full - s_tail).reshape(32, -1), axis=1) / n_full
                n_head = np.linalg.norm(s_head.reshape(32, -1), axis=1)
                with np.errstate(divide="ignore"):
                    log_bound = np.log10(n_head / n_full) + log_prod
                cells.append({"r": r, "rel_err_max": float(rel.max()), "rel_err_median": float(np.median(rel)),
                              "log10_bound_max": float(log_bound.max()),
                              "log10_prod_alpha_mean": float(log_prod.mean()),
                              "bound_holds_all_heads": bool(np.all(rel <= 10.0 ** log_bound + 4e-3)),
                              "t_replay_us": t_rep["p50"], "time_ratio_full_over_replay": t_full["p50"] / t_rep["p50"]})
            emit({"workload": f"full 32768-token prefill vs tail replay, one layer Hk=16 Hv=32 d=128 bf16, "
                              f"gate scale {gs}",
                  "t_full_forward_us": t_full["p50"], "cells": cells,
                  "cpu_oracle_full_prefix": oracle_time(full, synth.pack([], shape))})
            del xf, oF

    # ---- 16 concurrent hits (varlen), one replay launch + one forward launch
    if want("hits"):
        draw = workloads.workload3_draw()
        rl = [gdn.replay_len(m, ratio) for m, ratio, _ in draw]
        shape, hits = workloads.workload3(rl)
        xt = packed_dev(synth.pack([h.tail(shape) for h in hits]), shape)
        xs = packed_dev(synth.pack([h.suffix(shape) for h in hits]), shape)
        n = len(hits)
        wst, st, _ = buffers(xt, n, 16, 32, 128, False)
        wsf, st2, o = buffers(xs, n, 16, 32, 128, True)
        wsr = fused_ws(xt, xs, n, 16, 32, 128)
        rep = timed_us(lambda: replay(xt, st, wst))
        repq = timed_us(lambda: replay(xt, st, wst), queued=True)
        two = timed_us(lambda: (replay(xt, st, wst), forward(xs, st, o, st2, wsf)))
        both = timed_us(lambda: fused(xt, xs, st, o, st2, wsr))
        sr, ss = sum(h.r for h in hits), sum(h.s for h in hits)
        emit({"workload": f"16 varlen hits Hk=16 Hv=32 d=128 bf16: sum r={sr}, sum s={ss}",
              "rebuild_latency_us": rep, "rebuild_latency_queued_us": repq,
              "step_us": both, "step_two_calls_us": two,
              "tokens_per_s": (sr + ss) / (both["p50"] * 1e-6),
              "replay_tokens_per_s": sr / (rep["p50"] * 1e-6),
              "cpu_oracle": oracle_time(synth.pack([h.tail(shape) for h in hits]),
                                        synth.pack([h.suffix(shape) for h in hits]))})

    # ---- decode steps after the rebuild: one token per sequence from the state,
    #      state updated in place; HBM-bound (the state is read and written once,
    #      with streaming loads and stores).  Timed as a HIP graph of 20 launches
    #      (no host overhead per step); the 1-sequence line is the first token's
    #      latency after a hit, the others are batched decode throughput.
    if want("decode"):
        if args.calib_copy:
            # the PMC calibration kernel, as in the default run
            src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            for _ in range(3):
                torch.neg(src, out=dst)
            torch.cuda.synchronize()
            del src, dst
        for nb in (int(x) for x in args.decode_seqs.split(",")):
            xd = random_dev([1] * nb, 16, 32, 128, seed=900 + nb)
            sd = torch.randn((nb, 32, 128, 128), dtype=torch.float32, device=dev) * 0.1
            od = torch.empty((nb, 32, 128), dtype=torch.bfloat16, device=dev)
            calls = 20
            dec = lambda: [gdn.decode_step(xd["q"], xd["k"], xd["v"], xd["g"], xd["beta"], state_in=sd,
                                           state_out=sd, o=od, scale=128 ** -0.5) for _ in range(calls)]
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                dec()
            torch.cuda.current_stream().wait_stream(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                dec()
            t = timed_us(graph.replay)
            per = t["p50"] / calls
            nbytes = (2 * nb * 32 * 128 * 128 * 4 + 2 * nb * 16 * 128 * 2 + 2 * nb * 32 * 128 * 2
                      + 2 * nb * 32 * 4)
            emit({"workload": f"decode step Hk=16 Hv=32 d=128 bf16, {nb} sequences, state in place",
                  "us_per_step": per, "tokens_per_s": nb / (per * 1e-6),
                  "gbs": nbytes / (per * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (per * 1e-6) / 1e9 / HBM_PEAK_GBS,
                  "note": f"graph of {calls} launches per timed rep"})

    # ---- FA-KV transfer overlapped with the replay (paper Section 3, "Replay
    #      efficiency"): a hit of m tokens moves the full-attention KV of the
    #      matched prefix from pinned host memory while the linear-attention
    #      layers replay their tails; the transfer joins the compute stream only
    #      before the suffix forward.  Synthetic sizes: 24 GDN layers
    #      (Hk=16, Hv=32, d=128) and 32 KiB of FA KV per token (8 FA layers x
    #      K, V x 4 KV heads x 256 x bf16).  H2D-SER: copy, replays, forwards on
    #      one stream; H2D-OVL: copy on a second stream beside the replays.
    if want("h2d"):
        n_la, kv_per_token = 24, 32 << 10
        copy_stream = torch.cuda.Stream()
        for m in (8192, 32768):
            r = {8192: 819, 32768: 3277}[m]
            host_kv = torch.empty(m * kv_per_token, dtype=torch.uint8, pin_memory=True)
            dev_kv = torch.empty(m * kv_per_token, dtype=torch.uint8, device=dev)
            xl = [random_dev([r], 16, 32, 128, seed=2000 + l) for l in range(n_la)]
            xq = [random_dev([512], 16, 32, 128, seed=3000 + l) for l in range(n_la)]
            wst, st, _ = buffers(xl[0], 1, 16, 32, 128, False)
            wsf, st2, o = buffers(xq[0], 1, 16, 32, 128, True)

            def replays():
                for x in xl:
                    replay(x, st, wst)

            def forwards():
                for x in xq:
                    forward(x, st, o, st2, wsf)

            def h2d():
                dev_kv.copy_(host_kv, non_blocking=True)

            def serial():
                transfer.rebuild_serial(host_kv, dev_kv, replays, forwards)

            def overlapped():
                transfer.rebuild_overlapped(host_kv, dev_kv, replays, forwards, copy_stream)

            t_h2d = timed_us(h2d)
            t_rep = timed_us(replays)
            t_fwd = timed_us(forwards)
            t_ser = timed_us(serial)
            t_ovl = timed_us(overlapped)
            hidden = (t_ser["p50"] - t_ovl["p50"]) / min(t_h2d["p50"], t_rep["p50"])
            emit({"workload": f"FA-KV H2D overlapped with replay, m={m}, r={r}, {n_la} GDN layers, "
                              f"{m * kv_per_token >> 20} MiB FA KV, suffix 512",
                  "h2d_us": t_h2d["p50"], "h2d_gbs": m * kv_per_token / (t_h2d["p50"] * 1e-6) / 1e9,
                  "replay_us": t_rep["p50"], "suffix_forward_us": t_fwd["p50"],
                  "h2d_ser_us": t_ser["p50"], "h2d_ovl_us": t_ovl["p50"],
                  "ovl_vs_ser_reduction": 1 - t_ovl["p50"] / t_ser["p50"],
                  "hidden_fraction_of_shorter": hidden})
            del host_kv, dev_kv, xl, xq

    # ---- the whole linear-attention layer replayed from the cached hiddens
    #      (in-projection, conv, norms, gates, recurrence, gated norm,
    #      out-projection) at D = 2048, Hk = 16, Hv = 32, d = 128; weights and
    #      hiddens drawn on the device with the layer recipe's ranges (timing
    #      only).  "outputs": a layer whose output feeds the next layer of the
    #      group; "state only": the group's last layer (no q, z or output path,
    #      no feed-forward block).  "us": an eager call; "us_graph" (and
    #      tokens_per_s): the call replayed from a HIP graph, without host
    #      overhead.  Per-stage times from the library's stage events; the
    #      projections are priced against the bf16 MFMA peak.
    if want("block"):
        D, hk, hv, d = 2048, 16, 32, 128
        cq, cv = hk * d, hv * d
        gen = torch.Generator(device=dev).manual_seed(77)

        def dev_weights():
            rn = lambda *s: torch.randn(*s, device=dev, generator=gen)
            return dict(w_in=(rn(2 * cq + 2 * cv + 2 * hv, D) / D ** 0.5).to(torch.bfloat16),
                        conv_w=(torch.rand(2 * cq + cv, 4, device=dev, generator=gen) - 0.5),
                        a_log=torch.log(1 + 15 * torch.rand(hv, device=dev, generator=gen)),
                        dt_bias=torch.full((hv,), -4.0, device=dev),
                        norm_w=0.5 + torch.rand(d, device=dev, generator=gen),
                        w_out=(rn(D, cv) / cv ** 0.5).to(torch.bfloat16))

        wts = dev_weights()

        def block_line(lens, outputs, act, label):
            T = int(sum(lens))
            cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
            cu_d, cu_h = torch.from_numpy(cu).to(dev), torch.from_numpy(cu)
            x = torch.randn(T, D, device=dev, generator=gen).to(torch.bfloat16)
            st = torch.empty((len(lens), hv, d, d), dtype=torch.float32, device=dev)
            out = torch.empty((T, D), dtype=torch.bfloat16, device=dev) if outputs else None
            ws = torch.empty(gdn.la_block_workspace_size(D, hk, hv, d, d, cu.tolist(), outputs, act) + 256,
                             dtype=torch.uint8, device=dev)
            call = lambda ev=None: gdn.la_block_replay(x, wts, cu_d, hk, hv, d, d, d ** -0.5, cu_seqlens_host=cu_h,
                                                       outputs=outputs, act_dtype=act, state_out=st, out=out,
                                                       workspace=ws, events=ev)
            t = timed_us(call)
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                call()
            torch.cuda.current_stream().wait_stream(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                call()
            t_graph = timed_us(graph.replay)
            names = gdn.la_block_stage_names(outputs)
            per = {n: [] for n in names}
            for _ in range(reps):
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
                call(ev)
                torch.cuda.synchronize()
                for i, n in enumerate(names):
                    per[n].append(ev[i].elapsed_time(ev[i + 1]) * 1e3)
            stages = {n: float(np.median(v)) for n, v in per.items()}
            rows = 2 * cq + 2 * cv + 2 * hv if outputs else cq + cv + 2 * hv
            fl_in = 2.0 * T * D * rows
            rec = {"workload": f"LA layer replay D={D} Hk={hk} Hv={hv} d={d}, {label}, "
                               f"{'outputs' if outputs else 'state only'}, {act} intermediates",
                   "tokens": T, "us": t["p50"], "us_graph": t_graph["p50"],
                   "tokens_per_s": T / (t_graph["p50"] * 1e-6),
                   "stage_us": stages,
                   "in_proj_tflops": fl_in / (stages["in-projection"] * 1e-6) / 1e12,
                   "in_proj_frac_of_bf16_peak": fl_in / (stages["in-projection"] * 1e-6) / 1e12 / BF16_PEAK_TFLOPS}
            if outputs:
                fl_out = 2.0 * T * cv * D
                rec["out_proj_tflops"] = fl_out / (stages["out-projection"] * 1e-6) / 1e12
            emit(rec)
            return t["p50"]

        for act in ("f32", "bf16"):
            for lens, label in (([819], "tail 819 (10% of 8192)"), ([3277], "tail 3277 (10% of 32768)")):
                block_line(lens, True, act, label)
                block_line(lens, False, act, label)

    # ---- replay vs full prefill, suffix 512: t_full = forward(0, m + s) with
    #      outputs; t_replay = the fused replay(r) + forward(S_m, s); state-only
    #      full = replay(m + s)
    if want("full"):
        for m in (8192, 16384, 32768):
            x_full = random_dev([m + 512], 16, 32, 128, seed=m)
            wsF, stF, oF = buffers(x_full, 1, 16, 32, 128, True)
            wsR, stR, _ = buffers(x_full, 1, 16, 32, 128, False)
            t_full = timed_us(lambda: forward(x_full, None, oF, stF, wsF))
            t_state = timed_us(lambda: replay(x_full, stR, wsR))
            for pct in ("0.05", "0.1"):
                # the configs' integers where they round to nearest, else the paper's ceiling
                r = {(8192, "0.1"): 819, (32768, "0.05"): 1638}.get((m, pct), gdn.replay_len(m, pct))
                xt = random_dev([r], 16, 32, 128, seed=m + r)
                xs = random_dev([512], 16, 32, 128, seed=m + 1)
                st = torch.empty((1, 32, 128, 128), dtype=torch.float32, device=dev)
                st2 = torch.empty_like(st)
                o = torch.empty((512, 32, 128), dtype=torch.bfloat16, device=dev)
                wsr = fused_ws(xt, xs, 1, 16, 32, 128)
                t_rep = timed_us(lambda: fused(xt, xs, st, o, st2, wsr))
                emit({"workload": f"replay vs full prefill Hk=16 Hv=32 d=128 bf16, m={m}, r={r}, suffix 512",
                      "t_full_us": t_full["p50"], "t_full_state_only_us": t_state["p50"],
                      "t_replay_us": t_rep["p50"], "speedup": t_full["p50"] / t_rep["p50"],
                      "speedup_state_only_full": t_state["p50"] / t_rep["p50"]})


def _layer(p, l):
    """Sequence l of a packed batch as its own one-sequence batch."""
    import synth
    a, b = int(p.cu_seqlens[l]), int(p.cu_seqlens[l + 1])
    import numpy as np
    return synth.Packed(p.shape, p.q[a:b], p.k[a:b], p.v[a:b], p.g[a:b], p.beta[a:b],
                        np.array([0, b - a], np.int32))


def cpu_baseline(tails, sufs, r, s, seconds):
    """The fp64 oracle, as it stands, on the host cores, on the same seeded
    inputs as the GPU step: layer after layer (the tail replay from zero, then
    the suffix forward from the replayed state, all 32 heads), until about
    ``seconds`` of wall time have passed; once on every usable core and once on
    one thread.  ``value`` is the all-core rate."""
    import oracle

    def run(threads):
        layers = 0
        t0 = time.perf_counter()
        while True:
            t, f = _layer(tails, layers % tails.num_seqs), _layer(sufs, layers % sufs.num_seqs)
            et, ef = t.exact(), f.exact()
            _, st = oracle.recurrence(et["k"], et["v"], et["g"], et["beta"], et["cu_seqlens"], nthreads=threads)
            oracle.recurrence(ef["k"], ef["v"], ef["g"], ef["beta"], ef["cu_seqlens"], q=ef["q"], state_in=st,
                              nthreads=threads)
            layers += 1
            el = time.perf_counter() - t0
            if el >= seconds or layers >= tails.num_seqs:
                return layers, el

    cores = min(usable_cores(), oracle.max_threads())
    n_all, el_all = run(cores)
    n_one, el_one = run(1)
    model = cpu_model()
    return {"value": n_all * (r + s) / el_all, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{n_all} of the stack's layers (tail {r} from zero + suffix {s} with outputs, all 32 "
                      f"heads, the bench's own seeded inputs) in {el_all:.2f} s wall on {cores} threads, {model}; "
                      f"fp64 token-by-token recurrence, OpenMP over (sequence, value head)",
            "cpu_model": model,
            "single_thread": {"value": n_one * (r + s) / el_one, "unit": "tokens/s", "cores": 1,
                              "sample": f"{n_one} layer(s) in {el_one:.2f} s wall on 1 thread"}}


if __name__ == "__main__":
    main()
