#!/usr/bin/env python3
"""Benchmark of the GDN tail-replay hot path on one MI355X.

One step = the whole hot path over one batch of resident synthetic input:
Independent Tail-Replay of every value head's state from zero over the last
r tokens of the matched prefix (paper Section 3, Eq. 2), then the chunked
forward over the new suffix from the rebuilt states, emitting its outputs.

Default workload: one GDN layer with hybrid-model head shapes (16 key heads,
32 value heads, d_k = d_v = 128, bf16 q/k/v, fp32 g/beta/state), matched
prefix 8192 tokens, replay tail 819 tokens (10 %), 512 suffix tokens.

Prints ONE JSON line.  ``value`` is tokens through the path per second
(tail + suffix tokens per step / step time): the step is one
``gdn_replay_forward`` call (replay, then the suffix forward from the rebuilt
state, the suffix's chunk preparation overlapped with the tail's scan),
launched eagerly on one stream.  ``ms_per_step_two_calls`` times the same work
as ``gdn_tail_replay`` + ``gdn_chunk_forward``, ``ms_per_step_graph`` the fused
step replayed from a HIP graph.  Per-stage kernel durations come from HIP
events that the library records between its kernels on the stream the kernels
run on, in a separate pass of the same steps; ``roofline`` describes the
dominant kernel.

``--summarize-pmc FETCH_DIR WRITE_DIR`` (no GPU) turns two rocprofv3 --pmc
runs of ``bench.py --calib-copy`` (FETCH_SIZE, then WRITE_SIZE) into the
traffic summary under profiles/ that later runs report as ``traffic``.
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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic_workload1_r{r}.json")
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
    ap.add_argument("--replay", type=int, default=819, choices=[410, 819],
                    help="replay tail length of the 8192-token prefix")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time for the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches only")
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="tail replays timed after an Infinity Cache flush")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run plain device copies of a known size (PMC calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--pmc-out", default=None,
                    help="with --summarize-pmc: output .json (default: the default workload's file)")
    ap.add_argument("--pmc-workload", default=None,
                    help="with --summarize-pmc: workload description stored in the summary")
    ap.add_argument("--sweep", action="store_true",
                    help="time the other workloads instead (one JSON line each): small fp32 layer, "
                         "36-layer stack, 16 varlen hits, decode steps, FA-KV transfer overlap, layer-block replay, "
                         "replay-vs-full at 8K/16K/32K")
    ap.add_argument("--only", default="",
                    help="with --sweep: comma list of sections to run "
                         "(small, layer410, stack, hits, decode, h2d, block, full)")
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


def summarize_pmc(fetch_dir, write_dir, replay, out_path=None, workload=None):
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
        if not any(t in name for t in ("k_scan", "k_intra", "k_decode")):
            continue
        short = name.split("(")[0].replace("void ", "")
        fb = fetch[name] * 1024.0 * f_fetch
        wb = write.get(name, 0.0) * 1024.0 * f_write
        kernels[short] = {"fetch_kib": fetch[name], "write_kib": write.get(name, 0.0),
                          "fetch_bytes": fb, "write_bytes": wb, "traffic_bytes": fb + wb}
    summary = {"workload": workload or f"one layer Hk=16 Hv=32 d=128 bf16, tail {replay} + suffix 512",
               "source_sha256": kernel_source_hash(),
               "calibration": {"kernel": cname.split("(")[0], "bytes_each_way": CALIB_BYTES,
                               "fetch_kib": cal_fetch, "write_kib": cal_write,
                               "fetch_factor": f_fetch, "write_factor": f_write},
               "kernels": kernels,
               "commands": [
                   "cd /tmp && export TMPDIR=/tmp && timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE "
                   "--output-format csv -d $OUT/pmc_fetch -o fetch -- python3 $ROOT/bench.py "
                   "--no-cpu-baseline --no-graph --steps 5 --warmup 2 --cold-reps 0 --calib-copy",
                   "(same with WRITE_SIZE into $OUT/pmc_write)",
                   f"python bench.py --summarize-pmc $OUT/pmc_fetch $OUT/pmc_write"]}
    path = out_path or TRAFFIC_FILE.format(r=replay)
    with open(path, "w") as f:
        json.dump(summary, f, indent=1)
    print(json.dumps(summary, indent=1))
    return path


def load_traffic(replay, kernel_short):
    """Calibrated HBM bytes per launch of `kernel_short` from the committed PMC
    summary, or None when there is none or the kernels changed since."""
    path = TRAFFIC_FILE.format(r=replay)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        s = json.load(f)
    if s.get("source_sha256") != kernel_source_hash():
        return None
    k = s["kernels"].get(kernel_short)
    return None if k is None else k["traffic_bytes"]


# ---------------------------------------------------------------- main
def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.replay, args.pmc_out, args.pmc_workload)
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
    import torch

    import paper_2608_30310_amd as gdn
    import synth
    from synth import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    gdn.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    shape, hits = workloads.workload1(args.replay)
    hit = hits[0]
    tail = synth.pack([hit.tail(shape)])
    suf = synth.pack([hit.suffix(shape)])

    def to_dev(p):
        def qkv(a):
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return dict(q=qkv(p.q), k=qkv(p.k), v=qkv(p.v), g=torch.from_numpy(p.g).to(dev),
                    beta=torch.from_numpy(p.beta).to(dev),
                    cu=torch.from_numpy(p.cu_seqlens).to(dev),
                    cu_host=torch.from_numpy(p.cu_seqlens.copy()))

    xt, xs = to_dev(tail), to_dev(suf)
    N, hk, hv, dk, dv = 1, shape.hk, shape.hv, shape.dk, shape.dv
    state = torch.empty((N, hv, dk, dv), dtype=torch.float32, device=dev)
    state2 = torch.empty_like(state)
    o = torch.empty((suf.num_tokens, hv, dv), dtype=torch.bfloat16, device=dev)
    ws_t = torch.empty(gdn.workspace_size(N, hk, hv, dk, dv, tail.cu_seqlens.tolist()) + 256,
                       dtype=torch.uint8, device=dev)
    ws_f = torch.empty(gdn.workspace_size(N, hk, hv, dk, dv, suf.cu_seqlens.tolist(),
                                          with_outputs=True) + 256,
                       dtype=torch.uint8, device=dev)
    ws_rf = torch.empty(gdn.replay_forward_workspace_size(N, hk, hv, dk, dv, tail.cu_seqlens.tolist(),
                                                          suf.cu_seqlens.tolist()) + 256,
                        dtype=torch.uint8, device=dev)
    names_t = gdn.stage_names(False)
    names_f = gdn.stage_names(True)
    names_rf = gdn.replay_forward_stage_names()

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    def replay_call(ev=None):
        gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"],
                        state_out=state, workspace=ws_t, events=ev)

    def forward_call(ev=None):
        gdn.chunk_forward(xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"], xs["cu_host"],
                          state_in=state, o=o, state_out=state2, workspace=ws_f, events=ev)

    def two_calls(ev_t=None, ev_f=None):
        replay_call(ev_t)
        forward_call(ev_f)

    def step(ev=None):
        gdn.replay_forward(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xs["q"], xs["k"], xs["v"],
                           xs["g"], xs["beta"], xs["cu"], cu_tail_host=xt["cu_host"],
                           cu_suf_host=xs["cu_host"], state_mid=state, o=o, state_out=state2,
                           workspace=ws_rf, events=ev)

    for _ in range(args.warmup):
        step()
        two_calls()
    torch.cuda.synchronize()
    K = args.steps

    def timed(fn):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        for _ in range(K):
            fn()
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / K

    # ---- graph of one step, checked bitwise against the eager step on several replays
    graph, graph_note = None, None
    if not args.no_graph:
        step()
        torch.cuda.synchronize()
        want_s, want_o = state2.clone(), o.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        ok = True
        for _ in range(3):
            state2.zero_()
            o.zero_()
            g.replay()
            torch.cuda.synchronize()
            ok = ok and torch.equal(state2, want_s) and torch.equal(o, want_o)
            step()               # eager work between replays
            torch.cuda.synchronize()
        if ok:
            graph = g
        else:
            graph_note = "graph replay differed from the eager step; graph not timed"

    ms_per_step = timed(step)
    ms_two = timed(two_calls)
    ms_graph = timed(graph.replay) if graph is not None else None

    # ---- per-stage kernel durations: events recorded by the library on its stream
    ev_rf = [new_events(len(names_rf) + 1) for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        step(ev_rf[i])
    torch.cuda.synchronize()
    ev_t = [new_events(len(names_t) + 1) for _ in range(K)]
    ev_f = [new_events(len(names_f) + 1) for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        two_calls(ev_t[i], ev_f[i])
    torch.cuda.synchronize()
    stages = {}
    for prefix, names, evs in (("replay_forward", names_rf, ev_rf), ("tail_replay", names_t, ev_t),
                               ("chunk_forward", names_f, ev_f)):
        for j, nm in enumerate(names):
            d = [evs[i][j].elapsed_time(evs[i][j + 1]) * 1e3 for i in range(K)]
            stages[f"{prefix}.{nm}"] = {"mean_us": statistics.fmean(d),
                                        "median_us": statistics.median(d)}
    warm = quantiles([ev_t[i][0].elapsed_time(ev_t[i][-1]) * 1e3 for i in range(K)])

    # ---- the same with the call's launches already queued: a spin kernel
    # holds the GPU while the host enqueues the call, so the interval is the
    # device's alone (kernels and the gaps between them, no host pacing)
    def queued(fn):
        lat = []
        for _ in range(K):
            torch.cuda._sleep(QUEUE_SPIN_CYCLES)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            lat.append(a.elapsed_time(b) * 1e3)
        return quantiles(lat)

    queued_rebuild = queued(replay_call)

    # ---- cold rebuild latency: Infinity Cache flushed before each tail replay
    cold = None
    if args.cold_reps > 0:
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
        lat = []
        for i in range(args.cold_reps):
            flush.fill_(float(i))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            replay_call()
            b.record()
            torch.cuda.synchronize()
            lat.append(a.elapsed_time(b) * 1e3)
        cold = quantiles(lat)
        del flush

    if args.calib_copy:
        # a plain elementwise kernel that reads and writes CALIB_BYTES once each
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ---- algorithmic work
    elt = 2
    r, s = hit.r, hit.s
    ft, bt = per_token_work(hk, hv, dk, dv, elt, outputs=False)
    ff, bf = per_token_work(hk, hv, dk, dv, elt, outputs=True)
    state_bytes = N * hv * dk * dv * 4
    tail_flops, tail_bytes = r * hv * ft, r * hv * bt + state_bytes
    fwd_flops, fwd_bytes = s * hv * ff, s * hv * bf + 2 * state_bytes
    path_flops, path_bytes = tail_flops + fwd_flops, tail_bytes + fwd_bytes
    t_s = ms_per_step * 1e-3
    path_bound_s = max(path_flops / (BF16_PEAK_TFLOPS * 1e12), path_bytes / (HBM_PEAK_GBS * 1e9))

    # dominant kernel: the stage of the timed (fused) step with the largest
    # mean time; its algorithmic bytes are those of the part of the path it
    # runs (the tail replay's or the suffix forward's)
    fused = {k: v for k, v in stages.items() if k.startswith("replay_forward.")}
    dom = max(fused, key=lambda k: fused[k]["mean_us"])
    grp = hv // hk
    # the suffix's chunk preparation reads q, k (shared by the group), g and
    # beta and forms K K^T and Q K^T per chunk
    prep_bytes = s * hv * (2 * elt * dk / grp + 8)
    prep_flops = s * hv * (2 * 2 * CHUNK * dk / grp)
    kbytes, kflops = {"replay_forward.tail intra": (tail_bytes, tail_flops),
                      "replay_forward.tail scan + suffix intra": (tail_bytes + prep_bytes,
                                                                  tail_flops + prep_flops),
                      "replay_forward.suffix scan": (fwd_bytes, fwd_flops)}[dom]
    dom_s = stages[dom]["mean_us"] * 1e-6
    achieved = kbytes / dom_s / 1e9
    kname = {"replay_forward.tail intra": "gdn::k_intra<unsigned short, 128, false>",
             "replay_forward.tail scan + suffix intra": "gdn::k_scan_cols_intra<unsigned short, 128>",
             "replay_forward.suffix scan": "gdn::k_scan_cols<unsigned short, 128, true>"}.get(dom)
    traffic = load_traffic(args.replay, kname) if kname else None
    roofline = {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                "algorithmic_bytes_per_launch": kbytes,
                "mfma_frac": kflops / dom_s / (BF16_PEAK_TFLOPS * 1e12)}

    tokens = r + s
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
        "data": "synthetic",
        "config": {"workload": f"one GDN layer, Hk=16 Hv=32 d_k=d_v=128 bf16 q/k/v; "
                               f"prefix 8192, tail replay r={r} from zero + {s}-token suffix "
                               f"forward with outputs",
                   "global_batch": 1, "seq_len": r + s, "parallelism": "single GPU"},
        "launch": "eager, gdn_replay_forward",
        "ms_per_step_two_calls": ms_two,
        "ms_per_step_graph": ms_graph,
        "rebuild_latency_us": warm["p50"],
        "rebuild_latency_warm_us": warm,
        "rebuild_latency_cold_us": cold,
        "rebuild_latency_queued_us": queued_rebuild,
        "replay_tokens_per_s": r / (warm["p50"] * 1e-6),
        "stages": stages,
        "path": {"flops": path_flops, "bytes": path_bytes, "roofline_us": path_bound_s * 1e6,
                 "roofline_frac": path_bound_s / t_s,
                 "mfma_frac": path_flops / t_s / (BF16_PEAK_TFLOPS * 1e12)},
        "roofline": roofline,
        "cpu_baseline": None,
        "gpu": torch.cuda.get_device_name(dev),
    }
    if graph_note:
        result["note"] = graph_note

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(tail, suf, r, s, args.cpu_seconds)
    print(json.dumps(result), flush=True)


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
              "tokens_per_s": (205 + 256) / (both["p50"] * 1e-6)})

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

    # ---- 36-layer stack, m = 32768, r = 3277: 36 sequential per-layer replays,
    #      and the batched variant (layers as 36 sequences of one launch)
    if want("stack"):
        L, r2 = 36, 3277
        xl = [random_dev([r2], 16, 32, 128, seed=100 + l) for l in range(L)]
        wsl, stl, _ = buffers(xl[0], 1, 16, 32, 128, False)
        seq = timed_us(lambda: [replay(x, stl, wsl) for x in xl])
        xb = random_dev([r2] * L, 16, 32, 128, seed=7)
        wsb, stb, _ = buffers(xb, L, 16, 32, 128, False)
        bat = timed_us(lambda: replay(xb, stb, wsb))
        emit({"workload": "36-layer stack Hk=16 Hv=32 d=128 bf16, m=32768, tail 3277 per layer",
              "rebuild_latency_sequential_us": seq, "rebuild_latency_batched_us": bat,
              "replay_tokens_per_s_sequential": L * r2 / (seq["p50"] * 1e-6),
              "replay_tokens_per_s_batched": L * r2 / (bat["p50"] * 1e-6)})

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
              "replay_tokens_per_s": sr / (rep["p50"] * 1e-6)})

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

            def h2d(stream):
                with torch.cuda.stream(stream):
                    dev_kv.copy_(host_kv, non_blocking=True)

            main = torch.cuda.current_stream()

            def serial():
                h2d(main)
                replays()
                forwards()

            def overlapped():
                copy_stream.wait_stream(main)
                h2d(copy_stream)
                replays()
                main.wait_stream(copy_stream)
                forwards()

            t_h2d = timed_us(lambda: h2d(main))
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


def cpu_baseline(tail, suf, r, s, seconds):
    """The fp64 oracle, as it stands, on the host cores: the same step repeated
    until about ``seconds`` of CPU time have passed."""
    import oracle
    ext, exs = tail.exact(), suf.exact()
    threads = oracle.max_threads()
    reps = 0
    t0 = time.perf_counter()
    while True:
        _, st = oracle.recurrence(ext["k"], ext["v"], ext["g"], ext["beta"], ext["cu_seqlens"])
        oracle.recurrence(exs["k"], exs["v"], exs["g"], exs["beta"], exs["cu_seqlens"],
                          q=exs["q"], state_in=st)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or reps >= 200:
            break
    return {"value": reps * (r + s) / el, "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} steps of the default workload (all 32 heads, tail {r} + suffix {s}) "
                      f"in {el:.2f} s wall on {threads} threads ({platform.processor() or 'cpu'})"}


if __name__ == "__main__":
    main()
