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
(tail + suffix tokens per step / step time).  Per-stage durations come from
HIP events that the library records between its kernels on the stream the
kernels run on; ``roofline`` describes the dominant kernel.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import statistics
import sys
import time

METRIC = "GDN tail-replay tokens/sec/GPU + state-rebuild latency; % of MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
CHUNK = 64


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
    return ap.parse_args()


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


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the per-(sequence, head) work shards with no exchange; see DESIGN.md)",
              file=sys.stderr)
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
    names_t = gdn.stage_names(False)
    names_f = gdn.stage_names(True)

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    def step(ev_t=None, ev_f=None):
        gdn.tail_replay(xt["k"], xt["v"], xt["g"], xt["beta"], xt["cu"], xt["cu_host"],
                        state_out=state, workspace=ws_t, events=ev_t)
        gdn.chunk_forward(xs["q"], xs["k"], xs["v"], xs["g"], xs["beta"], xs["cu"], xs["cu_host"],
                          state_in=state, o=o, state_out=state2, workspace=ws_f, events=ev_f)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    ev_t = [new_events(len(names_t) + 1) for _ in range(K)]
    ev_f = [new_events(len(names_f) + 1) for _ in range(K)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(K):
        step(ev_t[i], ev_f[i])
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / K

    stages = {}
    for prefix, names, evs in (("tail_replay", names_t, ev_t), ("chunk_forward", names_f, ev_f)):
        for j, nm in enumerate(names):
            d = [evs[i][j].elapsed_time(evs[i][j + 1]) * 1e3 for i in range(K)]
            stages[f"{prefix}.{nm}"] = {"mean_us": statistics.fmean(d),
                                        "median_us": statistics.median(d)}
    rebuild = [ev_t[i][0].elapsed_time(ev_t[i][-1]) * 1e3 for i in range(K)]
    rebuild_us = statistics.median(rebuild)

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

    # dominant kernel: the stage with the largest mean time per step
    dom = max(stages, key=lambda k: stages[k]["mean_us"])
    dom_call = dom.split(".")[0]
    kbytes = tail_bytes if dom_call == "tail_replay" else fwd_bytes
    dom_s = stages[dom]["mean_us"] * 1e-6
    achieved = kbytes / dom_s / 1e9
    roofline = {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                "algorithmic_bytes_per_launch": kbytes}

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
        "rebuild_latency_us": rebuild_us,
        "replay_tokens_per_s": r / (rebuild_us * 1e-6),
        "stages": stages,
        "path": {"flops": path_flops, "bytes": path_bytes, "roofline_us": path_bound_s * 1e6,
                 "roofline_frac": path_bound_s / t_s,
                 "mfma_frac": path_flops / t_s / (BF16_PEAK_TFLOPS * 1e12)},
        "roofline": roofline,
        "cpu_baseline": None,
        "gpu": torch.cuda.get_device_name(dev),
    }

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(tail, suf, r, s, args.cpu_seconds)
    print(json.dumps(result), flush=True)


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
