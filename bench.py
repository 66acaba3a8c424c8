#!/usr/bin/env python3
"""Throughput of incremental ViT encoding on one MI355X.

Workload (default): SigLIP-So400m-shaped ViT (224x224, patch 14, N = 256,
D = 1152, 27 layers, 16 heads, MLP 4304), bf16, one camera stream in which a
56x56 textured square moves 4 px/frame over a static background (about 10% of
the tokens change per frame), threshold 0.98.  One step = incvit_step on one
frame (embedding + similarity + selection + all layers for the refreshed rows).

Prints one JSON line: frames/s of the timed steps, the speedup over the full
re-encode of a frame on the same GPU, the roofline of the dominant kernel
(per-kernel HIP events on the launch stream) and the CPU oracle's rate on a
bounded sample of the same stream.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

METRIC = "incremental ViT frames/sec at 10% refresh (So400m shape); speedup vs full encode"
HBM_PEAK_GBS = 8000.0


def gemm_bytes(m, M: float, kind: str) -> float:
    """Algorithmic HBM bytes of one launch of a layer kernel with M refreshed rows."""
    D, F, N, eb = m.dim, m.mlp_dim, m.n_tokens, (2 if m.dtype == "bf16" else 4)
    if kind == "qkv":
        return D * 3 * D * eb + M * D * eb + M * 3 * D * eb
    if kind == "oproj":
        return D * D * eb + 2 * M * D * eb + M * D * 4
    if kind == "fc1":
        return D * F * eb + M * D * 4 + M * F * eb
    if kind == "fc2":
        return F * D * eb + M * F * eb + M * D * 4 + M * D * eb
    if kind == "attn":
        return 2 * M * D * eb  # + K/V of the views, added by the caller
    raise KeyError(kind)


def cpu_baseline(wl, frames, seconds: float):
    """The oracle as it is, on this host: full encode of frame 0, then steps of
    the same stream until about `seconds` of step time have been spent."""
    import numpy as np
    from oracle import vit
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    model = vit.Model(wl.model, wl.weights())
    caches = [vit.full_encode(model, frames[0][v]) for v in range(wl.views)]
    spent, steps = 0.0, 0
    while steps < len(frames) - 1 and (spent < seconds or steps == 0):
        t = time.perf_counter()
        for v in range(wl.views):
            vit.step(model, frames[steps + 1][v], caches[v], wl.tau, wl.caps[v])
        spent += time.perf_counter() - t
        steps += 1
    return {"value": round(steps * wl.views / spent, 4), "unit": "frames/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{wl.name}: oracle full encode of frame 0, then {steps} incremental steps "
                      f"(frames 1..{steps}) of the same stream; value = frames / summed step time"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="so400m",
                    help="so400m (default), tiny, so400m_x3, so400m_448, vitl_x8")
    ap.add_argument("--rho", type=float, default=0.10, help="refresh ratio of so400m_448 (top-k)")
    ap.add_argument("--full-repeats", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel events")
    ap.add_argument("--eager", dest="graph", action="store_false",
                    help="launch kernel by kernel instead of replaying captured HIP graphs")
    ap.add_argument("--waves", default=None, help="waves per GEMM workgroup: four comma-separated values (0 = automatic)")
    ap.add_argument("--cols", default=None, help="column blocks per GEMM workgroup: four values (0 = automatic)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the encoder's state is per stream and this build runs "
              "single-GPU only (streams would shard across GPUs with no exchange); use --gpus 1.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2607_12287_amd import incvit, synth

    wl = synth.workload(args.workload, rho=args.rho)
    m = wl.model
    B = wl.views
    total = args.warmup + args.steps + 1
    frames_np = list(wl.patch_frames(total))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    frames = torch.from_numpy(np.stack(frames_np)).to(dev)  # [T][B][N][P], resident in HBM
    enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=B)
    if args.waves or args.cols:
        incvit._check(incvit.incvit_set_tuning(
            enc.h, [int(x) for x in args.waves.split(",")] if args.waves else None,
            [int(x) for x in args.cols.split(",")] if args.cols else None), enc.h)
    buf, caches = enc.new_caches(B)
    out = (torch.empty((B, m.n_tokens), dtype=torch.int32, device=dev),
           torch.empty((B,), dtype=torch.int32, device=dev),
           torch.empty((B, m.n_tokens, m.dim), dtype=enc.dtype, device=dev))
    counts = torch.zeros((total, B), dtype=torch.int32, device=dev)

    inp = torch.empty_like(frames[0])  # the fixed input buffer the graphs read

    # full re-encode: the baseline the speedup divides by (scratch caches)
    sbuf, scratch = enc.new_caches(B)
    inp.copy_(frames[0])
    gfull = enc.full_graph(inp, scratch) if args.graph else None
    run_full = (lambda: enc.launch(gfull)) if args.graph else (lambda: enc.full_encode(inp, scratch))
    for _ in range(3):
        run_full()
    torch.cuda.synchronize()
    full_ms = []
    for _ in range(args.full_repeats):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run_full()
        e1.record()
        e1.synchronize()
        full_ms.append(e0.elapsed_time(e1))
    if gfull is not None:
        enc.drop_graph(gfull)
    del sbuf, scratch

    # the stream: full encode of frame 0, warmup steps, timed steps
    enc.full_encode(frames[0], caches)
    gstep = enc.step_graph(inp, caches, wl.tau, wl.caps, out) if args.graph else None

    def one_step(t):
        inp.copy_(frames[t])
        if gstep is not None:
            enc.launch(gstep)
        else:
            enc.step(inp, caches, wl.tau, wl.caps, out=out)

    for t in range(1, args.warmup + 1):
        one_step(t)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    e0.record()
    for t in range(args.warmup + 1, total):
        one_step(t)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    dev_ms = e0.elapsed_time(e1)
    step_ms = wall * 1e3 / args.steps
    fps = args.steps * B / wall
    full_med = statistics.median(full_ms)
    if gstep is not None:
        enc.drop_graph(gstep)

    # same frames again, eagerly, with per-kernel events on the launch stream
    buf2, caches2 = enc.new_caches(B)
    enc.full_encode(frames[0], caches2)
    for t in range(1, args.warmup + 1):
        enc.step(frames[t], caches2, wl.tau, wl.caps, out=out)
    torch.cuda.synchronize()
    if not args.no_profile:
        incvit.incvit_profile_read(enc.h, reset=True)
        incvit.incvit_profile_enable(enc.h, True)
    for t in range(args.warmup + 1, total):
        enc.step(frames[t], caches2, wl.tau, wl.caps, out=out)
        counts[t].copy_(out[1])
    torch.cuda.synchronize()
    k = counts[args.warmup + 1:].float().cpu().numpy()
    mean_rows = float(k.sum(axis=1).mean())

    result = {
        "metric": METRIC, "value": round(fps, 2), "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": m.dtype,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {m.img_h}x{m.img_w} p{m.patch} N={m.n_tokens} D={m.dim} "
                               f"L={m.depth} h={m.heads} F={m.mlp_dim}, {B} stream(s), tau={wl.tau}, "
                               f"caps={wl.caps[:1]}{'...' if B > 1 else ''}",
                   "views": B, "tokens": m.n_tokens, "refresh_mean": round(mean_rows / (B * m.n_tokens), 4),
                   "rows_mean": round(mean_rows, 2)},
        "device_ms_per_step": round(dev_ms / args.steps, 5),
        "launch": "hip-graph" if args.graph else "eager",
        "full_encode_ms": round(full_med, 5),
        "full_encode_frames_per_s": round(B * 1e3 / full_med, 2),
        "speedup_vs_full_encode": round(full_med / step_ms, 3),
    }

    if not args.no_profile:
        prof = incvit.incvit_profile_read(enc.h, reset=True)
        incvit.incvit_profile_enable(enc.h, False)
        kinds = {k: v for k, v in prof.items() if v[1] > 0}
        dom = max(kinds, key=lambda k: kinds[k][0])
        avg_us = kinds[dom][0] * 1e3 / kinds[dom][1]
        if dom in ("qkv", "oproj", "fc1", "fc2"):
            nbytes = gemm_bytes(m, mean_rows, dom)
        elif dom == "attn":
            nbytes = gemm_bytes(m, mean_rows, "attn") + 2 * B * m.n_tokens * m.dim * (2 if m.dtype == "bf16" else 4)
        else:
            nbytes = None
        achieved = nbytes / (avg_us * 1e-6) / 1e9 if nbytes else None
        result["roofline"] = {
            "kernel": dom, "bound": "hbm", "achieved": round(achieved, 1) if achieved else None,
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
            "traffic": None, "avg_launch_us": round(avg_us, 3), "bytes_per_launch": nbytes,
        }
        result["kernel_us_per_launch"] = {k: round(v[0] * 1e3 / v[1], 3) for k, v in kinds.items()}
        result["kernel_ms_per_step"] = {k: round(v[0] / args.steps, 5) for k, v in kinds.items()}
    del buf2, caches2

    if not args.no_cpu_baseline:
        n_cpu = min(len(frames_np), 64)
        result["cpu_baseline"] = cpu_baseline(wl, frames_np[:n_cpu], args.cpu_seconds)

    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
