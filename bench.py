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
import csv
import glob
import hashlib
import json
import math
import os
import re
import statistics
import sys
import time

METRIC = "incremental ViT frames/sec at 10% refresh (So400m shape); speedup vs full encode"
HBM_PEAK_GBS = 8000.0
# non-packed fp32 FMA: 256 CUs x 4 SIMDs x 16 lanes x 2 FLOP x 2.4 GHz (packed fp32 is compiled out)
ALU_PEAK_TFLOPS = 78.6
ROOT = os.path.dirname(os.path.abspath(__file__))
PROFILES = os.path.join(ROOT, "profiles")
GEMM_KIND = {"0": "qkv", "1": "fc1", "2": "fc2", "3": "oproj", "4": "oproj", "5": "fc2"}  # epilogue template argument


def source_hash() -> str:
    """Hash of every kernel and ABI source (not the native driver that only runs
    them): stored counters are used only while it matches."""
    h = hashlib.sha256()
    files = sorted([f for f in glob.glob(os.path.join(ROOT, "paper_2607_12287_amd", "csrc", "*"))
                    if os.path.basename(f) != "incvit_drive.cpp"] +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_kind(name: str):
    """Kernel kind of a dispatch name in a rocprofv3 trace (None for other kernels)."""
    m = re.search(r"incvit::(\w+)_kernel(?:<([^>]*)>)?", name)
    if not m:
        return None
    if m.group(1) == "gemm":
        return GEMM_KIND.get(m.group(2).split(",")[1].strip())
    if m.group(1) == "gemm_tiled":  # template <EPI, BM, NS>
        return GEMM_KIND.get(m.group(2).split(",")[0].strip())
    if m.group(1) == "res":
        return "res_ln1"
    return {"keyln": "key_ln", "keyproj": "key_proj"}.get(m.group(1), m.group(1))


def kinds_in_order(names):
    """Kinds of dispatches given in launch order."""
    return [kernel_kind(n) for n in names]


def stored_traffic(workload: str, kind: str):
    """HBM bytes per launch of `kind` from the committed counter summary, if the
    kernels have not changed since it was taken."""
    path = os.path.join(PROFILES, f"step_hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    vals, src = {}, None
    for line in open(path):
        f = line.split()
        if len(f) == 2 and f[0] == "source_hash":
            src = f[1]
        if len(f) == 3 and f[0] == "traffic_bytes_per_launch":
            vals[f[1]] = float(f[2])
    if src != source_hash():
        return None
    return vals.get(kind)


def run_env(torch) -> dict:
    """Versions and clocks of the run (best effort: fields that cannot be read
    are left out)."""
    env = {"torch": torch.__version__, "hip": getattr(torch.version, "hip", None)}
    try:
        p = torch.cuda.get_device_properties(0)
        env.update({"device": p.name, "arch": getattr(p, "gcnArchName", None),
                    "compute_units": p.multi_processor_count, "hbm_gib": round(p.total_memory / 2**30, 1)})
    except Exception:
        pass
    try:
        with open("/sys/module/amdgpu/version") as f:
            env["amdgpu_driver"] = f.read().strip()
    except OSError:
        pass
    # current DPM levels (the line marked '*') of the first card that has them
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        clocks = {}
        for name in ("pp_dpm_sclk", "pp_dpm_mclk", "pp_dpm_fclk"):
            try:
                with open(os.path.join(dev, name)) as f:
                    cur = [ln.split(":", 1)[1].replace("*", "").strip() for ln in f if ln.rstrip().endswith("*")]
                if cur:
                    clocks[name[7:]] = cur[0]
            except (OSError, IndexError):
                pass
        if clocks:
            env["clocks"] = clocks
            break
    return env


def quantile(xs_sorted, q: float) -> float:
    """Linear-interpolation quantile of an ascending list."""
    if not xs_sorted:
        return float("nan")
    pos = q * (len(xs_sorted) - 1)
    i = int(pos)
    j = min(i + 1, len(xs_sorted) - 1)
    return xs_sorted[i] + (xs_sorted[j] - xs_sorted[i]) * (pos - i)


def rows_dist(k) -> dict:
    """Distribution of the refreshed rows: per step (summed over the streams)
    min / median / p90 / max, and the mean per stream."""
    tot = sorted(float(x) for x in k.sum(axis=1))
    return {"per_step": {"min": tot[0], "median": quantile(tot, 0.5), "p90": round(quantile(tot, 0.9), 2),
                         "max": tot[-1]},
            "per_stream_mean": [round(float(x), 2) for x in k.mean(axis=0)]}


def ksplit(m) -> int:
    """K split of the MLP down projection (the library's rule)."""
    nblocks = m.dim // 16
    kchunks = -(-m.mlp_dim // 32)
    return max(1, min(4, 256 // nblocks, kchunks // 8))


def kernel_bytes(m, M: float, kind: str):
    """Algorithmic HBM bytes of one launch of a layer kernel with M refreshed rows
    (weights once, each row operand once; partial sums of a split K counted as
    written and read once).  None for kinds without a figure here."""
    D, F, eb = m.dim, m.mlp_dim, (2 if m.dtype == "bf16" else 4)
    s2 = ksplit(m)
    if kind == "qkv":
        return 3 * D * D * eb + M * D * eb + 3 * M * D * eb
    if kind == "oproj":
        return D * D * eb + 3 * M * D * eb
    if kind == "fc1":
        return D * F * eb + M * D * eb + M * F * eb
    if kind == "fc2":
        return F * D * eb + M * F * eb + s2 * M * D * 4
    if kind == "res_ln1":  # partials + residual -> X^{l+1} (and Y after the last layer)
        return s2 * M * D * 4 + 3 * M * D * eb
    if kind == "attn":
        return 2 * M * D * eb  # + K/V of the streams, added by the caller
    return None


def gemm_flops(m, M: float, kind: str):
    """Algorithmic FLOP of one launch of a gathered GEMM over M rows (2 per
    multiply-add, the output columns the model has; the LayerNorm statistics
    the matrix cores form beside the products are not counted)."""
    D, F = m.dim, m.mlp_dim
    return {"qkv": 2 * M * D * 3 * D, "oproj": 2 * M * D * D, "fc1": 2 * M * D * F,
            "fc2": 2 * M * F * D}.get(kind)


def torch_full_forward(m, w, patches, repeats: int):
    """Context for the full-encode baseline: the same model's full forward over
    every token written with plain torch ops (hipBLASLt GEMMs in the storage
    type, fp32 LayerNorm/softmax/GELU).  Returns (median ms, launch mode): a
    HIP-graph replay when capturing works and every replay equals the eager
    result, else eager."""
    import torch
    import torch.nn.functional as F
    dev = patches.device
    dt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    B, N, D, H = patches.shape[0], m.n_tokens, m.dim, m.heads
    dh = D // H
    T = {k: torch.from_numpy(v).to(dev) for k, v in w.items()}
    Wd = {k: v.to(dt) for k, v in T.items()}

    def fwd():
        x = torch.matmul(patches, T["w_pe"]) + T["b_pe"] + T["pos"]       # fp32 embedding
        h = x.to(dt)
        for l in range(m.depth):
            g = lambda n: Wd[f"l{l}.{n}"]  # noqa: E731
            a = F.layer_norm(h.float(), (D,), T[f"l{l}.ln1_g"], T[f"l{l}.ln1_b"], m.ln_eps).to(dt)
            qkv = torch.matmul(a, g("w_qkv")) + g("b_qkv")
            q, k, v = (t.reshape(B, N, H, dh).permute(0, 2, 1, 3).contiguous() for t in qkv.split(D, dim=-1))
            sc = torch.matmul(q, k.transpose(-1, -2).contiguous()).float() * (dh ** -0.5)
            o = torch.matmul(torch.softmax(sc, dim=-1).to(dt), v)
            o = o.permute(0, 2, 1, 3).reshape(B, N, D)
            h = h + (torch.matmul(o, g("w_o")) + g("b_o"))
            a2 = F.layer_norm(h.float(), (D,), T[f"l{l}.ln2_g"], T[f"l{l}.ln2_b"], m.ln_eps).to(dt)
            f = F.gelu((torch.matmul(a2, g("w_1")) + g("b_1")).float(), approximate="tanh").to(dt)
            h = h + (torch.matmul(f, g("w_2")) + g("b_2"))
        return F.layer_norm(h.float(), (D,), T["lnf_g"], T["lnf_b"], m.ln_eps)

    def timed(run):
        for _ in range(3):
            run()
        torch.cuda.synchronize()
        ms = []
        for _ in range(repeats):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run()
            e1.record()
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        return statistics.median(ms)

    with torch.no_grad():
        ref = fwd()
        torch.cuda.synchronize()
        eager_ms = timed(fwd)
        try:
            st = torch.cuda.Stream()
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                fwd()
            torch.cuda.current_stream().wait_stream(st)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                out = fwd()
            ok = True
            for _ in range(3):  # replays with eager work in between, each checked
                graph.replay()
                torch.cuda.synchronize()
                ok = ok and bool(torch.equal(out, ref))
                fwd()
                torch.cuda.synchronize()
            if ok:
                graph_ms = timed(graph.replay)
                if graph_ms < eager_ms:
                    return graph_ms, "hip-graph"
        except Exception:  # capture not available: the eager time stands
            pass
    return eager_ms, "eager"


def approx_vs_full(enc, caches, frame):
    """Informational approximation error of the incremental outputs: cosine of
    each token's Y against a full encode of the same (last) frame, mean and
    minimum over tokens and streams."""
    import numpy as np
    buf, scratch = enc.new_caches(len(caches))
    enc.full_encode(frame, scratch)
    cos = []
    for c, sc in zip(caches, scratch):
        a, b = enc.export(c)["Y"], enc.export(sc)["Y"]
        cos.append((a * b).sum(1) / np.maximum(np.linalg.norm(a, axis=1) * np.linalg.norm(b, axis=1), 1e-30))
    cos = np.concatenate(cos)
    return {"mean": round(float(cos.mean()), 6), "min": round(float(cos.min()), 6)}


def measure_variant(wl, frames, score: str, period: int, steps: int, warmup: int, full_repeats: int,
                    mlp: str = "reuse"):
    """Frames/s of the same stream with another score (embedding or first-layer
    keys), another reading of the MLP over all tokens ("reuse" exact, "all")
    and, for period >= 1, under a refresh period: frame t is fully encoded when
    t % period == 0 (HIP-graph replays of the full encode), else incrementally
    (the step graph).  Period 0 = the rolling stream (one full encode of frame
    0 only).  Also the per-kernel times of an eager pass and the outputs'
    cosine against a full encode of the last frame."""
    import torch
    from paper_2607_12287_amd import incvit, synth
    m, B = wl.model, wl.views
    dev = frames.device
    enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=B, score=score, mlp=mlp)
    buf, caches = enc.new_caches(B)
    out = (torch.empty((B, m.n_tokens), dtype=torch.int32, device=dev),
           torch.empty((B,), dtype=torch.int32, device=dev),
           torch.empty((B, m.n_tokens, m.dim), dtype=enc.dtype, device=dev))
    inp = torch.empty_like(frames[0])
    inp.copy_(frames[0])
    gfull = enc.full_graph(inp, caches)
    full_ms = []
    for i in range(full_repeats + 3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        enc.launch(gfull)
        e1.record()
        e1.synchronize()
        if i >= 3:
            full_ms.append(e0.elapsed_time(e1))
    enc.launch(gfull)  # frame 0 encoded in full
    gstep = enc.step_graph(inp, caches, wl.tau, wl.caps, out)
    counts = torch.zeros((steps, B), dtype=torch.int32, device=dev)

    def frame(t):
        inp.copy_(frames[t])
        if period >= 1 and t % period == 0:
            enc.launch(gfull)
        else:
            enc.launch(gstep)

    for t in range(1, warmup + 1):
        frame(t)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for j, t in enumerate(range(warmup + 1, warmup + 1 + steps)):
        frame(t)
        counts[j].copy_(out[1])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    enc.drop_graph(gstep)
    enc.drop_graph(gfull)
    approx = approx_vs_full(enc, caches, frames[warmup + steps])
    k = counts.float().cpu().numpy()
    inc = [j for j, t in enumerate(range(warmup + 1, warmup + 1 + steps)) if not (period >= 1 and t % period == 0)]
    # per-kernel times: eager steps of the rolling stream with per-launch events
    enc.full_encode(frames[0], caches)
    incvit.incvit_profile_read(enc.h, reset=True)
    incvit.incvit_profile_enable(enc.h, True)
    n_prof = min(steps, 50)
    for t in range(1, n_prof + 1):
        enc.step(frames[t], caches, wl.tau, wl.caps, out=out)
    torch.cuda.synchronize()
    prof = incvit.incvit_profile_read(enc.h, reset=True)
    incvit.incvit_profile_enable(enc.h, False)
    enc.close()
    full_med = statistics.median(full_ms)
    res = {"score": score, "mlp": mlp, "period": period, "frames_per_s": round(steps * B / wall, 2),
           "ms_per_frame": round(wall * 1e3 / steps, 5), "full_encode_ms": round(full_med, 5),
           "speedup_vs_full_encode": round(full_med / (wall * 1e3 / steps), 3),
           "rows_mean_incremental": round(float(k[inc].sum(axis=1).mean()), 2) if inc else None,
           "kernel_us_per_launch": {kk: round(v[0] * 1e3 / v[1], 3) for kk, v in prof.items() if v[1] > 0},
           "approx_cos_vs_full": approx}
    kp = prof.get("key_proj")
    if kp and kp[1] > 0:
        us = kp[0] * 1e3 / kp[1]
        flop = 2.0 * B * m.n_tokens * m.dim * m.dim
        res["key_proj_roofline"] = {"bound": "alu", "achieved": round(flop / (us * 1e-6) / 1e12, 3),
                                    "peak": ALU_PEAK_TFLOPS, "unit": "TFLOP/s",
                                    "frac": round(flop / (us * 1e-6) / 1e12 / ALU_PEAK_TFLOPS, 4),
                                    "avg_launch_us": round(us, 3)}
    return res


def measure_flow(S: int, n: int, reps: int = 200):
    """The two-anchor flow update on S samples of n values (action chunks of
    horizon 50 x 32 dimensions by default): time per launch from HIP events
    over `reps` launches on the current stream, and its algorithmic bytes
    (x_0, v_0, v_7, b read, x_T written, fp32)."""
    import torch
    from paper_2607_12287_amd import incvit
    g = torch.Generator(device="cuda").manual_seed(7)
    x0, v0, v7, b = (torch.randn(S, n, device="cuda", generator=g) for _ in range(4))
    al, be = (torch.randn(S, device="cuda", generator=g) for _ in range(2))
    out = torch.empty_like(x0)
    for _ in range(10):
        incvit.flow_two_anchor(x0, v0, v7, al, be, b, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        incvit.flow_two_anchor(x0, v0, v7, al, be, b, out=out)
    e1.record()
    e1.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    nbytes = 5 * S * n * 4 + 2 * S * 4
    return {"samples": S, "values_per_sample": n, "us_per_launch": round(us, 3),
            "bytes_per_launch": nbytes, "achieved_gbs": round(nbytes / (us * 1e-6) / 1e9, 1),
            "note": "launch-bound at this size; back-to-back launches include the launch gap"}


def rho_sweep(steps: int, full_repeats: int) -> dict:
    """The 448x448 So400m configuration (N = 1024) under top-k refresh at every
    ratio of the sweep: graph-replayed steps over the ratio's own moving-blob
    stream against graph-replayed full encodes of the same model, and the
    break-even ratio where the step costs as much as the full encode (linear
    interpolation between the two measured ratios around it)."""
    import numpy as np
    import torch
    from paper_2607_12287_amd import incvit, synth
    dev = torch.device("cuda:0")
    enc = None
    rows = []
    for rho in synth.RHO_SWEEP:
        wl = synth.workload("so400m_448", rho=rho)
        m = wl.model
        if enc is None:  # the weights do not depend on the ratio
            enc = incvit.Encoder(m, synth.flatten_weights(m, wl.weights()), max_streams=1)
        frames = torch.from_numpy(np.stack(list(wl.patch_frames(steps + 1)))).to(dev)
        buf, caches = enc.new_caches(1)
        out = (torch.empty((1, m.n_tokens), dtype=torch.int32, device=dev),
               torch.empty((1,), dtype=torch.int32, device=dev),
               torch.empty((1, m.n_tokens, m.dim), dtype=enc.dtype, device=dev))
        inp = torch.empty_like(frames[0])
        inp.copy_(frames[0])
        gfull = enc.full_graph(inp, caches)
        full_ms = []
        for i in range(full_repeats + 3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            enc.launch(gfull)
            e1.record()
            e1.synchronize()
            if i >= 3:
                full_ms.append(e0.elapsed_time(e1))
        gstep = enc.step_graph(inp, caches, wl.tau, wl.caps, out)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for t in range(1, 4):  # warm-up
            inp.copy_(frames[t])
            enc.launch(gstep)
        torch.cuda.synchronize()
        e0.record()
        for t in range(1, steps + 1):
            inp.copy_(frames[t])
            enc.launch(gstep)
        e1.record()
        e1.synchronize()
        step_ms = e0.elapsed_time(e1) / steps
        enc.drop_graph(gstep)
        enc.drop_graph(gfull)
        full = statistics.median(full_ms)
        rows.append({"rho": rho, "rows": wl.caps[0], "step_ms": round(step_ms, 5), "full_encode_ms": round(full, 5),
                     "speedup": round(full / step_ms, 3)})
        del buf, caches, frames
    enc.close()
    even = None
    for a, b in zip(rows, rows[1:]):
        if a["speedup"] >= 1.0 >= b["speedup"] and a["speedup"] != b["speedup"]:
            f = (a["speedup"] - 1.0) / (a["speedup"] - b["speedup"])
            even = round(a["rho"] + f * (b["rho"] - a["rho"]), 4)
            break
    return {"workload": "so400m_448: 448x448 p14 N=1024 D=1152 L=27, top-k refresh, graph replay, "
                        f"{steps} steps per ratio", "sweep": rows, "break_even_rho": even}


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo) and its logical CPU count."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return f"{name} ({os.cpu_count()} logical CPUs visible)"


# The paper's own figures for this path (context, not the target): ViT latency
# of the pi0.5 pipeline without and with temporal token reuse, Table III, on
# the hardware of Appendix A.
PAPER_CONTEXT = {"vit_latency_ms_without_reuse": 40.1, "vit_latency_ms_with_token_reuse": 28.5,
                 "vit_speedup_from_reuse": 1.41, "hardware": "1x NVIDIA A100, FP16, PyTorch",
                 "workload": "LIBERO 224x224 observations inside the full VLA pipeline",
                 "source": "Table III; hardware in Appendix A"}


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
    import copy
    model = vit.Model(wl.model, wl.weights())
    caches = [vit.full_encode(model, frames[0][v]) for v in range(wl.views)]
    start = copy.deepcopy(caches)
    spent, steps = 0.0, 0
    while steps < len(frames) - 1 and (spent < seconds or steps == 0):
        t = time.perf_counter()
        for v in range(wl.views):
            vit.step(model, frames[steps + 1][v], caches[v], wl.tau, wl.caps[v])
        spent += time.perf_counter() - t
        steps += 1
    out = {"value": round(steps * wl.views / spent, 4), "unit": "frames/s", "cores": int(threads),
           "kind": "oracle", "cpu_model": cpu_model(),
           "oracle": "oracle/ as committed: numpy float64 layers (BLAS threads) and the fixed-order fp32 "
                     "embedding and cosine in C (OpenMP over tokens); not tuned for speed",
           "sample": f"{wl.name}: oracle full encode of frame 0, then {steps} incremental steps "
                     f"(frames 1..{steps}) of the same stream; value = frames / summed step time"}
    # the same steps on one thread, from a copy of the encoded caches, for
    # about a quarter of the time
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            spent1, steps1 = 0.0, 0
            while steps1 < steps and (spent1 < seconds / 4 or steps1 == 0):
                t = time.perf_counter()
                for v in range(wl.views):
                    vit.step(model, frames[steps1 + 1][v], start[v], wl.tau, wl.caps[v])
                spent1 += time.perf_counter() - t
                steps1 += 1
        out["value_1thread"] = round(steps1 * wl.views / spent1, 4)
        out["sample_1thread"] = f"frames 1..{steps1} on one thread"
    except Exception:  # pragma: no cover
        pass
    return out


def _csv_rows(directory: str, suffix: str):
    import gzip
    files = glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True)
    files += glob.glob(os.path.join(directory, "**", f"*{suffix}.gz"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    opener = gzip.open if files[0].endswith(".gz") else open
    with opener(files[0], "rt", newline="") as fh:
        return list(csv.DictReader(fh))


def _bench_json(path: str) -> dict:
    lines = [ln for ln in open(path) if ln.startswith("{")]
    return json.loads(lines[-1])


def summarize_trace(trace_dir: str, bench_log: str, plain_log: str, out: str, command: str) -> None:
    """Per-kind average dispatch duration from a rocprofv3 kernel trace of a
    bench.py run: the last n dispatches of each kind are the ones bench.py
    timed with its own per-launch events (n = its kernel_launches).  Shown next
    to bench.py's event averages in the traced run and in a run of the same
    command without the profiler (the run whose figures bench.py reports)."""
    b = _bench_json(bench_log)
    plain = _bench_json(plain_log)
    rows = sorted(_csv_rows(trace_dir, "kernel_trace.csv"), key=lambda r: int(r["Dispatch_Id"]))
    by_kind = {}
    for r, k in zip(rows, kinds_in_order([r["Kernel_Name"] for r in rows])):
        if k:
            by_kind.setdefault(k, []).append((r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3))
    stats = _csv_rows(trace_dir, "kernel_stats.csv")
    lines = [f"# rocprofv3 kernel trace of one bench.py run: {b['config']['workload']}",
             f"# command: {command}",
             f"# bench: {b['value']} {b['unit']}, {b['ms_per_step']} ms/step ({b['launch']}), "
             f"full encode {b['full_encode_ms']} ms, mean rows/step {b['config']['rows_mean']}",
             f"# same command without the profiler: {plain['value']} {plain['unit']}, {plain['ms_per_step']} ms/step, "
             f"full encode {plain['full_encode_ms']} ms",
             "# per kind: the last n dispatches (bench.py's own event-timed launches); events_traced = bench.py's",
             "# dispatch events in the traced run (the tracer delays event completion), events_plain = the same",
             "# events without the profiler; ratio = events_plain / rocprof",
             f"{'kind':8s} {'n':>7s} {'rocprof_us':>11s} {'events_traced_us':>17s} {'events_plain_us':>16s} "
             f"{'ratio':>6s}  kernel"]
    for k, n in b["kernel_launches"].items():
        d = by_kind.get(k, [])[-n:]
        if not d:
            continue
        avg = statistics.mean(x[1] for x in d)
        ev = b["kernel_us_per_launch"][k]
        evp = plain["kernel_us_per_launch"].get(k, float("nan"))
        lines.append(f"{k:8s} {n:7d} {avg:11.3f} {ev:17.3f} {evp:16.3f} {evp / avg:6.3f}  {d[-1][0]}")
    lines.append("")
    lines.append("# rocprofv3 --stats (whole run: includes the full-encode timing and warm-up dispatches)")
    lines.append(f"{'calls':>7s} {'avg_us':>10s} {'min_us':>10s} {'max_us':>10s} {'pct':>6s}  name")
    for r in stats[:24]:
        lines.append(f"{int(r['Calls']):7d} {float(r['AverageNs']) * 1e-3:10.3f} {float(r['MinNs']) * 1e-3:10.3f} "
                     f"{float(r['MaxNs']) * 1e-3:10.3f} {float(r['Percentage']):6.2f}  {r['Name'][:110]}")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _pmc_per_dispatch(directory: str, counter: str):
    vals = {}
    for r in _csv_rows(directory, "counter_collection.csv"):
        if r["Counter_Name"] == counter:
            key = (int(r["Dispatch_Id"]), r["Kernel_Name"])
            vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    return [(d, n, v) for (d, n), v in sorted(vals.items())]


def summarize_pmc(fetch_dir: str, write_dir: str, copy_fetch_dir: str, copy_write_dir: str,
                  bench_log: str, copy_log: str, out: str, commands: str) -> None:
    """HBM bytes per launch of each kernel kind from FETCH_SIZE and WRITE_SIZE
    passes (KiB per dispatch), each scaled by what the same counter reads for a
    plain device copy of known size."""
    b = _bench_json(bench_log)
    nbytes = _bench_json(copy_log)["copy_bytes"]
    scale = {}
    for name, d in (("FETCH_SIZE", copy_fetch_dir), ("WRITE_SIZE", copy_write_dir)):
        big = [v for _, n, v in _pmc_per_dispatch(d, name) if "copy" in n.lower() and v * 1024 > 0.5 * nbytes]
        if not big:
            raise RuntimeError(f"no copy dispatch with {name} near {nbytes} bytes in {d}")
        scale[name] = nbytes / (statistics.median(big) * 1024.0)
    per = {}
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        by_kind = {}
        disp = _pmc_per_dispatch(d, name)
        for (_, n, v), k in zip(disp, kinds_in_order([n for _, n, _ in disp])):
            if k:
                by_kind.setdefault(k, []).append(v)
        for k, n in b["kernel_launches"].items():
            vals = by_kind.get(k, [])[-n:]
            if vals:
                per.setdefault(k, {})[name] = statistics.mean(vals) * 1024.0 * scale[name]
    lines = [f"# HBM traffic per launch from rocprofv3 --pmc passes (workload in {b['config']['workload']})",
             f"# commands: {commands}",
             f"# mean rows/step {b['config']['rows_mean']}; per kind: mean over the last n dispatches "
             "(the incremental steps; n from the run's own launch counts)",
             f"# copy calibration ({nbytes} bytes copied): FETCH_SIZE scale {scale['FETCH_SIZE']:.4f}, "
             f"WRITE_SIZE scale {scale['WRITE_SIZE']:.4f}",
             f"source_hash {source_hash()}",
             f"# {'kind':8s} {'fetch_bytes':>14s} {'write_bytes':>14s}"]
    for k, v in per.items():
        lines.append(f"# {k:8s} {v.get('FETCH_SIZE', float('nan')):14.0f} {v.get('WRITE_SIZE', float('nan')):14.0f}")
    for k, v in per.items():
        if "FETCH_SIZE" in v and "WRITE_SIZE" in v:
            lines.append(f"traffic_bytes_per_launch {k} {v['FETCH_SIZE'] + v['WRITE_SIZE']:.0f}")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_mfma(directory: str, drive_log: str, out: str, command: str) -> None:
    """Matrix-core use per kernel kind from one rocprofv3 --pmc pass of the
    derived counters MfmaUtil (MFMA-busy cycles over active cycles x SIMDs, %)
    and MfmaFlopsBF16 (bf16 MFMA operations x 512), averaged over the last n
    dispatches of each kind (the incremental steps of the driver's run)."""
    b = _bench_json(drive_log)
    vals = {}
    for name in ("MfmaUtil", "MfmaFlopsBF16"):
        disp = _pmc_per_dispatch(directory, name)
        by_kind = {}
        for (_, n, v), k in zip(disp, kinds_in_order([n for _, n, _ in disp])):
            if k:
                by_kind.setdefault(k, []).append(v)
        for k, n in b["kernel_launches"].items():
            got = by_kind.get(k, [])[-n:]
            if got:
                vals.setdefault(k, {})[name] = statistics.mean(got)
    lines = [f"# matrix-core use per launch from rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 ({b['config']['workload']})",
             f"# command: {command}",
             f"# mean rows/step {b['config']['rows_mean']}; per kind: mean over the last n dispatches (the incremental "
             "steps); mfma_util_pct = MFMA-busy cycles / (active cycles x SIMDs); mfma_flop = bf16 MFMA operations "
             "x 512 per launch (includes the LayerNorm statistics products and the padded rows of a 32-row block)",
             f"source_hash {source_hash()}",
             f"{'kind':8s} {'mfma_util_pct':>14s} {'mfma_flop':>14s}"]
    for k, v in vals.items():
        lines.append(f"{k:8s} {v.get('MfmaUtil', float('nan')):14.3f} {v.get('MfmaFlopsBF16', float('nan')):14.0f}")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_full(trace_dir: str, pmc_dir: str, drive_log: str, out: str, command: str) -> None:
    """Full encodes of the native driver (its third argument repeats them):
    per kernel kind the mean dispatch duration of the last encode's dispatches
    (kernel trace), the matrix cores' busy fraction from the MfmaUtil counter
    pass, and for the four GEMMs the algorithmic FLOP (2 M K N, M = views x
    tokens) per launch over that duration against the dense bf16 peak."""
    b = _bench_json(drive_log)
    reps, L = b["full_encodes"], b["depth"]
    M, D, F = b["views"] * b["tokens"], b["dim"], b["mlp"]
    flop = {"qkv": 2.0 * M * D * 3 * D, "oproj": 2.0 * M * D * D, "fc1": 2.0 * M * D * F, "fc2": 2.0 * M * F * D}
    rows = sorted(_csv_rows(trace_dir, "kernel_trace.csv"), key=lambda r: int(r["Dispatch_Id"]))
    dur = {}
    for r, k in zip(rows, kinds_in_order([r["Kernel_Name"] for r in rows])):
        if k:
            dur.setdefault(k, []).append(((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3, r["Kernel_Name"]))
    util = {}
    disp = _pmc_per_dispatch(pmc_dir, "MfmaUtil")
    for (_, n, v), k in zip(disp, kinds_in_order([n for _, n, _ in disp])):
        if k:
            util.setdefault(k, []).append(v)
    for k in ("pack", "fold", "conv"):  # weight packing before the encodes
        dur.pop(k, None)
    lines = [f"# full encodes of {b['config']['workload']}: {b['views']} stream(s) x {b['tokens']} tokens = {M} rows, "
             f"D={D}, F={F}, {L} layers; last of {reps} encodes",
             f"# command: {command}",
             "# per kind: mean over the last encode's dispatches; us from the kernel trace; mfma_util_pct from the",
             "# MfmaUtil pass (busy cycles / active cycles x SIMDs); tflops = algorithmic 2 M K N / us; frac = / 2500",
             f"source_hash {source_hash()}",
             f"{'kind':8s} {'n':>4s} {'us':>9s} {'mfma_util_pct':>14s} {'tflops':>9s} {'frac':>7s}  kernel"]
    total = 0.0
    for k, d in dur.items():
        last = d[-max(1, len(d) // reps):]  # every encode launches the same kernels
        us = statistics.mean(x[0] for x in last)
        total += sum(x[0] for x in last)
        u = util.get(k, [])[-len(last):]
        tf = flop[k] / (us * 1e-6) / 1e12 if k in flop else float("nan")
        lines.append(f"{k:8s} {len(last):4d} {us:9.2f} {statistics.mean(u) if u else float('nan'):14.2f} "
                     f"{tf:9.1f} {tf / 2500.0:7.3f}  {last[-1][1][:70]}")
    lines.append(f"# summed kernel time of the last encode: {total:.1f} us")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(directory: str, drive_log: str, out: str, command: str) -> None:
    """Every counter of one rocprofv3 --pmc pass, per kernel kind: the mean per
    dispatch over the last n dispatches of each kind (the incremental steps of
    the driver's run).  SQ counters are summed over the chip's shader engines
    (cycles are counted per SIMD or per wave as the counter defines)."""
    b = _bench_json(drive_log)
    names = sorted({r["Counter_Name"] for r in _csv_rows(directory, "counter_collection.csv")})
    vals = {}
    for name in names:
        disp = _pmc_per_dispatch(directory, name)
        by_kind = {}
        for (_, n, v), k in zip(disp, kinds_in_order([n for _, n, _ in disp])):
            if k:
                by_kind.setdefault(k, []).append(v)
        for k, n in b["kernel_launches"].items():
            got = by_kind.get(k, [])[-n:]
            if got:
                vals.setdefault(k, {})[name] = statistics.mean(got)
    lines = [f"# rocprofv3 --pmc {' '.join(names)} per launch ({b['config']['workload']})",
             f"# command: {command}",
             f"# mean rows/step {b['config']['rows_mean']}; per kind: mean per dispatch over the last n dispatches "
             "(the incremental steps)",
             f"source_hash {source_hash()}",
             f"{'kind':8s} " + " ".join(f"{n:>20s}" for n in names)]
    for k, v in vals.items():
        lines.append(f"{k:8s} " + " ".join(f"{v.get(n, float('nan')):20.0f}" for n in names))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def dump_workload(name: str, rho: float, directory: str, frames: int) -> int:
    """Write a workload for the native driver (CPU only): config.txt,
    weights.bin (canonical, storage dtype) and frames.bin ([frames][views][N][P] f32)."""
    import numpy as np
    from paper_2607_12287_amd import synth
    wl = synth.workload(name, rho=rho)
    m = wl.model
    os.makedirs(directory, exist_ok=True)
    w = synth.flatten_weights(m, wl.weights())
    if m.dtype == "bf16":  # the weights are bf16 values already: keep the high halves
        w = (w.view(np.uint32) >> 16).astype(np.uint16)
    w.tofile(os.path.join(directory, "weights.bin"))
    np.stack(list(wl.patch_frames(frames))).astype(np.float32).tofile(os.path.join(directory, "frames.bin"))
    fields = [m.img_h, m.img_w, m.channels, m.patch, m.dim, m.depth, m.heads, m.mlp_dim,
              1 if m.dtype == "bf16" else 0, repr(float(m.ln_eps)), wl.views, frames, repr(float(wl.tau))]
    fields += list(wl.caps)
    with open(os.path.join(directory, "config.txt"), "w") as fh:
        fh.write(" ".join(str(x) for x in fields) + "\n")
    print(json.dumps({"workload": wl.name, "dir": directory, "frames": frames}))
    return 0


def copy_pass(mib: int) -> int:
    """A plain device-to-device copy of known size: the calibration for the HBM counters."""
    import torch
    n = mib << 20
    a = torch.full((n,), 7, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "reps": 3}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--copy-pass", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device (calibration of the HBM counters)")
    ap.add_argument("--dump-workload", metavar="DIR", help="write the workload for the native driver and exit (CPU)")
    ap.add_argument("--summarize-trace", nargs=5, metavar=("TRACE_DIR", "TRACED_BENCH_LOG", "PLAIN_BENCH_LOG", "OUT",
                                                           "COMMAND"))
    ap.add_argument("--summarize-mfma", nargs=4, metavar=("PMC_DIR", "DRIVE_LOG", "OUT", "COMMAND"))
    ap.add_argument("--summarize-full", nargs=5, metavar=("TRACE_DIR", "PMC_DIR", "DRIVE_LOG", "OUT", "COMMAND"))
    ap.add_argument("--summarize-counters", nargs=4, metavar=("PMC_DIR", "DRIVE_LOG", "OUT", "COMMAND"))
    ap.add_argument("--summarize-pmc", nargs=8, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR",
                                                         "COPY_WRITE_DIR", "BENCH_LOG", "COPY_LOG", "OUT", "COMMANDS"))
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="so400m",
                    help="so400m (default), tiny, so400m_x3, so400m_448, vitl_x8")
    ap.add_argument("--rho", type=float, default=0.10, help="refresh ratio of so400m_448 (top-k)")
    ap.add_argument("--full-repeats", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-torch-full", action="store_true", help="skip the torch full forward (context)")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel events")
    ap.add_argument("--rho-sweep", action="store_true",
                    help="only the refresh-ratio sweep of the 448x448 configuration and its break-even ratio")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the key-score and odd/even-schedule measurements")
    ap.add_argument("--eager", dest="graph", action="store_false",
                    help="launch kernel by kernel instead of replaying captured HIP graphs")
    ap.add_argument("--cols", default=None, help="column blocks per GEMM workgroup: four comma-separated values "
                                                 "(QKV, O-proj, fc1, fc2; 0 = automatic)")
    ap.add_argument("--attn-qtiles", type=int, default=0, help="16-query tiles per attention workgroup (0 = automatic)")
    ap.add_argument("--row-groups", type=int, default=0,
                    help="GEMM row groups of threshold steps (0 = ceil(mean rows / 32) of 8 calibration steps)")
    ap.add_argument("--attn-waves", type=int, default=0, help="waves per attention workgroup (0 = automatic)")
    ap.add_argument("--tiled", type=int, default=0, help="large-row GEMM for calls of 512+ known rows: "
                    "0 automatic, 1 never")
    ap.add_argument("--fc2-mode", type=int, default=0, help="MLP down projection: 1 split-K + row kernel, "
                                                            "2 unsplit with the residual in the epilogue (0 = default)")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return 0
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return 0
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return 0
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return 0
    if args.summarize_full:
        summarize_full(*args.summarize_full)
        return 0
    if args.dump_workload:
        return dump_workload(args.workload, args.rho, args.dump_workload, args.steps + 1)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the encoder's state is per stream and the library runs "
              "on one GPU only (streams would shard across GPUs with no exchange); use --gpus 1.",
              file=sys.stderr)
        return 2
    if args.copy_pass:
        return copy_pass(args.copy_pass)
    if args.rho_sweep:
        print(json.dumps(rho_sweep(min(args.steps, 30), args.full_repeats)), flush=True)
        return 0

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
    row_groups = args.row_groups
    if row_groups == 0 and math.isfinite(wl.tau):
        # a caller that knows how many rows its streams refresh sets the GEMM
        # row groups of threshold steps (the library cannot know M on the
        # host): eight eager steps on scratch caches give the mean rows
        cbuf, ccaches = enc.new_caches(B)
        enc.full_encode(frames[0], ccaches)
        seen = []
        for t in range(1, min(9, total)):
            seen.append(int(enc.step(frames[t], ccaches, wl.tau, wl.caps)[1].sum()))
        row_groups = max(1, min(8, math.ceil(statistics.mean(seen) / 32)))
        del cbuf, ccaches
    if args.cols or args.attn_qtiles or row_groups > 1 or args.attn_waves or args.fc2_mode or args.tiled:
        cols = [int(x) for x in args.cols.split(",")] if args.cols else None
        incvit._check(incvit.incvit_set_tuning(enc.h, cols, args.attn_qtiles, row_groups, args.attn_waves,
                                               args.fc2_mode, args.tiled), enc.h)
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
    approx = approx_vs_full(enc, caches, frames[total - 1])

    # the same stream again on fresh caches, each step bracketed by its own
    # events (outside the timed region above): the median and p90 of a step
    buf3, caches3 = enc.new_caches(B)
    enc.full_encode(frames[0], caches3)
    g3 = enc.step_graph(inp, caches3, wl.tau, wl.caps, out) if args.graph else None

    def step3(t):
        inp.copy_(frames[t])
        if g3 is not None:
            enc.launch(g3)
        else:
            enc.step(inp, caches3, wl.tau, wl.caps, out=out)

    for t in range(1, args.warmup + 1):
        step3(t)
    torch.cuda.synchronize()
    evs = []
    for t in range(args.warmup + 1, total):
        inp.copy_(frames[t])
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record()
        if g3 is not None:
            enc.launch(g3)
        else:
            enc.step(inp, caches3, wl.tau, wl.caps, out=out)
        a1.record()
        evs.append((a0, a1))
    torch.cuda.synchronize()
    each_ms = sorted(a0.elapsed_time(a1) for a0, a1 in evs)
    if g3 is not None:
        enc.drop_graph(g3)
    del buf3, caches3

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
                   "rows_mean": round(mean_rows, 2), "gemm_row_groups": row_groups},
        "device_ms_per_step": round(dev_ms / args.steps, 5),
        "launch": "hip-graph" if args.graph else "eager",
        "full_encode_ms": round(full_med, 5),
        "full_encode_frames_per_s": round(B * 1e3 / full_med, 2),
        "speedup_vs_full_encode": round(full_med / step_ms, 3),
        "approx_cos_vs_full": approx,
        "step_ms_dist": {"median": round(statistics.median(each_ms), 5), "p90": round(quantile(each_ms, 0.9), 5),
                         "min": round(each_ms[0], 5), "max": round(each_ms[-1], 5)},
        "full_encode_ms_dist": {"median": round(full_med, 5), "p90": round(quantile(sorted(full_ms), 0.9), 5)},
        "rows_dist": rows_dist(k),
        "paper_context": PAPER_CONTEXT,
    }
    if not args.no_torch_full:
        tms, tmode = torch_full_forward(m, wl.weights(), frames[0], max(5, args.full_repeats // 2))
        best = min(full_med, tms)
        result["torch_full_forward_ms"] = round(tms, 5)
        result["torch_full_forward_launch"] = tmode
        # the speedup against the faster of the two full re-encodes
        result["speedup_vs_best_full"] = round(best / step_ms, 3)

    if not args.no_profile:
        prof = incvit.incvit_profile_read(enc.h, reset=True)
        incvit.incvit_profile_enable(enc.h, False)
        kinds = {k: v for k, v in prof.items() if v[1] > 0}
        dom = max(kinds, key=lambda k: kinds[k][0])
        avg_us = kinds[dom][0] * 1e3 / kinds[dom][1]
        nbytes = kernel_bytes(m, mean_rows, dom)
        if dom == "attn":
            nbytes += 2 * B * m.n_tokens * m.dim * (2 if m.dtype == "bf16" else 4)
        achieved = nbytes / (avg_us * 1e-6) / 1e9 if nbytes else None
        result["roofline"] = {
            "kernel": dom, "bound": "hbm", "achieved": round(achieved, 1) if achieved else None,
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
            "traffic": stored_traffic(wl.name, dom), "avg_launch_us": round(avg_us, 3),
            "bytes_per_launch": nbytes,
        }
        # the gathered GEMMs against the dense bf16 (fp32 for fp32 models) matrix-core peak
        peak = 2500.0 if m.dtype == "bf16" else 157.3
        gm = {}
        for k in ("qkv", "oproj", "fc1", "fc2"):
            if k in kinds:
                us = kinds[k][0] * 1e3 / kinds[k][1]
                tf = gemm_flops(m, mean_rows, k) / (us * 1e-6) / 1e12
                gm[k] = {"tflops": round(tf, 2), "frac": round(tf / peak, 4), "us": round(us, 3)}
        result["gemm_mfma"] = {"peak_tflops": peak, "rows": round(mean_rows, 2), "kernels": gm,
                               "note": "weight-streaming below ~315 rows: the HBM roofline binds, not MFMA"}
        result["kernel_launches"] = {k: int(v[1]) for k, v in kinds.items()}
        result["kernel_us_per_launch"] = {k: round(v[0] * 1e3 / v[1], 3) for k, v in kinds.items()}
        result["kernel_ms_per_step"] = {k: round(v[0] / args.steps, 5) for k, v in kinds.items()}
    del buf2, caches2

    if not args.no_variants:
        # the paper's own score (first-layer keys, eq. 3) on the rolling stream,
        # and its odd/even chunk schedule (period 2) with that score
        vsteps, vwarm = min(args.steps, 200), min(args.warmup, 20)
        result["variants"] = [measure_variant(wl, frames, "key", p, vsteps, vwarm, args.full_repeats)
                              for p in (0, 2)]
        # the non-exact reading of the MLP over all tokens (embedding score)
        result["variants"].append(measure_variant(wl, frames, "embed", 0, vsteps, vwarm, args.full_repeats,
                                                  mlp="all"))

    if not args.no_variants:
        result["flow_two_anchor"] = measure_flow(64, 50 * 32)

    if not args.no_cpu_baseline:
        n_cpu = min(len(frames_np), 64)
        result["cpu_baseline"] = cpu_baseline(wl, frames_np[:n_cpu], args.cpu_seconds)

    result["env"] = run_env(torch)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
