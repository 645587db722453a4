"""Benchmark of the streaming Token2Wav decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one chunk step of the whole decode path (embedding, pre-stack,
upsampling stages with their resblocks, head, inverse STFT) for every stream
of the workload, replayed as one HIP graph through the C ABI.  For a flow
workload (--workload flow_*) a step is one flow-decoder call of f_call frames
for every stream (n_steps guided Euler steps of the DiT estimator over the
carried attention state), also one graph replay; it yields f_chunk new frames
per stream, f_chunk / 50 seconds of audio at the 50 Hz frame clock.  Token chunks
are resident in HBM before the timed region; each step stages its chunk into
the state's token buffer (counted in the step) and leaves the PCM in the
state's audio buffer.  Prints one JSON line:

  value        audio-seconds decoded per wall-second (streams * samples / 24 kHz)
  ms_per_step  wall milliseconds per chunk step in the timed loop
  p50/p99      per-chunk latency: host wall time of dc_decode_chunk with host
               token and PCM buffers (synchronous call: token upload, graph
               replay, PCM download); the same for device-resident buffers and
               the HIP-event device time of one replay are reported beside it
  roofline     the kernel with the largest share of step time, its algorithmic
               FLOPs (or bytes) per launch over its mean launch duration, timed
               with HIP events on the state's stream
               and against peaks measured on this device (a device copy and
               library GEMMs), beside the datasheet ones
  cpu_baseline the plain fp64 oracle on the host cores, on a bounded sample
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "audio-seconds decoded per wall-second (1 GPU) + p50 per-chunk latency ms"
PROFILES = os.path.join(ROOT, "profiles")
# rocprofv3 PMC counters against a plain 256 MiB device copy on MI355X: FETCH_SIZE
# reads half the bytes the copy moves, WRITE_SIZE all of them.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
DEFAULT_WORKLOAD = "real_f32_b1_n25"
RNG_SEED = 11   # key of the harmonic source's generator (workloads with a source)
PEAK = {"hbm": 8000.0, "bf16": 2500.0, "f32": 157.3}   # GB/s, TFLOP/s (MI355X, dense)


class _Addr:
    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr


def cpu_baseline(arch, dtype, blob, tokens, budget_s: float, f0=None, streams=(0,), max_tokens=None):
    """Time the oracle (as it stands) decoding a prefix of each stream in
    `streams` (budget_s split evenly between them), growing the prefix until
    one run takes its share of the budget or the workload's tokens (or
    max_tokens) run out.  Returns the baseline record and each stream's
    oracle PCM of its prefix (the parity reference on the same subset)."""
    import oracle
    from paper_2609_35115_amd import synth
    spt = synth.samples_per_token(arch)
    fpt = arch["frames_per_token"]
    T_full = tokens.shape[1] if max_tokens is None else min(tokens.shape[1], max_tokens)
    share = budget_s / len(streams)
    total_audio, total_wall, refs, parts = 0.0, 0.0, {}, []
    for b in streams:
        T = min(T_full, 4)
        while True:
            t0 = time.perf_counter()
            if f0 is None:
                ref = oracle.decode(arch, dtype, blob, tokens[b, :T])
            else:
                ref = oracle.decode(arch, dtype, blob, tokens[b, :T], f0=f0[b, :T * fpt], seed=RNG_SEED, stream=b)
            dt = time.perf_counter() - t0
            if dt >= share or T >= T_full:
                break
            T = min(T_full, max(2 * T, int(T * share / max(dt, 1e-3) * 1.05)))
        total_audio += T * spt / synth.SAMPLE_RATE
        total_wall += dt
        refs[b] = ref
        parts.append(f"{b}: [0,{T})")
    rec = {"value": total_audio / total_wall, "unit": "audio-s/s", "cores": oracle.num_threads(),
           "kind": "oracle",
           "sample": f"stream{'s' if len(streams) > 1 else ''} {', '.join(parts)} of the workload's tokens decoded "
                     f"offline in fp64{' on bf16-rounded weights' if dtype == 'bf16' else ''}, "
                     f"{total_wall:.1f} s wall"}
    return rec, refs


FLOW_FRAME_RATE = 50.0   # frames per second of audio: 2 frames per 25 Hz token
FLOW_SOURCES = ("flow_kernels.hip", "flow_internal.h")


def kernel_source_hash(files=("dc_kernels.hip", "dc_internal.h")) -> str:
    """Hash of the kernel sources: a traffic figure taken on other sources is stale."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2609_35115_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profiles(workload: str, kernel: str, files=("dc_kernels.hip", "dc_internal.h")):
    """HBM bytes per launch of `kernel` recorded under profiles/ for this workload
    with the current kernel sources, else None."""
    path = os.path.join(PROFILES, f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    if rec.get("kernel_source_hash") != kernel_source_hash(files):
        return None
    if rec.get("kernel") == kernel:
        return float(rec["hbm_bytes_per_launch"])
    # the other kernels of the same runs (which kernel dominates a step can
    # change between runs when two take about the same time)
    for line in open(path):
        if line.startswith(f"hbm_bytes_per_launch[{kernel}]:"):
            return float(line.rsplit(":", 1)[1])
    return None


def roofline(layers, us, dtype):
    """Group launches by kernel; the one with the most time per step is reported."""
    groups = {}
    for info, t in zip(layers, us):
        g = groups.setdefault(info["kernel"], {"us": 0.0, "flops": 0.0, "bytes": 0.0, "launches": 0})
        g["us"] += t
        g["flops"] += info["flops"]
        g["bytes"] += info["bytes"]
        g["launches"] += 1
    name, g = max(groups.items(), key=lambda kv: kv[1]["us"])
    step_us = sum(us)
    conv = name.startswith(("dc::conv_kernel", "dc::wconv_kernel", "dc::pair_kernel"))   # MFMA kernels
    op = "bf16" if "<true" in name or name.startswith(("dc::pair_kernel", "dc::wconv_kernel")) else "f32"
    if conv and g["flops"] / g["bytes"] > PEAK[op] * 1e12 / (PEAK["hbm"] * 1e9):
        bound, achieved, peak, unit = "mfma", g["flops"] / (g["us"] * 1e-6) / 1e12, PEAK[op], "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", g["bytes"] / (g["us"] * 1e-6) / 1e9, PEAK["hbm"], "GB/s"
    per_kernel = sorted(((k, v["us"] / step_us) for k, v in groups.items()), key=lambda kv: -kv[1])
    src = None
    if "dc::source_kernel" in groups:
        sg, pg = groups["dc::source_kernel"], groups.get("dc::phase_kernel", {"us": 0.0})
        src = {"source_kernel_us": round(sg["us"], 3), "phase_kernel_us": round(pg["us"], 3),
               "share_of_step": round((sg["us"] + pg["us"]) / step_us, 4)}
    return {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": None,
            "kernel": name, "operand": op, "launches_per_step": g["launches"],
            "mean_launch_us": round(g["us"] / g["launches"], 3),
            "flops_per_launch": g["flops"] / g["launches"], "bytes_per_launch": g["bytes"] / g["launches"],
            "share_of_step": round(g["us"] / step_us, 4),
            "kernels_by_share": [[k, round(v, 4)] for k, v in per_kernel[:6]], "source": src}


def calibrate_copy():
    """A plain device copy of 256 MiB, three times (the counter calibration run)."""
    import torch
    n = 256 << 20
    a = torch.ones(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {n} bytes 3 times", flush=True)


def calibrate_read():
    """A read-only pass over 256 MiB, three times (torch's sum of 64 Mi floats):
    checks the FETCH_SIZE factor of the copy calibration on a kernel that
    writes nothing but its partial sums."""
    import torch
    x = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    for _ in range(3):
        s = x.sum()
    torch.cuda.synchronize()
    print(f"read {x.numel() * 4} bytes 3 times (sum {float(s)})", flush=True)


def measured_peaks():
    """Achievable rates on this device: a 1 GiB device copy (read + write bytes)
    and 8192^3 library GEMMs in bf16 and fp32, best of several timed runs."""
    import torch
    out = {}
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def best(fn, reps):
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            ev[0].record()
            fn()
            ev[1].record()
            ev[1].synchronize()
            t.append(ev[0].elapsed_time(ev[1]) * 1e-3)
        return min(t)

    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    out["hbm_copy_GBs"] = round(2 * n / best(lambda: b.copy_(a), 10) / 1e9, 1)
    del a, b
    m = 8192
    for name, dt, reps in (("bf16_gemm_TFLOPs", torch.bfloat16, 10), ("f32_gemm_TFLOPs", torch.float32, 5)):
        x = torch.randn(m, m, device="cuda").to(dt)
        y = torch.randn(m, m, device="cuda").to(dt)
        out[name] = round(2 * m ** 3 / best(lambda: torch.mm(x, y), reps) / 1e12, 1)
        del x, y
    torch.cuda.empty_cache()
    return out


def _csv(path):
    import csv
    with open(path) as fh:
        return list(csv.DictReader(fh))


def _sources_for(path: str):
    """The kernel sources a profile of this workload covers (flow workloads: the flow kernels)."""
    return FLOW_SOURCES if "flow_" in os.path.basename(path) else ("dc_kernels.hip", "dc_internal.h")


def summarize_stats(prof_dir: str, out: str, command: str):
    """Text summary of a rocprofv3 --kernel-trace --stats --output-format csv run."""
    import glob
    rows = _csv(glob.glob(os.path.join(prof_dir, "**", "*kernel_stats.csv"), recursive=True)[0])
    lines = [f"# rocprofv3 kernel statistics", f"# command: {command}",
             f"# kernel sources: {kernel_source_hash(_sources_for(out))}", "",
             f"{'kernel':64s} {'calls':>7s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'total_ms':>9s} {'pct':>6s}"]
    for r in rows:
        name = r["Name"].replace("void ", "")
        name = name[:name.index("(")] if "(" in name else name
        lines.append(f"{name[:64]:64s} {int(r['Calls']):7d} {float(r['AverageNs'])/1e3:9.3f} "
                     f"{float(r['MinNs'])/1e3:9.3f} {float(r['MaxNs'])/1e3:9.3f} "
                     f"{float(r['TotalDurationNs'])/1e6:9.3f} {float(r['Percentage']):6.2f}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_traffic(fetch_dir: str, write_dir: str, workload: str, kernel: str, out: str, command: str):
    """Mean HBM bytes per dispatch of `kernel` from FETCH_SIZE and WRITE_SIZE runs."""
    import glob
    def per_kernel(d, counter):
        rows = _csv(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0])
        vals, grid = {}, {}
        for r in rows:
            name = r["Kernel_Name"].replace("void ", "")
            name = name[:name.index("(")] if "(" in name else name
            if r["Counter_Name"] == counter and name.startswith(("dc::", "dcf::")):
                i = int(r["Dispatch_Id"])
                vals.setdefault(name, {})
                vals[name][i] = vals[name].get(i, 0.0) + float(r["Counter_Value"])
                grid.setdefault(name, {})[i] = int(r["Grid_Size"])
        return vals, grid
    def mean_kib(tables, name):
        vals, grid = tables[0][name], tables[1][name]
        if workload.startswith("flow_"):
            # the timed calls' launches only: the prompt passes that set up
            # the streams run the same kernels over other row counts
            g_last = grid[max(grid)]
            vals = {i: v for i, v in vals.items() if grid[i] == g_last}
        return sum(vals.values()) / len(vals), len(vals), grid[max(grid)]
    ft, wt = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    f, nf, g = mean_kib(ft, kernel)
    w, nw, _ = mean_kib(wt, kernel)
    hbm = (f * FETCH_SCALE + w * WRITE_SCALE) * 1024.0
    others = []
    for name in sorted(set(ft[0]) & set(wt[0])):
        if name != kernel:
            fo, wo = mean_kib(ft, name)[0], mean_kib(wt, name)[0]
            others.append(f"hbm_bytes_per_launch[{name}]: {(fo * FETCH_SCALE + wo * WRITE_SCALE) * 1024.0:.0f}")
    lines = ["# HBM traffic per launch from rocprofv3 PMC counters", f"# command: {command}",
             f"# FETCH_SIZE x {FETCH_SCALE} + WRITE_SIZE x {WRITE_SCALE} (KiB per dispatch; scale factors from a "
             "plain 256 MiB device copy: python3 bench.py --calibrate-copy)",
             f"workload: {workload}", f"kernel: {kernel}", f"kernel_source_hash: {kernel_source_hash(_sources_for(out))}",
             f"dispatches: {nf} / {nw}" + (f" (grid size {g}: the timed calls' launches)" if workload.startswith("flow_") else ""),
             f"fetch_kib_per_dispatch: {f:.1f}", f"write_kib_per_dispatch: {w:.1f}",
             f"hbm_bytes_per_launch: {hbm:.0f}"]
    if others:
        lines += ["# the run's other kernels, the same measure"] + others
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_mfma(prof_dir: str, workload: str, out: str, command: str):
    """Per-kernel MFMA counters of a rocprofv3 --pmc run (one row per dispatch
    and counter, values summed over the device's XCDs)."""
    import glob
    rows = _csv(glob.glob(os.path.join(prof_dir, "**", "*counter_collection.csv"), recursive=True)[0])
    per = {}
    for r in rows:
        name = r["Kernel_Name"].replace("void ", "")
        name = name[:name.index("(")] if "(" in name else name
        if not name.startswith(("dc::", "dcf::")):
            continue
        d = per.setdefault(name, {}).setdefault(r["Dispatch_Id"], {})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    xcds, simds = 8, 1024
    lines = ["# MFMA counters per kernel from rocprofv3 PMC counters", f"# command: {command}",
             f"# workload: {workload}", f"# kernel sources: {kernel_source_hash(_sources_for(out))}",
             "# mfma_flops = (SQ_INSTS_VALU_MFMA_MOPS_BF16 + SQ_INSTS_VALU_MFMA_MOPS_F32) * 512 per dispatch",
             "# mfma_util  = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs * 1024 SIMDs); for dispatches "
             "of a few microseconds GRBM_GUI_ACTIVE also counts the collection window, so it reads low there",
             "# us = mean dispatch duration under counter collection (dispatches are serialised)", "",
             f"{'kernel':48s} {'disp':>5s} {'us':>8s} {'mfma_GFLOP':>11s} {'TFLOP/s':>8s} {'util%':>6s}"]
    tot = []
    for name, ds in per.items():
        n = len(ds)
        us = sum(d["ns"] for d in ds.values()) / n / 1e3
        fl = sum((d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) + d.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0)) * 512
                 for d in ds.values()) / n
        busy = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) for d in ds.values())
        gui = sum(d.get("GRBM_GUI_ACTIVE", 0) for d in ds.values()) / xcds
        tot.append((us * n, f"{name[:48]:48s} {n:5d} {us:8.2f} {fl / 1e9:11.3f} {fl / (us * 1e-6) / 1e12:8.1f} "
                            f"{100.0 * busy / max(gui * simds, 1.0):6.1f}"))
    lines += [l for _, l in sorted(tot, key=lambda t: -t[0])]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


FLOW_GEMM = {   # role -> (epilogue, LayerNorm operand) of the GEMM that runs it
    "gemm:in": (0, False), "gemm:qkv": (1, True), "gemm:o": (2, False), "gemm:fc2": (2, False),
    "gemm:fc1": (3, True), "gemm:out": (4, True),
}
SKINNY_ROWS = 512   # calls of at most this many rows (2 per stream and frame) run the skinny GEMM
SKINNY_LN = (8, 2, 1)   # LayerNorm-operand skinny GEMM: waves, 16-column blocks, 16-row blocks per block


ATTN_WIDE_BLOCKS = 64   # (stream, branch, head) x 64-query blocks from which attention takes its wide shape


TILE_BIG_BLOCKS = 1024   # 64 x 64 tiles of a GEMM from which the tiled kernel takes 128 x 128
TILE_MID_BLOCKS = 256    # ... and from which it takes 128 rows x 64 columns


def flow_kernel_name(role: str, dtype: str, rows: int, attn_blocks: int = 0, arch: dict | None = None) -> str:
    b = "true" if dtype == "bf16" else "false"
    if role == "attn":
        return f"dcf::attn_kernel<{b}, 4, 8>" if attn_blocks >= ATTN_WIDE_BLOCKS else f"dcf::attn_kernel<{b}, 1, 4>"
    if role in FLOW_GEMM:
        epi, ln = FLOW_GEMM[role]
        D = arch["dim"] if arch else 512
        N, K = {"gemm:in": (D, 4 * (arch["n_mel"] if arch else 80)), "gemm:qkv": (3 * D, D), "gemm:o": (D, D),
                "gemm:fc1": (arch["mlp"] if arch else 2048, D), "gemm:fc2": (D, arch["mlp"] if arch else 2048),
                "gemm:out": (arch["n_mel"] if arch else 80, D)}[role]
        if rows <= SKINNY_ROWS:
            if ln:
                waves, nblk, rb = SKINNY_LN if K % (16 * SKINNY_LN[0] // SKINNY_LN[2]) == 0 else (4, SKINNY_LN[1], 1)
            else:
                waves, nblk, rb = (8 if K >= 1024 else 4), 1, 1
            return f"dcf::skinny_kernel<{b}, {epi}, {'true' if ln else 'false'}, {waves}, {nblk}, {rb}>"
        blocks = ((N + 63) // 64) * ((rows + 63) // 64)
        tile = "4, 4" if blocks >= TILE_BIG_BLOCKS else "4, 2" if blocks >= TILE_MID_BLOCKS else "1, 1"
        return f"dcf::gemm_kernel<{b}, {epi}, {tile}>"
    return f"dcf::{role}_kernel<{b}>" if role in ("assemble", "euler") else role


def flow_roofline(prof, dtype, rows, attn_blocks, arch):
    """The role with the most device time per call, against its bound."""
    step_us = sum(r["us"] for r in prof)
    top = max(prof, key=lambda r: r["us"])
    op = "bf16" if dtype == "bf16" else "f32"
    if top["mfma"] and top["flops"] / top["bytes"] > PEAK[op] * 1e12 / (PEAK["hbm"] * 1e9):
        bound, achieved, peak, unit = "mfma", top["flops"] / (top["us"] * 1e-6) / 1e12, PEAK[op], "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", top["bytes"] / (top["us"] * 1e-6) / 1e9, PEAK["hbm"], "GB/s"
    kern = flow_kernel_name(top["name"], dtype, rows, attn_blocks, arch)
    return {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": None, "kernel": kern, "role": top["name"],
            "operand": op, "launches_per_step": top["launches"],
            "mean_launch_us": round(top["us"] / top["launches"], 3),
            "flops_per_launch": top["flops"] / top["launches"], "bytes_per_launch": top["bytes"] / top["launches"],
            "share_of_step": round(top["us"] / step_us, 4),
            "kernels_by_share": [[r["name"], round(r["us"] / step_us, 4)]
                                 for r in sorted(prof, key=lambda r: -r["us"])[:6]],
            "step_us_launch_by_launch": round(step_us, 2)}


def flow_cpu_baseline(arch, dtype, blob, budget_s: float, prompt_frames: int = 64):
    """The oracle on stream 0: a short prompt (untimed), then chunk calls of
    f_call frames until one budget's worth of time has passed."""
    import oracle
    from paper_2609_35115_amd import synth
    fc, fcall = arch["f_chunk"], arch["f_call"]
    P = min(prompt_frames, arch["f_prompt"])
    s = oracle.FlowStream(arch, dtype, blob, seed=RNG_SEED, key=0)
    s.prompt(*synth.make_flow_prompt(arch, P))
    mu = synth.make_flow_mu(arch, 1, 64 * fc + fcall)[0]
    calls, t0 = 0, time.perf_counter()
    while True:
        s.chunk(mu[calls * fc:calls * fc + fcall])
        calls += 1
        dt = time.perf_counter() - t0
        if dt >= budget_s or calls >= 64:
            break
    return {"value": calls * fc / FLOW_FRAME_RATE / dt, "unit": "audio-s/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"stream 0, {calls} chunk calls of {fcall} frames after a {P}-frame prompt (untimed), "
                      f"fp64{' on bf16-rounded weights' if dtype == 'bf16' else ''}, {dt:.1f} s wall"}


def bench_flow(args):
    import numpy as np
    import torch

    from paper_2609_35115_amd import flow, synth

    w = synth.workload(args.workload)
    arch, dtype, B, chunks = w["arch"], w["dtype"], w["batch"], w["chunks"]
    fc, fcall, P, M = arch["f_chunk"], arch["f_call"], arch["f_prompt"], arch["n_mel"]
    torch.cuda.set_device(0)
    blob = synth.make_flow_weights(arch, 0)
    prompts = [synth.make_flow_prompt(arch, P, stream=b) for b in range(B)]
    mu = synth.make_flow_mu(arch, B, chunks * fc + fcall)
    mu_dev = torch.from_numpy(np.ascontiguousarray(np.stack([mu[:, k * fc:k * fc + fcall] for k in range(chunks)]))).cuda()
    mel = torch.empty((B, fcall, M), dtype=torch.float32, device="cuda")
    dec = flow.FlowDecoder(arch, dtype, blob, B, rng_seed=RNG_SEED)
    for b in range(B):
        dec.prompt(b, *prompts[b])
    dec.sync()
    torch.cuda.synchronize()

    def step(d, i):
        st = flow.dc_flow_decode_chunk(d.h, mu_dev[i % chunks], fcall, mel)
        if st != 0:
            raise RuntimeError(flow.dc_flow_last_error(d.h))

    print(f"# workload {args.workload}: batch {B}, f_call {fcall}, f_chunk {fc}, {dtype}; warmup {args.warmup}, "
          f"steps {args.steps}", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(dec, i)
    dec.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(dec, args.warmup + i)
    dec.stream.synchronize()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dec.sync()
    ms_per_step = 1000.0 * wall / args.steps
    audio_s = B * fc / FLOW_FRAME_RATE
    value = audio_s * args.steps / wall
    print(f"# timed {args.steps} steps in {wall:.3f} s", file=sys.stderr, flush=True)
    if args.only_steps:
        dec.close()
        print(json.dumps({"workload": args.workload, "steps": args.steps, "ms_per_step": round(ms_per_step, 4)}),
              flush=True)
        return

    lat_dev, lat_ev = [], []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for i in range(args.latency_chunks):
        t = time.perf_counter()
        ev[0].record(dec.stream)
        step(dec, i)
        ev[1].record(dec.stream)
        dec.stream.synchronize()
        lat_dev.append(1000.0 * (time.perf_counter() - t))
        lat_ev.append(ev[0].elapsed_time(ev[1]))
    prof = dec.profile(args.layer_reps)
    roof = flow_roofline(prof, dtype, B * 2 * fcall, B * 2 * arch["heads"] * ((fcall + 63) // 64), arch)
    roof["traffic"] = traffic_from_profiles(args.workload, roof["kernel"], FLOW_SOURCES)
    stats = dec.stats()
    dec.close()

    hdec = flow.FlowDecoder(arch, dtype, blob, B, flags=flow.DC_HOST_PTRS, rng_seed=RNG_SEED)
    for b in range(B):
        hdec.prompt(b, *prompts[b])
    host_mu = [np.ascontiguousarray(mu[:, k * fc:k * fc + fcall]) for k in range(chunks)]
    out = np.empty((B, fcall, M), dtype=np.float32)
    lat = []
    for i in range(min(args.warmup, 5) + args.latency_chunks):
        t = time.perf_counter()
        st = flow.dc_flow_decode_chunk(hdec.h, host_mu[i % chunks], fcall, out)
        dt = 1000.0 * (time.perf_counter() - t)
        if st != 0:
            raise RuntimeError(flow.dc_flow_last_error(hdec.h))
        if i >= min(args.warmup, 5):
            lat.append(dt)
    hdec.close()

    if not args.skip_peaks:
        peaks = measured_peaks()
        key = "hbm_copy_GBs" if roof["bound"] == "hbm" else f"{roof['operand']}_gemm_TFLOPs"
        roof["measured_peak"] = peaks[key]
        roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks[key], 4)
        roof["measured_peaks"] = peaks
    print(f"# roofline: {roof['kernel']} ({roof['role']}) {roof['achieved']} {roof['unit']} ({roof['frac']:.1%})",
          file=sys.stderr, flush=True)
    cpu = flow_cpu_baseline(arch, dtype, blob, args.cpu_budget) if args.cpu_budget > 0 else None
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "audio-s/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic (seeded random-weight DiT flow decoder, N(0,1) encoder features, synthetic prompts)",
        "config": {"workload": args.workload, "stage": "flow decoder",
                   "arch": "real" if arch["dim"] == 512 else "tiny", "batch": B, "f_call": fcall, "f_chunk": fc,
                   "f_prompt": P, "f_retained": arch["f_retained"], "n_steps": arch["n_steps"],
                   "chunks_cycled": chunks, "audio_s_per_step": audio_s, "graph_replay": stats["replays"] > 0,
                   "kernels_per_step": stats["kernels_per_call"],
                   "flops_per_step": sum(r["flops"] for r in prof),
                   "carry_bytes": stats["carry_bytes"], "carry_live_bytes": stats["carry_live_bytes"]},
        "p50_chunk_ms": round(float(np.percentile(lat, 50)), 4),
        "p99_chunk_ms": round(float(np.percentile(lat, 99)), 4),
        "latency_path": "host mu in, host mel out, synchronous dc_flow_decode_chunk",
        "p50_chunk_ms_device_buffers": round(float(np.percentile(lat_dev, 50)), 4),
        "p99_chunk_ms_device_buffers": round(float(np.percentile(lat_dev, 99)), 4),
        "p50_replay_ms_hip_events": round(float(np.percentile(lat_ev, 50)), 4),
        "capture_ms": round(stats["capture_ms"], 3),
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize-mfma":
        return summarize_mfma(*sys.argv[2:6])
    if len(sys.argv) > 1 and sys.argv[1] == "--calibrate-copy":
        return calibrate_copy()
    if len(sys.argv) > 1 and sys.argv[1] == "--calibrate-read":
        return calibrate_read()
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize-stats":
        return summarize_stats(sys.argv[2], sys.argv[3], sys.argv[4])
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize-traffic":
        return summarize_traffic(*sys.argv[2:8])
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--latency-chunks", type=int, default=100)
    ap.add_argument("--layer-reps", type=int, default=10)
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of one oracle run (0 skips it)")
    ap.add_argument("--tile-variant", type=int, default=0)
    ap.add_argument("--skip-peaks", action="store_true", help="skip the device copy and GEMM peak runs "
                    "(for profiler runs; the roofline then has no measured-peak fraction)")
    ap.add_argument("--no-configs", action="store_true", help="time only the named workload (by default the "
                    "headline workload is followed by the other configurations in a 'configs' object)")
    ap.add_argument("--only-steps", action="store_true", help="flow workloads: run the warmup and timed steps only "
                    "and print their timing (for hardware-counter runs, which serialise every dispatch)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (--gpus {args.gpus} requested). Streams are "
              "independent, so a multi-GPU deployment runs one state per GPU with no collectives; "
              "run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.workload.startswith("flow_"):
        return bench_flow(args)

    peaks = None if args.skip_peaks else measured_peaks()
    out = bench_vocoder(args.workload, args.steps, args.warmup, args, peaks, headline=True)
    if not args.no_configs and args.workload == DEFAULT_WORKLOAD:
        out["configs"] = {}
        for name, (steps, warmup, latency) in CONFIG_RUNS.items():
            out["configs"][name] = bench_vocoder(name, steps, warmup, args, peaks, latency_chunks=latency)
    print(json.dumps(out), flush=True)


# The other configurations timed beside the headline (steps, warmup, latency
# calls): the tiny decoder, batch 16, the 4-token chunk, batch 128.
CONFIG_RUNS = {
    "tiny_f32_b1_n8": (200, 8, 100),
    "real_bf16_b16_n25": (100, 20, 50),
    "real_bf16_b1_n4": (400, 50, 200),
    "real_bf16_b128_n25": (40, 20, 20),
}
# Oracle subsets of the CPU baseline and the parity check (streams of each
# workload): the batch-16 and batch-128 workloads on three and two streams.
CPU_STREAMS = {"real_bf16_b16_n25": (0, 7, 15), "real_bf16_b128_n25": (0, 127), "real_bf16_b16_n25_nsf": (0, 7, 15)}


def bench_vocoder(name, steps, warmup, args, peaks, headline=False, latency_chunks=None):
    """Time one vocoder workload; returns its record (the headline fields, or
    the per-configuration fields for a non-headline workload)."""
    import numpy as np
    import torch

    import paper_2609_35115_amd as dc
    from paper_2609_35115_amd import synth

    w = synth.workload(name)
    arch, dtype, B, n, chunks = w["arch"], w["dtype"], w["batch"], w["chunk_tokens"], w["chunks"]
    spt = synth.samples_per_token(arch)
    fpt = arch["frames_per_token"]
    has_src = arch.get("n_harmonics", 0) > 0
    latency_chunks = args.latency_chunks if latency_chunks is None else latency_chunks
    torch.cuda.set_device(0)
    blob = synth.make_weights(arch, 0)
    tokens = synth.make_tokens(arch, B, chunks * n)
    tok_dev = torch.from_numpy(np.ascontiguousarray(tokens.reshape(B, chunks, n).transpose(1, 0, 2))).cuda()
    f0 = f0_dev = None
    if has_src:   # the source's f0 contour, resident like the tokens
        f0 = synth.make_f0(arch, B, chunks * n)
        f0_dev = torch.from_numpy(np.ascontiguousarray(f0.reshape(B, chunks, n * fpt).transpose(1, 0, 2))).cuda()
    dec = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, tile_variant=args.tile_variant, rng_seed=RNG_SEED)
    audio = _Addr(dc.dc_audio_buffer(dec.h))
    torch.cuda.synchronize()

    def step(i):
        if has_src:
            st = dc.dc_decode_chunk_f0(dec.h, tok_dev[i % chunks], f0_dev[i % chunks], n, audio)
        else:
            st = dc.dc_decode_chunk(dec.h, tok_dev[i % chunks], n, audio)
        if st != dc.DC_OK:
            raise dc.DcError(st, dc.dc_last_error(dec.h))

    print(f"# workload {name}: batch {B}, chunk {n} tokens, {dtype}; warmup {warmup}, steps {steps}",
          file=sys.stderr, flush=True)
    # warmup: the first chunks of every stream from the start, replayed like
    # the timed steps; the PCM of the oracle subset's streams is kept for the
    # parity check
    cpu_streams = CPU_STREAMS.get(name, (0,))
    sel = torch.tensor(cpu_streams, device="cuda")
    kept = []
    for i in range(warmup):
        if has_src:
            out_i = dec.decode(tok_dev[i % chunks], f0_dev[i % chunks])
        else:
            out_i = dec.decode(tok_dev[i % chunks])
        if i < chunks:
            kept.append(out_i.index_select(0, sel))
    dec.sync()
    kept = torch.cat(kept, dim=1).cpu().numpy() if kept else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(warmup + i)
    dec.stream.synchronize()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dec.sync()
    ms_per_step = 1000.0 * wall / steps
    audio_s = B * n * spt / synth.SAMPLE_RATE
    value = audio_s * steps / wall
    print(f"# timed {steps} steps in {wall:.3f} s", file=sys.stderr, flush=True)

    # device-resident buffers: submit, then wait for the PCM on the device
    lat_dev, lat_ev = [], []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for i in range(latency_chunks):
        t = time.perf_counter()
        ev[0].record(dec.stream)
        step(i)
        ev[1].record(dec.stream)
        dec.stream.synchronize()
        lat_dev.append(1000.0 * (time.perf_counter() - t))
        lat_ev.append(ev[0].elapsed_time(ev[1]))
    dec.sync()

    layers = dec.layers()
    us = dec.time_layers(args.layer_reps)
    roof = roofline(layers, us, dtype)
    roof["traffic"] = traffic_from_profiles(name, roof["kernel"])
    flops_step = sum(l["flops"] for l in layers)
    op = "bf16" if dtype == "bf16" else "f32"
    # the whole step against the MFMA peak of its operand type: step FLOPs over
    # the timed loop's wall time per step
    roof["step"] = {"achieved": round(flops_step / (ms_per_step * 1e-3) / 1e12, 2), "peak": PEAK[op],
                    "unit": "TFLOP/s", "frac": round(flops_step / (ms_per_step * 1e-3) / 1e12 / PEAK[op], 4)}
    stats = dec.stats()
    dec.close()
    del tok_dev, f0_dev
    torch.cuda.empty_cache()

    # host buffers: dc_decode_chunk uploads the tokens, replays the step and
    # returns once the PCM is in host memory
    hdec = dc.Decoder(arch, dtype, blob, batch=B, chunk_tokens=n, flags=dc.DC_HOST_PTRS,
                      tile_variant=args.tile_variant, rng_seed=RNG_SEED)
    pcm = np.empty((B, n * spt), dtype=np.float32)
    host_tok = [np.ascontiguousarray(tokens[:, c * n:(c + 1) * n]) for c in range(chunks)]
    host_f0 = [np.ascontiguousarray(f0[:, c * n * fpt:(c + 1) * n * fpt]) for c in range(chunks)] if has_src else None
    lat = []
    for i in range(min(warmup, 20) + latency_chunks):
        t = time.perf_counter()
        if has_src:
            st = dc.dc_decode_chunk_f0(hdec.h, host_tok[i % chunks], host_f0[i % chunks], n, pcm)
        else:
            st = dc.dc_decode_chunk(hdec.h, host_tok[i % chunks], n, pcm)
        dt = 1000.0 * (time.perf_counter() - t)
        if st != dc.DC_OK:
            raise dc.DcError(st, dc.dc_last_error(hdec.h))
        if i >= min(warmup, 20):
            lat.append(dt)
    hdec.close()

    if peaks is not None:
        key = "hbm_copy_GBs" if roof["bound"] == "hbm" else f"{roof['operand']}_gemm_TFLOPs"
        roof["measured_peak"] = peaks[key]
        roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks[key], 4)
        if headline:
            roof["measured_peaks"] = peaks
    print(f"# roofline: {roof['kernel']} {roof['achieved']} {roof['unit']} ({roof['frac']:.1%}); "
          f"step {roof['step']['achieved']} TFLOP/s ({roof['step']['frac']:.1%})", file=sys.stderr, flush=True)

    cpu = parity = None
    if args.cpu_budget > 0:
        cpu, refs = cpu_baseline(arch, dtype, blob, tokens, args.cpu_budget, f0, streams=cpu_streams,
                                 max_tokens=min(warmup, chunks) * n)
        # the GPU's replayed warmup chunks against the oracle on the same subset
        tol = 1e-4 if dtype == "f32" else 2e-2
        worst = 0.0
        for j, b in enumerate(cpu_streams):
            ref = refs[b]
            got = kept[j, :ref.size].astype(np.float64)
            e = float(np.abs(got - ref).max() / np.sqrt(np.mean(ref ** 2)))
            worst = max(worst, e)
        parity = {"streams": list(cpu_streams), "samples_per_stream": [int(refs[b].size) for b in cpu_streams],
                  "max_abs_err_over_rms": round(worst, 6), "tolerance": tol, "ok": worst <= tol}

    lat_fields = {
        "p50_chunk_ms": round(float(np.percentile(lat, 50)), 4),
        "p99_chunk_ms": round(float(np.percentile(lat, 99)), 4),
        "latency_path": "host tokens in, host PCM out, synchronous dc_decode_chunk",
        "p50_chunk_ms_device_buffers": round(float(np.percentile(lat_dev, 50)), 4),
        "p99_chunk_ms_device_buffers": round(float(np.percentile(lat_dev, 99)), 4),
        "p50_replay_ms_hip_events": round(float(np.percentile(lat_ev, 50)), 4),
    }
    config = {"workload": name, "arch": "real" if arch["embed"] == 512 else "tiny",
              "batch": B, "chunk_tokens": n, "chunks_cycled": chunks,
              "audio_s_per_step": audio_s, "graph_replay": stats["replays"] > 0,
              "kernels_per_step": stats["kernels_per_step"], "flops_per_step": flops_step}
    if not headline:
        return {"value": round(value, 3), "unit": "audio-s/s" if arch["embed"] == 512 else "nominal audio-s/s",
                "steps": steps, "warmup": warmup, "ms_per_step": round(ms_per_step, 4), "dtype": dtype,
                "config": config, **lat_fields, "capture_ms": round(stats["capture_ms"], 3),
                "roofline": roof, "cpu_baseline": cpu, "parity": parity}
    return {
        "metric": METRIC, "value": round(value, 3), "unit": "audio-s/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic (seeded random-weight decoder and uniform token ids"
                + (", synthetic f0 contours)" if has_src else ")"),
        "config": config, **lat_fields, "capture_ms": round(stats["capture_ms"], 3),
        "roofline": roof, "cpu_baseline": cpu, "parity": parity,
    }


if __name__ == "__main__":
    main()
