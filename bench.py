"""Benchmark: spliced decode attention over a full synthetic sweep on one GPU.

A "step" is one decode step of the sweep: all N layers' calls of
splice_decode_attn (the whole hot path) for all C cells at decode position
s.  K timed steps take s evenly spaced over [0, S) -- the default K = S is
exactly one full sweep.  Each step's N calls are captured once in a HIP
graph (torch.cuda.CUDAGraph) and replayed; every layer has its own caches,
all resident in HBM before the timed region starts.

Reported (one JSON line):
  value       algorithmic bytes / wall time of the timed region (GB/s); the
              algorithmic bytes of a call count each shared prompt tile once
              (q, visible non-span prompt, clean span if a clean cell reads
              it, donor span if a spliced cell reads a donor buffer, every
              cell's visible generated rows, out and lse);
  cell_steps_per_s   C * K / wall time;
  per_step    time per launch and GB/s of one step's N launches at
              s = 0, S/4, S/2, S - 1 (measured after the timed region);
  per_step_cold  the same steps with the last-level cache flushed before
              each launch (a 512 MiB read outside the timed events; eager
              launches, so each includes its dispatch);
  roofline    bound "hbm": achieved = algorithmic bytes per call / average
              call duration (HIP events on the launch stream, over the timed
              region; a call is one kernel launch), peak 8000 GB/s,
              and the HBM traffic per call from the committed rocprofv3
              counter summary when it was taken on the current kernel source
              (else null);
  cpu_baseline  the fp64 oracle timed on this host's cores on a stratified
              sample of the same workload's calls;
  forked      the same sweep through splice_decode_forked (one clean run,
              each cell forked from it at its onset W; a never-spliced cell
              of the grid is the trunk): ms per step, cell-steps/s, GB/s of
              its algorithmic bytes, the fraction of cell-steps computed,
              and the speed-up over the lock-step region;
  e2e         the decode loop around the attention with a synthetic model
              (the workload's attention shape, its model's hidden sizes):
              ms per pass of all N layers plus the argmax, at the bucket
              steps, cell-steps/s, and the attention's share of a pass;
  read_ceiling  the rate of a plain stream read of a 4 GiB device buffer
              (libsplice_calib.so: contiguous parts per work group, 16-byte
              non-temporal loads; the best of three grid sizes, HIP events
              over ten launches each), measured in the same process before
              anything else is allocated (the buffer stays allocated for the
              run), and the sweep's GB/s as a share of it;
  decode_step  splice_decode_step passes (each cell at its own step, the
              current token's K/V appended, finished cells skipped) over two
              seeded step mixes -- 1/8 and 1/2 of the cells finished --
              measured after the timed region: time per launch, GB/s of
              the pass's algorithmic bytes, active cells, cell-steps/s.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config qwen3-8b] [--also llama3-8b]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2605_30574_amd", "csrc")
KERNEL_SOURCES = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                        if f.endswith((".hip", ".hpp")))


def log(msg: str) -> None:
    sys.stderr.write(f"[bench] {msg}\n")
    sys.stderr.flush()


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# ------------------------------------------------------------------ algorithmic bytes

def call_bytes(w, layer: int, step: int, spliced_flags) -> int:
    """Bytes a call must move at minimum: each prompt tile once per call."""
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e            # K + V row of every KV head
    Tp, (a, b) = w.prompt_len, w.span
    win = w.window(layer)
    p = Tp + step
    j0 = p - win + 1 if win > 0 else 0
    jp0 = min(max(j0, 0), Tp)
    i0 = max(0, j0 - Tp)
    n_gen = step + 1 - i0
    sa = min(max(a, jp0), Tp)
    sb = min(max(b, sa), Tp)
    n_sv = sb - sa
    n_ns = (Tp - jp0) - n_sv
    C = w.n_cells
    any_clean = any(not f for f in spliced_flags)
    any_spl = any(spliced_flags)
    buffer_donor = w.donor != "zero"
    total = C * w.n_q_heads * w.head_dim * e                     # q
    total += n_ns * row                                         # non-span prompt
    total += (n_sv * row) if any_clean else 0                   # clean span
    total += (n_sv * row) if (any_spl and buffer_donor) else 0  # donor span
    total += C * n_gen * row                                    # generated rows
    total += C * w.n_q_heads * (4 * w.head_dim + 4)             # out + lse
    return total


def step_bytes(w, layer: int, steps, cells) -> int:
    """Bytes a splice_decode_step call must move at minimum: the prompt slots
    some active cell sees (each once), each active cell's visible generated
    rows before its own step, its new K/V row read and written once, q, out
    and lse of the active cells.  Finished cells (step < 0) move nothing."""
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e
    Tp, (a, b) = w.prompt_len, w.span
    win = w.window(layer)
    act = [(s, L, W) for s, (L, W) in zip(steps, cells) if s >= 0]
    if not act:
        return 0
    total = 0
    vis = [0] * Tp                       # per prompt slot: 1 clean read, 2 donor read (bit mask)
    for s, L, W in act:
        p = Tp + s
        j0 = p - win + 1 if win > 0 else 0
        jp0 = min(max(j0, 0), Tp)
        i0 = max(0, j0 - Tp)
        total += (s - i0) * row + 2 * row                        # cached rows, new row in and out
        spl = layer >= L and s >= W
        donor_read = spl and w.donor != "zero"
        for j in range(jp0, Tp):
            in_span = a <= j < b
            if not in_span or not spl:
                vis[j] |= 1
            elif donor_read:
                vis[j] |= 2
    total += sum(bin(v).count("1") for v in vis) * row           # prompt slots, once per source
    n_act = len(act)
    total += n_act * w.n_q_heads * w.head_dim * e                  # q
    total += n_act * w.n_q_heads * (4 * w.head_dim + 4)            # out + lse
    return total


def forked_bytes(w, layer: int, step: int, cells, trunk: int) -> int:
    """Bytes a splice_decode_forked call must move at minimum: the prompt as
    in call_bytes for the diverged cells, the trunk's visible generated rows
    once (its own and, below their onsets, the forked cells'), each diverged
    cell's own rows from its onset on, q of the diverged cells, out and lse
    of every cell."""
    e = w.elem_bytes
    row = 2 * w.n_kv_heads * w.head_dim * e
    Tp, (a, b) = w.prompt_len, w.span
    win = w.window(layer)
    p = Tp + step
    j0 = p - win + 1 if win > 0 else 0
    jp0 = min(max(j0, 0), Tp)
    i0 = max(0, j0 - Tp)
    sa = min(max(a, jp0), Tp)
    sb = min(max(b, sa), Tp)
    n_sv, n_ns = sb - sa, (Tp - jp0) - (sb - sa)
    N = w.n_layers
    div = [c for c, (L, W) in enumerate(cells) if c == trunk or (L < N and step >= W)]
    spl = [layer >= cells[c][0] and step >= cells[c][1] for c in div]
    total = n_ns * row
    total += n_sv * row if not all(spl) else 0
    total += n_sv * row if any(spl) and w.donor != "zero" else 0
    total += (step + 1 - i0) * row                                       # the trunk's rows
    total += sum(max(0, step + 1 - max(i0, cells[c][1])) for c in div if c != trunk) * row
    total += len(div) * w.n_q_heads * w.head_dim * e
    total += len(cells) * w.n_q_heads * (4 * w.head_dim + 4)
    return total


def launch_kernels(w) -> str:
    """The kernel one splice_decode_attn call launches on this workload: bf16
    calls launch the one kernel of shared-prompt and generated-row items."""
    if w.dtype != "bf16":
        return "cellwise_kernel" if w.prompt_len <= 512 else "items_kernel"
    return "fused_kernel"


def spliced_flags(w, layer, step):
    return [layer >= L and step >= W for (L, W) in w.cells]


# ------------------------------------------------------------------ CPU baseline

def host_cpu():
    """(logical CPUs of this host, CPUs this process may run on, CPU model)."""
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return os.cpu_count() or 1, usable, model


def cpu_baseline(w, seconds_cap: float = 20.0):
    """Time the fp64 oracle (as it stands) on a stratified sample of calls of
    workload w: with every thread OpenMP gives it, then with one thread on a
    smaller sample; plus the full sweep of the tiny workload."""
    import numpy as np
    import oracle
    import workloads
    N, S = w.n_layers, w.n_steps
    layers = sorted({0, N // 2, N - 1})
    lw = workloads.cell_lw(w)
    osh = oracle.shape_of(w)
    lib = oracle.load()
    threads = oracle.max_threads()
    n_cpu, n_usable, model = host_cpu()

    def one_call(hb, layer, step, nt):
        q = workloads.to_numpy(workloads.make_q(w, layer, step, device="cpu"))
        t0 = time.perf_counter()
        oracle.attn(osh, layer, step, w.window(layer), w.scale, lw, q, hb["clean_k"], hb["clean_v"],
                    hb["donor_k"], hb["donor_v"], hb["gen_k"], hb["gen_v"], n_threads=nt, lib=lib)
        return time.perf_counter() - t0

    def sample(nt, cap):
        # pilot (untimed): one call at the middle step sizes the stratified
        # grid so that the sample takes about `cap` seconds; a call's cost is
        # affine in the step, so the middle step is the grid's average
        hb = {k: workloads.to_numpy(v) for k, v in workloads.make_layer(w, layers[0], device="cpu").items()}
        t_mid = max(one_call(hb, layers[0], S // 2, nt), 1e-4)
        n_s = int(max(2, min(S, cap / (len(layers) * t_mid))))
        steps = sorted({min(S - 1, int((i + 0.5) * S / n_s)) for i in range(n_s)})
        done_bytes, done_time, n_calls = 0, 0.0, 0
        t_start = time.time()
        for layer in layers:
            if layer != layers[0]:
                hb = {k: workloads.to_numpy(v) for k, v in workloads.make_layer(w, layer, device="cpu").items()}
            for step in steps:
                done_time += one_call(hb, layer, step, nt)
                done_bytes += call_bytes(w, layer, step, spliced_flags(w, layer, step))
                n_calls += 1
                if time.time() - t_start > 2 * cap:   # a bad pilot estimate: stop the sample
                    break
            del hb
            if time.time() - t_start > 2 * cap:
                break
        return done_bytes, done_time, n_calls, len(steps)

    b_all, t_all, n_all, k_all = sample(threads, seconds_cap)
    b_one, t_one, n_one, k_one = sample(1, seconds_cap / 2)
    # the tiny f32 workload: its whole sweep (every layer, step and cell), all threads
    tw = workloads.get(0)
    tlw, tosh = workloads.cell_lw(tw), oracle.shape_of(tw)
    t_tiny, tiny_calls = 0.0, 0
    for layer in range(tw.n_layers):
        hb = {k: workloads.to_numpy(v) for k, v in workloads.make_layer(tw, layer, device="cpu").items()}
        for step in range(tw.n_steps):
            q = workloads.to_numpy(workloads.make_q(tw, layer, step, device="cpu"))
            t0 = time.perf_counter()
            oracle.attn(tosh, layer, step, tw.window(layer), tw.scale, tlw, q, hb["clean_k"], hb["clean_v"],
                        hb["donor_k"], hb["donor_v"], hb["gen_k"], hb["gen_v"], n_threads=threads, lib=lib)
            t_tiny += time.perf_counter() - t0
            tiny_calls += 1
    return {"value": round(b_all / t_all / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_all} calls of {w.name}: layers {layers} x {k_all} steps evenly "
                      f"spaced over [0, {S}) (stratified), all {w.n_cells} cells x {w.n_q_heads} heads, "
                      f"fp64, {threads} OpenMP threads, {t_all:.1f} s",
            "calls": n_all, "seconds": round(t_all, 2),
            # a cell-step is one cell at one step over all N layers: the
            # stratified sample's calls per second times C / N
            "cell_steps_per_s": round(n_all / t_all * w.n_cells / N, 3),
            "host": {"nproc": n_cpu, "usable_cpus": n_usable, "cpu_model": model},
            "one_thread": {"value": round(b_one / t_one / 1e9, 4), "unit": "GB/s", "calls": n_one,
                           "seconds": round(t_one, 2),
                           "sample": f"layers {layers} x {k_one} steps, 1 thread"},
            "tiny_full_sweep": {"workload": tw.name, "calls": tiny_calls, "cell_steps": tw.n_cells * tw.n_steps,
                                "seconds": round(t_tiny, 4),
                                "cell_steps_per_s": round(tw.n_cells * tw.n_steps / t_tiny, 1)}}


# ------------------------------------------------------------------ traffic from profiles

def stored_traffic(w_name: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source and workload."""
    path = os.path.join(PROFILES, f"splice_decode_attn_{w_name}_traffic.txt")
    if not os.path.exists(path):
        return None, "no counter summary"
    fields = {}
    for ln in open(path):
        if ":" in ln and not ln.startswith("#"):
            k, v = ln.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256_16") != kernel_source_hash():
        return None, "kernel changed since the counters were taken"
    try:
        return float(fields["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)
    except (KeyError, ValueError):
        return None, "malformed counter summary"


class _Sweep:
    pass


def timed_sweep(w, K: int, warmup: int, eager: bool, dev, extra_steps=()):
    """Make workload w's inputs resident, capture one graph per decode step
    (N launches of splice_decode_attn), replay `warmup` steps, then time K
    steps evenly spaced over [0, S) between two HIP events on the launch
    stream.  Returns the buffers, the runner and the timings."""
    import torch

    import paper_2605_30574_amd as sp
    import workloads
    N, S, C = w.n_layers, w.n_steps, w.n_cells
    r = _Sweep()
    r.timed_steps = [min(S - 1, int((i + 0.5) * S / K)) for i in range(K)]
    r.warm_steps = [min(S - 1, int((i + 0.5) * S / max(1, warmup))) for i in range(warmup)]
    log(f"workload {w.name}: N={N} C={C} Hq={w.n_q_heads} Hkv={w.n_kv_heads} D={w.head_dim} "
        f"T_p={w.prompt_len} S={S}; timed steps K={K}")
    t0 = time.time()
    r.layers = [workloads.make_layer(w, l, device=dev) for l in range(N)]
    r.qs = [workloads.make_q(w, l, 0, device=dev) for l in range(N)]
    torch.cuda.synchronize()
    log(f"inputs resident in HBM ({time.time() - t0:.1f} s, "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB)")
    r.shape = sp.make_shape(C, N, w.n_q_heads, w.n_kv_heads, w.head_dim, w.prompt_len, w.span, S,
                            w.donor == "zero", w.dtype)
    r.lw = workloads.cell_lw(w)
    r.ws = sp.new_workspace(r.shape, device=dev)
    r.out = torch.empty((C, w.n_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    r.lse = torch.empty((C, w.n_q_heads), dtype=torch.float32, device=dev)

    def issue_step(s: int):
        for l in range(N):
            b = r.layers[l]
            sp.splice_decode_attn(r.shape, sp.make_call(l, s, w.window(l), w.scale), r.lw, r.qs[l],
                                  b["clean_k"], b["clean_v"], b["donor_k"], b["donor_v"],
                                  b["gen_k"], b["gen_v"], r.out, r.lse, r.ws)

    r.stream = torch.cuda.Stream(device=dev)
    r.stream.wait_stream(torch.cuda.current_stream(dev))
    graphs = {}
    if not eager:
        t0 = time.time()
        for s in sorted(set(r.timed_steps) | set(r.warm_steps) | set(extra_steps)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=r.stream):
                issue_step(s)
            graphs[s] = g
        torch.cuda.synchronize()
        log(f"captured {len(graphs)} step graphs of {N} launches ({time.time() - t0:.1f} s)")
    r.graphs = graphs

    def run(steps_list):
        with torch.cuda.stream(r.stream):
            for s in steps_list:
                if eager:
                    issue_step(s)
                else:
                    graphs[s].replay()
    r.run = run

    run(r.warm_steps)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(r.stream)
    run(r.timed_steps)
    ev1.record(r.stream)
    torch.cuda.synchronize()
    r.ms = ev0.elapsed_time(ev1)
    r.sec = r.ms / 1e3
    r.launches = K * N
    r.alg_bytes = sum(call_bytes(w, l, s, spliced_flags(w, l, s)) for s in r.timed_steps for l in range(N))
    r.gbs = r.alg_bytes / r.sec / 1e9
    r.handovers = sp.splice_workspace_handovers(r.ws, r.stream)
    log(f"timed {r.launches} launches in {r.ms:.2f} ms: {r.gbs:.1f} GB/s algorithmic, "
        f"{C * K / r.sec:.0f} cell-steps/s, {r.handovers} merges handed over")
    return r


def sweep_summary(w, r, K: int):
    """The sweep figures of a timed_sweep result, with its roofline."""
    traffic, traffic_src = stored_traffic(w.name)
    per_launch = r.alg_bytes / r.launches
    avg_s = r.sec / r.launches
    return {"GB/s": round(r.gbs, 2), "pct_of_hbm_peak": round(100 * r.gbs / HBM_PEAK_GBS, 2),
            "cell_steps_per_s": round(w.n_cells * K / r.sec, 1), "ms_per_step": round(r.ms / K, 4),
            "steps": K, "merges_handed_over": r.handovers,
            "roofline": {"bound": "hbm", "achieved": round(per_launch / avg_s / 1e9, 2), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(per_launch / avg_s / 1e9 / HBM_PEAK_GBS, 4),
                         "traffic": traffic, "kernel": launch_kernels(w), "bytes_per_launch": round(per_launch),
                         "avg_launch_us": round(avg_s * 1e6, 3), "traffic_source": traffic_src},
            "config": {"workload": w.name, "layers": w.n_layers, "cells": w.n_cells, "q_heads": w.n_q_heads,
                       "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "prompt_len": w.prompt_len,
                       "span": list(w.span), "decode_steps": w.n_steps, "donor": w.donor}}


# ------------------------------------------------------------ read ceiling

def read_ceiling(dev, gib: int = 4, reps: int = 10, keep: list = None) -> dict:
    """The rate of libsplice_calib.so's stream read over a `gib` GiB device
    buffer (16 times the last-level cache, so every launch reads from HBM):
    HIP events over `reps` launches after one untimed launch, for 1024, 2048
    and 4096 work groups; the best of the three.  Device memory handed out
    again after a large free reads ~5% slower than a fresh allocation, so
    the bench measures this first, on fresh memory, and keeps the buffer
    (appended to `keep`) so that its own caches do not reuse that range."""
    import torch

    from paper_2605_30574_amd import calib
    n = gib << 30
    buf = torch.empty(n, dtype=torch.uint8, device=dev)
    sink = torch.empty(calib.MAX_BLOCKS, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream(device=dev)
    stream.wait_stream(torch.cuda.current_stream(dev))
    rates = {}
    for blocks in (1024, 2048, 4096):
        calib.stream_read(buf, sink, blocks, stream)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            calib.stream_read(buf, sink, blocks, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        rates[blocks] = n * reps / (e0.elapsed_time(e1) / 1e3) / 1e9
    if keep is not None:
        keep.append(buf)
    del buf, sink
    torch.cuda.empty_cache()
    best = max(rates, key=rates.get)
    return {"GB/s": round(rates[best], 1), "blocks": best, "bytes": n, "launches": reps,
            "kernel": "stream_read_kernel", "per_blocks": {str(b): round(r, 1) for b, r in rates.items()}}


# ------------------------------------------------------------------ main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0, help="timed decode steps (default: S = one sweep)")
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", default="qwen3-8b")
    ap.add_argument("--also", default="llama3-8b",
                    help="comma-separated workloads whose sweep is timed after the main one ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--eager", action="store_true", help="launch without graphs")
    ap.add_argument("--no-forked", action="store_true", help="skip the forked-sweep measurement")
    ap.add_argument("--no-e2e", action="store_true", help="skip the decode-loop measurement")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--read-ceiling-only", action="store_true",
                    help="only measure the stream-read ceiling and print it")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the sweep shards cells across GPUs with no "
              "exchange, and multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2605_30574_amd as sp
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "launches": 5}))
        return

    if args.read_ceiling_only:
        print(json.dumps({"read_ceiling": read_ceiling(dev)}))
        return

    sp.load_library()
    held = []
    ceiling = read_ceiling(dev, keep=held)
    w = workloads.get(args.config)
    N, S, C = w.n_layers, w.n_steps, w.n_cells
    K = args.steps if args.steps > 0 else S
    bucket_steps = sorted({0, S // 4, S // 2, S - 1})
    sw = timed_sweep(w, K, args.warmup, args.eager, dev, extra_steps=bucket_steps)
    layers, qs, shape, lw, ws, out, lse = sw.layers, sw.qs, sw.shape, sw.lw, sw.ws, sw.out, sw.lse
    stream, run, timed_steps, warm_steps = sw.stream, sw.run, sw.timed_steps, sw.warm_steps
    ms, sec, launches, alg_bytes, gbs = sw.ms, sw.sec, sw.launches, sw.alg_bytes, sw.gbs

    # per-step buckets (outside the timed region): one step's N launches,
    # replayed a few times, at s = 0, S/4, S/2, S - 1
    per_step = {}
    for s in bucket_steps:
        reps = 5
        run([s])
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        run([s] * reps)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 1e3 / reps
        b = sum(call_bytes(w, l, s, spliced_flags(w, l, s)) for l in range(N))
        per_step[str(s)] = {"us_per_launch": round(t / N * 1e6, 2), "GB/s": round(b / t / 1e9, 1)}
    log("per-step buckets: " + ", ".join(f"s={k}: {v['us_per_launch']} us/launch, {v['GB/s']} GB/s"
                                          for k, v in per_step.items()))

    # the same buckets cold: before every timed launch a 512 MiB buffer is
    # read (outside the events), which leaves no tile of the call in the
    # 256 MiB last-level cache -- and no dirty lines either, as after the
    # weight reads of a model's other layers
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
    flush_sum = torch.empty((), dtype=torch.float32, device=dev)
    with torch.cuda.stream(stream):
        torch.sum(flush, 0, out=flush_sum)
    torch.cuda.synchronize()
    per_step_cold = {}
    for s in bucket_steps:
        tot, nb = 0.0, 0
        for l in range(N):
            b = layers[l]
            with torch.cuda.stream(stream):
                torch.sum(flush, 0, out=flush_sum)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                sp.splice_decode_attn(shape, sp.make_call(l, s, w.window(l), w.scale), lw, qs[l],
                                      b["clean_k"], b["clean_v"], b["donor_k"], b["donor_v"],
                                      b["gen_k"], b["gen_v"], out, lse, ws)
                e1.record(stream)
            torch.cuda.synchronize()
            tot += e0.elapsed_time(e1) / 1e3
            nb += call_bytes(w, l, s, spliced_flags(w, l, s))
        per_step_cold[str(s)] = {"us_per_launch": round(tot / N * 1e6, 2), "GB/s": round(nb / tot / 1e9, 1)}
    del flush, flush_sum
    log("per-step buckets, cold: " + ", ".join(f"s={k}: {v['us_per_launch']} us/launch, {v['GB/s']} GB/s"
                                                for k, v in per_step_cold.items()))

    # decode passes with cells at their own steps (splice_decode_step: KV
    # append + attention, finished cells skipped), outside the timed region:
    # one pass = the N layers' launches, graph-captured like the sweep steps
    decode_step = None
    if w.dtype == "bf16":
        mixes = {"ragged": workloads.cell_steps(w, seed=1, n_cells=C, finished=0.125),
                 "ragged-half-finished": workloads.cell_steps(w, seed=2, n_cells=C, finished=0.5)}
        news = [workloads.make_new_rows(w, l, 0, device=dev) for l in range(N)]
        call0 = [sp.make_call(l, 0, w.window(l), w.scale) for l in range(N)]
        decode_step = {}
        for name, st in mixes.items():
            def issue_pass(st=st):
                for l in range(N):
                    b = layers[l]
                    sp.splice_decode_step(shape, call0[l], lw, st, qs[l], news[l]["k_new"], news[l]["v_new"],
                                          b["clean_k"], b["clean_v"], b["donor_k"], b["donor_v"],
                                          b["gen_k"], b["gen_v"], out, lse, ws)
            g = None
            if not args.eager:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    issue_pass()
            reps = 10
            with torch.cuda.stream(stream):
                (g.replay() if g else issue_pass())
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            with torch.cuda.stream(stream):
                for _ in range(reps):
                    (g.replay() if g else issue_pass())
            e1.record(stream)
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) / 1e3 / reps
            bts = sum(step_bytes(w, l, st.tolist(), w.cells) for l in range(N))
            act = st[st >= 0]
            decode_step[name] = {"us_per_launch": round(t / N * 1e6, 2), "GB/s": round(bts / t / 1e9, 1),
                                 "active_cells": int(act.size), "mean_step": round(float(act.mean()), 1),
                                 "cell_steps_per_s": round(int(act.size) / t, 1)}
        log("decode passes: " + ", ".join(f"{k}: {v['us_per_launch']} us/launch, {v['GB/s']} GB/s, "
                                           f"{v['active_cells']} active" for k, v in decode_step.items()))

    # the same sweep decoded as one clean run that the cells fork from at
    # their onsets (splice_decode_forked), when the grid has a never-spliced
    # cell to be the trunk; timed after the main region, graph per step
    forked = None
    never = [c for c, (L, W) in enumerate(w.cells) if L >= N]
    if w.dtype == "bf16" and never and not args.no_forked:
        trunk = never[0]
        cells = list(w.cells)

        def issue_forked(s: int):
            for l in range(N):
                b = layers[l]
                sp.splice_decode_forked(shape, sp.make_call(l, s, w.window(l), w.scale), lw, trunk, qs[l],
                                        b["clean_k"], b["clean_v"], b["donor_k"], b["donor_v"],
                                        b["gen_k"], b["gen_v"], out, lse, ws)
        fgraphs = {}
        if not args.eager:
            for s in sorted(set(timed_steps) | set(warm_steps)):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    issue_forked(s)
                fgraphs[s] = g

        def run_forked(steps_list):
            with torch.cuda.stream(stream):
                for s in steps_list:
                    if args.eager:
                        issue_forked(s)
                    else:
                        fgraphs[s].replay()
        run_forked(warm_steps)
        torch.cuda.synchronize()
        f0 = torch.cuda.Event(enable_timing=True)
        f1 = torch.cuda.Event(enable_timing=True)
        f0.record(stream)
        run_forked(timed_steps)
        f1.record(stream)
        torch.cuda.synchronize()
        fsec = f0.elapsed_time(f1) / 1e3
        fbytes = sum(forked_bytes(w, l, s, cells, trunk) for s in timed_steps for l in range(N))
        n_div = [sum(1 for c, (L, W) in enumerate(cells) if c == trunk or (L < N and s >= W)) for s in timed_steps]
        forked = {"trunk_cell": list(cells[trunk]), "ms_per_step": round(fsec * 1e3 / K, 4),
                  "cell_steps_per_s": round(C * K / fsec, 1), "GB/s": round(fbytes / fsec / 1e9, 1),
                  "computed_cells_frac": round(sum(n_div) / (C * K), 4),
                  "speedup_vs_lockstep": round(sec / fsec, 3)}
        del fgraphs
        log(f"forked sweep: {forked['ms_per_step']} ms/step, {forked['cell_steps_per_s']} cell-steps/s, "
            f"{forked['computed_cells_frac']:.3f} of the cell-steps computed, x{forked['speedup_vs_lockstep']}")

    # the whole decode loop around the attention (Algorithm 1): a synthetic
    # model of the workload's attention shape and its model's hidden sizes,
    # one pass = all N layers' projections, norms and MLPs (library GEMMs)
    # plus this library's KV append + attention, then the argmax; each
    # pass captured once per starting step and replayed
    e2e = None
    from workloads.model import MODELS, make_weights
    if w.dtype == "bf16" and w.name in MODELS and not args.no_e2e:
        from paper_2605_30574_amd import decode
        m = MODELS[w.name]
        t0 = time.time()
        wt = make_weights(w, m, dtype=torch.bfloat16, device=dev, draw_on_device=True)
        torch.cuda.synchronize()
        n_params = sum(t.numel() for t in (wt["embed"], wt["lm_head"])) + \
            sum(t.numel() for L in wt["layers"] for t in L.values())
        log(f"synthetic model: {n_params / 1e9:.2f} B parameters drawn in {time.time() - t0:.1f} s")
        dec = decode.SweepDecoder(w, m, wt, layers, lw, device=dev)
        passes = {}
        for s0 in bucket_steps:
            steps = np.full(C, s0, dtype=np.int32)
            pos = dec.positions(steps)
            tok = torch.full((C,), 1, dtype=torch.long, device=dev)
            with torch.cuda.stream(stream):
                dec.step(tok, steps, pos)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                dec.step(tok, steps, pos)
            with torch.cuda.stream(stream):
                g.replay()
            reps = 10
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            with torch.cuda.stream(stream):
                for _ in range(reps):
                    g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            ms_pass = e0.elapsed_time(e1) / reps
            att_ms = per_step[str(s0)]["us_per_launch"] * N / 1e3
            passes[str(s0)] = {"ms_per_pass": round(ms_pass, 3), "cell_steps_per_s": round(C / ms_pass * 1e3, 1),
                               "attention_share": round(att_ms / ms_pass, 3)}
            del g
        e2e = {"model": {"layers": N, "d_model": m.d_model, "d_ff": m.d_ff, "vocab": m.vocab,
                         "params_B": round(n_params / 1e9, 2), "weights": "synthetic bf16"},
               "passes": passes}
        log("decode loop: " + ", ".join(f"s={k}: {v['ms_per_pass']} ms/pass, {v['cell_steps_per_s']} cell-steps/s, "
                                        f"attention {100 * v['attention_share']:.0f}%" for k, v in passes.items()))
        del dec, wt

    traffic, traffic_src = stored_traffic(w.name)
    per_launch_bytes = alg_bytes / launches
    avg_launch_s = sec / launches
    roofline = {"bound": "hbm", "achieved": round(per_launch_bytes / avg_launch_s / 1e9, 2),
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(per_launch_bytes / avg_launch_s / 1e9 / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": launch_kernels(w),
                "bytes_per_launch": round(per_launch_bytes),
                "avg_launch_us": round(avg_launch_s * 1e6, 3),
                "traffic_source": traffic_src, "kernel_source_sha256_16": kernel_source_hash()}

    handovers = sw.handovers
    # the other workloads' sweeps, timed the same way after this one's
    # buffers are freed
    del sw, layers, qs, ws, out, lse, run
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"stream-read ceiling (measured first, on fresh memory): {ceiling['GB/s']} GB/s "
        f"({ceiling['blocks']} work groups); the sweep reaches {100 * gbs / ceiling['GB/s']:.1f}% of it")
    also = {}
    for name in [n for n in args.also.split(",") if n and n != w.name]:
        w2 = workloads.get(name)
        K2 = args.steps if args.steps > 0 else w2.n_steps
        r2 = timed_sweep(w2, K2, args.warmup, args.eager, dev)
        also[name] = sweep_summary(w2, r2, K2)
        del r2
        torch.cuda.synchronize()
        torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on host cores (CPU baseline)")
        cpu = cpu_baseline(w, args.cpu_seconds)
        log(f"oracle: {cpu['value']} GB/s on {cpu['cores']} threads, {cpu['sample']}")

    res = {
        "metric": "spliced decode-attn HBM GB/s (% of peak) and sweep-cell decode steps/sec",
        "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms / K, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "cell_steps_per_s": round(C * K / sec, 1),
        "merges_handed_over": handovers,
        "read_ceiling": ceiling,
        "pct_of_read_ceiling": round(100 * gbs / ceiling["GB/s"], 2),
        "config": {"workload": w.name, "layers": N, "cells": C, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "prompt_len": w.prompt_len,
                   "span": list(w.span), "decode_steps": S, "donor": w.donor,
                   "launch": "eager" if args.eager else "hip-graph per decode step",
                   "timed_steps": "evenly spaced over the sweep" if K != S else "full sweep"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "also": also,
        "per_step": per_step,
        "per_step_cold": per_step_cold,
        "decode_step": decode_step,
        "forked": forked,
        "e2e": e2e,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
