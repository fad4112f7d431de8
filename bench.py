#!/usr/bin/env python3
"""Frame-step benchmark of windowed-KV frame attention on one MI355X.

Workload (default): Qwen3-Omni-30B-A3B-shaped attention -- 48 layers, 32 query
heads over 4 KV heads, head_dim 128, bf16 KV with fp32 accumulation, 128
sessions, each frame a 25-token chunk prefill then 16 decode steps, 4 pinned
sinks plus a 4096-token window in a paged pool of 16-token blocks.  Sessions
are first brought to steady state (window full and wrapping) by append-only
plans; every timed step is then one whole frame for all 128 sessions:
48 x (append + chunk prefill) followed by 16 x 48 x decode, each decode
launch appending its own token.

Inputs are synthetic N(0, 1) draws (torch's seeded device generator) in a
two-frame bank; they stand in for the paper's real-audio sessions.

Prints one JSON line: session-frames/s (whole job), decode-attention HBM
GB/s against the 8 TB/s peak (the dominant kernel, timed with HIP events
inside the library on the launch stream), and the float64 oracle timed on a
bounded sample on the host.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
COPY_PROBE_BYTES = 4 << 30
# sources of the decode kernel of the 128-session bf16 workload (the counters
# go stale when these change)
_CSRC = os.path.join(ROOT, "paper_2607_02640_amd", "csrc")
# the device sources each counted kernel is compiled from: a summary counts
# only while they are unchanged
KERNEL_SRC = {
    "decode": [os.path.join(_CSRC, f) for f in ("mtn_mfma.hip", "mtn_device.h", "mtn_kernels.h")],
    "prefill": [os.path.join(_CSRC, f) for f in ("mtn_kernels.hip", "mtn_device.h",
                                                  "mtn_kernels.h")],
}
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_traffic_qwen3omni_128s.json")
PREFILL_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "prefill_traffic_qwen3omni_128s.json")
READ_PROBE_BYTES = 8 << 30


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="qwen3-omni")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=48,
                    help="layers of one session-frame the oracle sample covers")
    ap.add_argument("--cpu-workers", type=int, default=0,
                    help="oracle baseline processes (0 = the host cores this process may "
                         "use, at most 16)")
    ap.add_argument("--cpu-frames", type=int, default=2,
                    help="consecutive session-frames each oracle process times")
    ap.add_argument("--n-split", type=int, default=0)
    ap.add_argument("--kv-dtype", choices=["bf16", "fp8"], default=None,
                    help="KV cache element type (default: the workload's); fp8 keeps E4M3 "
                         "codes with per-token power-of-two scales and bf16 io")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--call", action="store_true",
                    help="run a whole simulated call from empty sessions and report the "
                         "per-frame tick latency and pool occupancy series")
    ap.add_argument("--frames", type=int, default=0, help="--call: frames (0 = the workload's)")
    ap.add_argument("--kernel-times", action="store_true",
                    help="--call: HIP events around every launch, for the decode's achieved "
                         "GB/s over the call (the events add about 3 %% to each tick)")
    ap.add_argument("--pool-blocks", type=int, default=0,
                    help="--call: pool capacity in blocks (0 = exact windowed reservation)")
    ap.add_argument("--stagger", type=int, default=1,
                    help="--call: session start phases staggered over the frame period in "
                         "this many groups; each group's frames run in its own sub-tick")
    ap.add_argument("--admission", choices=["windowed", "unbounded"], default=None,
                    help="open-system admission ramp: sessions arrive at a fixed rate, an "
                         "AIMD controller on the measured tick latency admits or rejects "
                         "them, every tick runs one frame for all admitted sessions")
    ap.add_argument("--offered", type=int, default=512, help="--admission: sessions offered")
    ap.add_argument("--arrivals", type=int, default=12,
                    help="--admission: arrivals per tick (8/s at a 1.5 s frame)")
    ap.add_argument("--target-frac", type=float, default=0.3,
                    help="--admission: latency target as a fraction of the frame budget")
    ap.add_argument("--max-ticks", type=int, default=70, help="--admission: ticks to run")
    ap.add_argument("--recycle", action="store_true",
                    help="application-level recycling arm: an unbounded engine whose sessions "
                         "are dropped and re-prefilled with their sinks plus last W tokens "
                         "whenever the context would pass S + 2W")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this "
                         "bench into " + os.path.relpath(TRAFFIC_SUMMARY, ROOT) + " and exit")
    return ap.parse_args()


def _code_only(text: str) -> str:
    """C/C++ source with comments removed and whitespace runs collapsed: a
    counter summary stays valid across comment and layout edits."""
    import re
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == '"':  # string literal, copied as is
            j = i + 1
            while j < n and text[j] != '"':
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return re.sub(r"\s+", " ", "".join(out)).strip()


def kernel_src_hash(kernel: str = "decode") -> str:
    """Hash of the code (comments and layout aside) of the device sources the
    kernel compiles from, and of the options its source is compiled with."""
    import hashlib
    from paper_2607_02640_amd import build as pkg_build
    h = hashlib.sha256()
    for fn in KERNEL_SRC[kernel]:
        with open(fn, encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    main = os.path.basename(KERNEL_SRC[kernel][0])
    h.update(" ".join(pkg_build.compile_flags(main)).replace(ROOT, "").encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(w, kvd="bf16", fused_append=None):
    """Per-launch algorithmic bytes of the steady-state decode and chunk
    prefill of workload w (every query sees S + W keys).  Both launches may
    append their tokens (read k, v; write the pool copy): the decode always,
    the prefill when the chunk append is fused into it (by default for the
    fp8 pool, whose frame step fuses it at this shape)."""
    if fused_append is None:
        fused_append = kvd == "fp8"
    esz = 4 if kvd == "f32" else 2
    N, Hq, Hkv, D = w.n_sessions, w.n_q_heads, w.n_kv_heads, w.head_dim
    C = w.chunk[1]
    vis = w.n_sink + w.window
    beta = Hkv * (2 * D + 2) if kvd == "fp8" else 2 * Hkv * D * esz
    app = 2 * Hkv * D * esz + beta                       # one token's append
    dec = N * (vis * beta + Hq * D * 2 * esz + app)
    pre = N * ((vis + C - 1) * beta + C * Hq * D * 2 * esz + (C * app if fused_append else 0))
    return dec, pre


def traffic_summary(fetch_dir, write_dir):
    """Per-dispatch HBM bytes of the decode and of the chunk prefill from
    FETCH_SIZE / WRITE_SIZE (KiB per dispatch), each scaled by what the same
    counter reads for the bench's own copy kernel (COPY_PROBE_BYTES read and
    written per dispatch), against the kernels' algorithmic bytes."""
    import csv
    import glob
    import workload as W

    def avg(d, counter, needle):
        vals = []
        for fn in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(fn)):
                if r["Counter_Name"] == counter and needle in r["Kernel_Name"]:
                    vals.append(float(r["Counter_Value"]))
        if not vals:
            raise SystemExit(f"no {counter} samples for {needle} under {d}")
        return sum(vals) / len(vals), len(vals)

    kib = COPY_PROBE_BYTES / 1024
    f_copy, _ = avg(fetch_dir, "FETCH_SIZE", "k_copy")
    w_copy, _ = avg(write_dir, "WRITE_SIZE", "k_copy")
    fs, ws = kib / f_copy, kib / w_copy
    alg_dec, alg_pre = algorithmic_bytes(W.QWEN3_OMNI)
    commands = [
        "rocprofv3 --pmc FETCH_SIZE --output-format csv -d " + fetch_dir +
        " -o p -- python3 bench.py --steps 1 --warmup 0 --no-cpu-baseline",
        "rocprofv3 --pmc WRITE_SIZE --output-format csv -d " + write_dir +
        " -o p -- python3 bench.py --steps 1 --warmup 0 --no-cpu-baseline",
        "python3 bench.py --traffic-summary " + fetch_dir + " " + write_dir,
    ]
    for kernel, needle, label, alg, path in (
            ("decode", "k_attn_mfma", "k_attn_mfma<bf16> (decode attention)", alg_dec,
             TRAFFIC_SUMMARY),
            ("prefill", "k_prefill_mfma", "k_prefill_mfma<8, bf16> (chunk prefill)", alg_pre,
             PREFILL_TRAFFIC_SUMMARY)):
        f_k, nf = avg(fetch_dir, "FETCH_SIZE", needle)
        w_k, nw = avg(write_dir, "WRITE_SIZE", needle)
        rd, wr = f_k * fs * 1024, w_k * ws * 1024
        out = {
            "kernel": label + ", 128-session Qwen3-Omni-shaped workload",
            "kernel_src_sha256_16": kernel_src_hash(kernel),
            "commands": commands,
            "copy_kernel_KiB_per_dispatch": {"FETCH_SIZE": f_copy, "WRITE_SIZE": w_copy,
                                             "actual_read_KiB": kib, "actual_write_KiB": kib},
            "scale": {"fetch": fs, "write": ws},
            "KiB_per_dispatch_raw": {"FETCH_SIZE": f_k, "WRITE_SIZE": w_k, "dispatches": [nf, nw]},
            "bytes_per_launch": {"read": rd, "write": wr, "total": rd + wr},
            "algorithmic_bytes_per_launch": alg,
            "measured_over_algorithmic": (rd + wr) / alg,
        }
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
            f.write("\n")
        print(json.dumps(out, indent=1))


def measured_traffic(workload_name: str):
    """HBM bytes per decode launch from the committed counter summary, or None
    when the kernel source changed since the counters were taken or the
    counters cover another workload (they are taken on the 128-session
    Qwen3-Omni-shaped frame step)."""
    if workload_name != "qwen3-omni":
        return None
    try:
        with open(TRAFFIC_SUMMARY) as f:
            t = json.load(f)
    except OSError:
        return None
    if t.get("kernel_src_sha256_16") != kernel_src_hash("decode"):
        return None
    return t["bytes_per_launch"]["total"]


def measured_prefill_traffic(workload_name: str):
    """The same for the chunk prefill: (bytes per launch, measured /
    algorithmic), or None."""
    if workload_name != "qwen3-omni":
        return None
    try:
        with open(PREFILL_TRAFFIC_SUMMARY) as f:
            t = json.load(f)
    except OSError:
        return None
    if t.get("kernel_src_sha256_16") != kernel_src_hash("prefill"):
        return None
    return t["bytes_per_launch"]["total"], t["measured_over_algorithmic"]


def pick(name):
    import workload as W
    table = {"qwen3-omni": W.QWEN3_OMNI, "moshi": W.MOSHI, "minicpm-o": W.MINICPM_O,
             "tiny": W.TINY, "pool-stress-windowed": W.POOL_STRESS_WINDOWED,
             "pool-stress-unbounded": W.POOL_STRESS_UNBOUNDED}
    return table[name]


def steady_len(w):
    """Smallest length at which every query of a frame sees S + W keys."""
    return w.n_sink + w.window


def run_gpu(args, w):
    import torch
    import paper_2607_02640_amd as mtn
    from workload import device_bank

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    kvd = args.kv_dtype or w.dtype
    tdt = torch.float32 if kvd == "f32" else torch.bfloat16   # io element type
    esz = 4 if kvd == "f32" else 2
    N, Lyr, Hq, Hkv, D = w.n_sessions, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim
    C, tau = w.chunk[1], w.n_decode[1]
    if w.chunk[0] != w.chunk[1] or w.n_decode[0] != w.n_decode[1]:
        raise SystemExit("bench drives fixed chunk/decode counts; pick a fixed-shape workload")
    R = -(-(w.window + C - 1) // 16) * 16
    blocks_per = -(-w.n_sink // 16) + R // 16
    n_blocks = N * blocks_per
    kw = dict(n_layers=Lyr, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, n_sink=w.n_sink,
              window=w.window, max_chunk=C, max_sessions=N, n_blocks=n_blocks, dtype=kvd,
              rope_theta=w.rope_theta)
    nbytes = mtn.Pool.required(**kw)
    log(f"[bench] pool {nbytes / 1e9:.1f} GB ({n_blocks} blocks), workload {w.name}, kv {kvd}")
    kv = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    pool = mtn.Pool(**kw, kv=kv)
    sids = [pool.session_open() for _ in range(N)]

    # two-frame input bank
    Tc = N * C
    bank = []
    for b in range(2):
        s0 = 1000 * w.workload_id + 10 * b
        bank.append(dict(
            qc=device_bank((Lyr, Tc, Hq, D), tdt, dev, s0 + 1, w.act_scale),
            kc=device_bank((Lyr, Tc, Hkv, D), tdt, dev, s0 + 2, w.act_scale),
            vc=device_bank((Lyr, Tc, Hkv, D), tdt, dev, s0 + 3, w.act_scale),
            qd=device_bank((tau, Lyr, N, Hq, D), tdt, dev, s0 + 4, w.act_scale),
            kd=device_bank((tau, Lyr, N, Hkv, D), tdt, dev, s0 + 5, w.act_scale),
            vd=device_bank((tau, Lyr, N, Hkv, D), tdt, dev, s0 + 6, w.act_scale)))
    oc = torch.empty((Lyr, Tc, Hq, D), dtype=tdt, device=dev)
    od = torch.empty((tau, Lyr, N, Hq, D), dtype=tdt, device=dev)

    # fast-forward to steady state with append-only plans (bank 0 chunk rows)
    t0 = time.time()
    L0 = steady_len(w)
    n_ff = -(-L0 // C)
    for p in range(n_ff):
        pool.plan_begin(sids, [C] * N)
        for l in range(Lyr):
            pool.frame_append_kv(l, bank[0]["kc"][l], bank[0]["vc"][l])
        pool.plan_commit()
    torch.cuda.synchronize()
    log(f"[bench] fast-forward {n_ff * C} tokens/session in {time.time() - t0:.1f}s")

    def step(f):
        bk = bank[f % 2]
        pool.frame_step(sids, [C] * N, [tau] * N, bk["qc"], bk["kc"], bk["vc"], oc,
                        bk["qd"], bk["kd"], bk["vd"], od, n_split=args.n_split)

    # copy probe: achievable HBM bandwidth (read + write bytes / time); also
    # the calibration kernel of the profiler's byte counters
    probe_bytes = COPY_PROBE_BYTES
    src = torch.empty(probe_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    mtn.hbm_copy(src, dst, probe_bytes)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        mtn.hbm_copy(src, dst, probe_bytes)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 5 * 2 * probe_bytes / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    # read probe: achievable read bandwidth of the decode's copy mechanism
    # (non-temporal LDS DMA of 8 KiB chunks), the ceiling beside the nominal peak
    rsrc = torch.empty(READ_PROBE_BYTES, dtype=torch.uint8, device=dev)
    rsrc.fill_(7)
    mtn.hbm_read(rsrc, READ_PROBE_BYTES)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        mtn.hbm_read(rsrc, READ_PROBE_BYTES)
    e1.record()
    torch.cuda.synchronize()
    read_gbps = 5 * READ_PROBE_BYTES / (e0.elapsed_time(e1) * 1e-3) / 1e9
    # the same read at one decode launch's size (rounded down to 8 KiB), timed
    # per launch like the decode: a launch that only streamed its bytes, with
    # no fixed cost beyond one kernel's start and drain
    vis = w.n_sink + w.window
    beta = Hkv * (2 * D + 2) if kvd == "fp8" else 2 * Hkv * D * esz
    dec_bytes_est = N * (vis * beta + Hq * D * 2 * esz + 2 * Hkv * D * esz + beta)
    same_bytes = min(READ_PROBE_BYTES, dec_bytes_est // 8192 * 8192)
    mtn.hbm_read(rsrc, same_bytes)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(20)]
    for a, b in pairs:
        a.record()
        mtn.hbm_read(rsrc, same_bytes)
        b.record()
    torch.cuda.synchronize()
    read_same_ms = sum(a.elapsed_time(b) for a, b in pairs) / len(pairs)
    del rsrc
    torch.cuda.synchronize()

    # warm-up frames last, right before the timed frames (the probes above
    # stream 16 GB of other memory)
    for f in range(args.warmup):
        step(f)
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} frames done")

    # Timed region 1: K frames with only frame-boundary events -> value.
    # Timed region 2: the same K frames again (steady state, so the same
    # work) with HIP events around every launch on the launch stream -> the
    # per-kernel averages of the roofline.  Per-launch events cost the frame
    # step about 3 % (≈1700 event records per frame), so they stay out of the
    # throughput measurement.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_start = time.time()
    evs[0].record()
    for f in range(args.steps):
        step(args.warmup + f)
        evs[f + 1].record()
    torch.cuda.synchronize()
    wall = time.time() - t_start
    ticks = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    total_ms = evs[0].elapsed_time(evs[-1])
    log(f"[bench] {args.steps} frames in {total_ms:.1f} ms (wall {wall:.2f}s)")
    pool.set_timing(True)
    pool.kernel_times()  # reset
    ek0, ek1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ek0.record()
    for f in range(args.steps):
        step(args.warmup + args.steps + f)
    ek1.record()
    torch.cuda.synchronize()
    kt = pool.kernel_times()
    pool.set_timing(False)
    timed_ms = ek0.elapsed_time(ek1)
    log(f"[bench] {args.steps} frames with per-launch events in {timed_ms:.1f} ms; kernels {kt}")

    # algorithmic bytes (steady state: every query sees S + W keys).  A decode
    # launch also appends its token (read k, v; write the pool copy), and so
    # does a chunk prefill with the append fused in (no append launches in the
    # timed frames)
    # pool bytes of one token (all kv heads): K and V rows, plus the two scale
    # exponent bytes per head of the fp8 cache
    n_dec, ms_dec = kt["decode"]
    n_mrg, ms_mrg = kt["merge"]
    n_pre, ms_pre = kt["prefill"]
    n_app, ms_app = kt["append"]
    vis = w.n_sink + w.window
    beta = Hkv * (2 * D + 2) if kvd == "fp8" else 2 * Hkv * D * esz
    app_tok = 2 * Hkv * D * esz + beta
    # per decode launch: the visible keys, q in and out, the new token's k and v
    # in (io type) and its pool copy out
    dec_bytes = N * (vis * beta + Hq * D * 2 * esz + app_tok)
    dec_flops = N * 4 * Hq * D * vis
    chunk_union = vis + C - 1                                 # keys a chunk reads
    pre_fused = n_app == 0
    pre_bytes = N * (chunk_union * beta + C * Hq * D * 2 * esz + (C * app_tok if pre_fused else 0))
    pre_flops = N * 4 * Hq * D * vis * C
    avg_dec = ms_dec / max(n_dec, 1)
    dec_gbps = dec_bytes / (avg_dec * 1e-3) / 1e9
    dec_merge_gbps = dec_bytes * n_dec / ((ms_dec + ms_mrg) * 1e-3) / 1e9
    avg_pre = ms_pre / max(n_pre, 1)
    pre_gbps = pre_bytes / (avg_pre * 1e-3) / 1e9 if n_pre else None
    pre_tflops = pre_flops / (avg_pre * 1e-3) / 1e12 if n_pre else None
    ms_per_step = total_ms / args.steps
    sfps = N * args.steps / (total_ms * 1e-3)
    srt = sorted(ticks)
    res = dict(
        sfps=sfps, ms_per_step=ms_per_step, ticks=ticks, ms_per_step_ktiming=timed_ms / args.steps,
        tick_p50=srt[len(srt) // 2], tick_max=srt[-1],
        dec_gbps=dec_gbps, dec_merge_gbps=dec_merge_gbps, avg_dec_ms=avg_dec,
        dec_bytes=dec_bytes, dec_launches=n_dec, dec_flops=dec_flops,
        merge_ms_avg=ms_mrg / max(n_mrg, 1), append_ms_avg=ms_app / max(n_app, 1),
        pre_gbps=pre_gbps, pre_tflops=pre_tflops, avg_pre_ms=avg_pre, pre_bytes=pre_bytes,
        pre_fused=pre_fused,
        copy_gbps=copy_gbps, read_gbps=read_gbps, n_blocks=n_blocks, pool_gb=nbytes / 1e9,
        kv_dtype=kvd, read_same_ms=read_same_ms, read_same_bytes=same_bytes)
    pool.close()
    return res


def run_call(args, w):
    """A whole simulated call: sessions start empty and run `frames` frames
    back to back (each tick serves every session: chunk prefill, then ragged
    decode rounds).  Ragged workloads draw chunk / decode counts per
    session-frame, start from mixed lengths (fast-forwarded by append-only
    plans) and churn sessions.  Records the tick latency of every frame
    (HIP events on the launch stream), pool occupancy, and the first frame a
    plan fails (pool exhausted)."""
    import numpy as np
    import torch
    import paper_2607_02640_amd as mtn
    from workload import device_bank

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    N, Lyr, Hq, Hkv, D = w.n_sessions, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim
    Cmax, Tmax = w.chunk[1], w.n_decode[1]
    frames = args.frames or w.frames
    ragged = w.chunk[0] != w.chunk[1] or w.n_decode[0] != w.n_decode[1]
    if w.window is None:
        # unbounded arm: the pool gets a fixed ~150 GB of HBM
        max_len = frames * (Cmax + Tmax) + 64
        block_bytes = Lyr * Hkv * 2 * 16 * D * (2 if w.dtype == "bf16" else 4)
        n_blocks = args.pool_blocks or int(150e9 // block_bytes)
    else:
        max_len = 0
        R = -(-(w.window + Cmax - 1) // 16) * 16
        n_blocks = args.pool_blocks or N * (-(-w.n_sink // 16) + R // 16)
    kw = dict(n_layers=Lyr, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, n_sink=w.n_sink,
              window=w.window, max_chunk=Cmax, max_sessions=N, n_blocks=n_blocks, dtype=w.dtype,
              rope_theta=w.rope_theta, max_len=max_len)
    nbytes = mtn.Pool.required(**kw)
    log(f"[call] {w.name}: pool {nbytes / 1e9:.1f} GB ({n_blocks} blocks), {frames} frames")
    kv = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    pool = mtn.Pool(**kw, kv=kv)
    sids = [pool.session_open() for _ in range(N)]
    s0 = 1000 * w.workload_id + 500
    # chunk tensors are [layer][sum(chunk_len)][H][D] with the frame's own row
    # count, so each frame views a prefix of one flat bank
    rows = Lyr * N * Cmax
    qc_flat = device_bank((rows, Hq, D), tdt, dev, s0 + 1, w.act_scale)
    kc_flat = device_bank((rows, Hkv, D), tdt, dev, s0 + 2, w.act_scale)
    vc_flat = device_bank((rows, Hkv, D), tdt, dev, s0 + 3, w.act_scale)
    oc_flat = torch.empty_like(qc_flat)
    # staggered start phases: K groups of sessions, group k served in sub-tick
    # k of every frame period (its first frame starts k / K of a period late)
    K = max(1, args.stagger)
    if N % K:
        raise SystemExit(f"--stagger {K} must divide the session count {N}")
    ng = N // K
    groups = [list(range(k * ng, (k + 1) * ng)) for k in range(K)]
    qd = device_bank((Tmax, Lyr, ng, Hq, D), tdt, dev, s0 + 4, w.act_scale)
    kd = device_bank((Tmax, Lyr, ng, Hkv, D), tdt, dev, s0 + 5, w.act_scale)
    vd = device_bank((Tmax, Lyr, ng, Hkv, D), tdt, dev, s0 + 6, w.act_scale)
    od = torch.empty_like(qd)

    def chunk_view(t, tc):
        return t[:Lyr * tc].view(Lyr, tc, *t.shape[1:])
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.workload_id, 77])))
    churn = 0
    if ragged:
        # mixed lengths: 30 % still filling the window, 70 % wrapped
        S_W = w.n_sink + w.window
        target = np.where(rng.random(N) < 0.3, rng.integers(0, S_W, N),
                          rng.integers(S_W, 4 * S_W, N))
        have = np.zeros(N, dtype=np.int64)
        while True:
            idx = [i for i in range(N) if have[i] < target[i]]
            if not idx:
                break
            ntok = [int(min(Cmax, target[i] - have[i])) for i in idx]
            pool.plan_begin([sids[i] for i in idx], ntok)
            kf, vf = chunk_view(kc_flat, sum(ntok)), chunk_view(vc_flat, sum(ntok))
            for l in range(Lyr):
                pool.frame_append_kv(l, kf[l], vf[l])
            pool.plan_commit()
            for i, n in zip(idx, ntok):
                have[i] += n
        churn = max(1, round(0.02 * N))
        torch.cuda.synchronize()
        log(f"[call] fast-forwarded to mixed lengths (mean {have.mean():.0f} tokens)")
    else:
        have = np.zeros(N, dtype=np.int64)
    # algorithmic bytes of the decode and the chunk prefill launches, from the
    # sessions' lengths (a one-token chunk runs on the decode kernel)
    esz = 4 if w.dtype == "f32" else 2
    beta = 2 * Hkv * D * esz
    io_tok = Hq * D * 2 * esz + 2 * Hkv * D * esz
    SW = None if w.window is None else w.n_sink + w.window
    acct = dict(dec_bytes=0.0, pre_bytes=0.0, dec_ms=0.0, pre_ms=0.0, app_ms=0.0, mrg_ms=0.0,
                dec_n=0, pre_n=0, served=0)

    def vis(t):
        return t + 1 if SW is None else min(t + 1, SW)

    def account(grp, cl, nd, fused):
        """fused: the chunk prefill appended the chunk (no append launches)"""
        dec = pre = 0.0
        for i, c, d in zip(grp, cl, nd):
            L = int(have[i])
            if max(cl) == 1:
                dec += vis(L) * beta + io_tok + beta
            else:
                # keys the chunk's queries see: sinks, then the window run
                # [max(S, L - W + 1), L + c - 1]
                if SW is None:
                    union = L + c
                else:
                    union = min(w.n_sink, L + c) + max(0, L + c - max(w.n_sink, L - w.window + 1))
                pre += union * beta + c * Hq * D * 2 * esz + (c * (io_tok - Hq * D * 2 * esz + beta)
                                                              if fused else 0)
            for j in range(d):
                dec += vis(L + c + j) * beta + io_tok + beta
            have[i] = L + c + d
        acct["dec_bytes"] += dec * Lyr
        acct["pre_bytes"] += pre * Lyr
        acct["served"] += len(grp)

    def collect():
        """Kernel times since the last call; whether a chunk append ran as its
        own launch (else the chunk prefill took it)."""
        if not args.kernel_times:
            return False
        kt = pool.kernel_times()
        acct["dec_n"] += kt["decode"][0]
        acct["dec_ms"] += kt["decode"][1]
        acct["pre_n"] += kt["prefill"][0]
        acct["pre_ms"] += kt["prefill"][1]
        acct["app_ms"] += kt["append"][1]
        acct["mrg_ms"] += kt["merge"][1]
        return kt["append"][0] > 0
    if args.kernel_times:
        pool.set_timing(True)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * frames * K)]
    occ, fail_frame, fail_code = [], None, None
    n_sub = 0
    stats0 = pool.stats()
    for f in range(frames):
        for k, grp in enumerate(groups):
            if ragged:
                cl = rng.integers(w.chunk[0], w.chunk[1] + 1, ng).tolist()
                nd = rng.integers(w.n_decode[0], w.n_decode[1] + 1, ng).tolist()
            else:
                cl, nd = [Cmax] * ng, [Tmax] * ng
            tc = sum(cl)
            evs[2 * n_sub].record()
            try:
                pool.frame_step([sids[i] for i in grp], cl, nd, chunk_view(qc_flat, tc),
                                chunk_view(kc_flat, tc), chunk_view(vc_flat, tc),
                                chunk_view(oc_flat, tc), qd, kd, vd, od)
            except mtn.MtnError as e:
                fail_frame, fail_code = f + 1, e.code
                log(f"[call] frame {f + 1}: {e}")
                evs[2 * n_sub + 1].record()
                break
            evs[2 * n_sub + 1].record()
            n_sub += 1
            # with --kernel-times, every sub-tick's launches are read back at
            # once (a host wait per sub-tick), so the bytes follow the path
            # each chunk plan took
            separate = collect()
            account(grp, cl, nd, args.kernel_times and not separate)
        if fail_frame is not None:
            break
        st = pool.stats()
        occ.append(st["assigned"] / st["capacity"])
        if churn:
            for i in rng.choice(N, churn, replace=False):
                pool.session_close(sids[i])
                sids[i] = pool.session_open()
                have[i] = 0
        if (f + 1) % 50 == 0:
            torch.cuda.synchronize()
            log(f"[call] frame {f + 1}/{frames}")
    torch.cuda.synchronize()
    collect()
    done = len(occ)
    ticks = [evs[2 * j].elapsed_time(evs[2 * j + 1]) for j in range(done * K)]
    pool.close()
    return dict(ticks=ticks, occupancy=occ, fail_frame=fail_frame, fail_code=fail_code,
                n_blocks=n_blocks, frames=frames, reserved0=stats0["reserved"], stagger=K,
                acct=acct if args.kernel_times else None, served=acct["served"])


def call_report(args, w, r):
    """Tick statistics of a simulated call.  With K staggered groups a tick is
    one group's sub-tick and its deadline is its slot, B / K."""
    import numpy as np
    K = r.get("stagger", 1)
    t = np.array(r["ticks"])
    per10 = 10 * K                                   # ticks in 10 frame periods
    buckets = [round(float(np.median(t[i:i + per10])), 3) for i in range(0, len(t), per10)]
    fill = None
    if w.window is not None and w.chunk[0] == w.chunk[1]:
        per = w.chunk[1] + w.n_decode[1]
        fill = -(-(w.n_sink + w.window) // per)     # frames until every query sees S + W keys
    slot_ms = w.frame_period_s * 1e3 / K
    out = {
        "metric": "per-frame tick latency over a simulated call",
        "workload": w.name, "sessions": w.n_sessions, "frames_run": len(t) // K,
        "frames_planned": r["frames"], "frame_budget_ms": w.frame_period_s * 1e3,
        "stagger_groups": K, "sessions_per_tick": w.n_sessions // K, "tick_budget_ms": slot_ms,
        "tick_ms_p50_per_10_frames": buckets,
        "tick_ms_p50": round(float(np.median(t)), 3) if len(t) else None,
        "tick_ms_p99": round(float(np.percentile(t, 99)), 3) if len(t) else None,
        "tick_ms_max": round(float(t.max()), 3) if len(t) else None,
        "deadline_misses": int((t > slot_ms).sum()),
        "pool_blocks": r["n_blocks"],
        "occupancy_first_last": [round(r["occupancy"][0], 4), round(r["occupancy"][-1], 4)]
        if r["occupancy"] else None,
        "occupancy_per_10_frames": [round(float(x), 4) for x in r["occupancy"][9::10]],
        "pool_exhausted_in_frame": r["fail_frame"],
        "session_frames_per_s": round(r["served"] / (float(t.sum()) * 1e-3), 2) if len(t) else None,
    }
    a = r.get("acct")
    if a:
        out["kernel_times"] = {
            "note": "HIP events around every launch (ticks above include their cost)",
            "decode_launches": a["dec_n"], "decode_ms_total": round(a["dec_ms"], 2),
            "decode_algorithmic_GB": round(a["dec_bytes"] / 1e9, 3),
            "decode_GBps": round(a["dec_bytes"] / (a["dec_ms"] * 1e-3) / 1e9, 1)
            if a["dec_ms"] else None,
            "decode_frac_of_8TBps": round(a["dec_bytes"] / (a["dec_ms"] * 1e-3) / 8e12, 4)
            if a["dec_ms"] else None,
            "prefill_launches": a["pre_n"], "prefill_ms_total": round(a["pre_ms"], 2),
            "prefill_GBps": round(a["pre_bytes"] / (a["pre_ms"] * 1e-3) / 1e9, 1)
            if a["pre_ms"] else None,
            "append_ms_total": round(a["app_ms"], 2), "merge_ms_total": round(a["mrg_ms"], 2),
        }
    if fill is not None and len(t) > (fill + 10) * K:
        steady = t[fill * K:]
        mean = float(steady.mean())
        post = [float(np.median(steady[i:i + per10]))
                for i in range(0, len(steady) - per10 + 1, per10)]
        out["window_full_from_frame"] = fill + 1
        out["steady_mean_ms"] = round(mean, 3)
        out["steady_bucket_p50_max_dev_frac"] = round(max(abs(p / mean - 1) for p in post), 4)
    print(json.dumps(out), flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(json.dumps(out) + "\n")


def run_admission(args):
    """Open-system admission ramp on the Qwen3-Omni shapes (the paper's run
    offers 512 sessions at 8/s with a latency target of 0.3 of the budget).
    Every tick: offer the tick's arrivals to the AIMD controller, open the
    admitted ones (each arrives with S + W tokens of history, appended
    untimed, so a windowed session costs its steady-state work from its
    first tick), run one frame for every admitted session, and feed the
    tick's latency (HIP events) back to the controller.  The windowed arm
    sizes its pool to the controller's max cap; the unbounded arm gets the
    pool-stress capacity (150 GB) and keeps growing every session."""
    import numpy as np
    import torch
    import paper_2607_02640_amd as mtn
    from workload import device_bank, QWEN3_OMNI as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bf = torch.bfloat16
    Lyr, Hq, Hkv, D = W.n_layers, W.n_q_heads, W.n_kv_heads, W.head_dim
    C, tau = W.chunk[1], W.n_decode[1]
    max_cap = 448
    windowed = args.admission == "windowed"
    hist = W.n_sink + W.window                       # history each arrival brings
    if windowed:
        R = -(-(W.window + C - 1) // 16) * 16
        n_blocks = max_cap * (-(-W.n_sink // 16) + R // 16)
        window, max_len = W.window, 0
    else:
        block_bytes = Lyr * Hkv * 2 * 16 * D * 2
        n_blocks = int(150e9 // block_bytes)
        window, max_len = None, hist + args.max_ticks * (C + tau) + 64
    kw = dict(n_layers=Lyr, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, n_sink=W.n_sink,
              window=window, max_chunk=C, max_sessions=max_cap, n_blocks=n_blocks, dtype="bf16",
              rope_theta=W.rope_theta, max_len=max_len)
    nbytes = mtn.Pool.required(**kw)
    log(f"[admission] {args.admission}: pool {nbytes / 1e9:.1f} GB ({n_blocks} blocks)")
    kv = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    pool = mtn.Pool(**kw, kv=kv)
    budget_ms = W.frame_period_s * 1e3
    ctrl = mtn.Admission(target_ms=args.target_frac * budget_ms, backoff=0.8, increase=16,
                         initial_cap=16, min_cap=1, max_cap=max_cap, hold_ticks=2)
    s0 = 1000 * W.workload_id + 900
    # flat banks sized for max_cap sessions; each tick views a prefix
    qc = device_bank((Lyr * max_cap * C, Hq, D), bf, dev, s0 + 1)
    kc = device_bank((Lyr * max_cap * C, Hkv, D), bf, dev, s0 + 2)
    vc = device_bank((Lyr * max_cap * C, Hkv, D), bf, dev, s0 + 3)
    oc = torch.empty_like(qc)
    qd = device_bank((tau * Lyr * max_cap, Hq, D), bf, dev, s0 + 4)
    kd = device_bank((tau * Lyr * max_cap, Hkv, D), bf, dev, s0 + 5)
    vd = device_bank((tau * Lyr * max_cap, Hkv, D), bf, dev, s0 + 6)
    od = torch.empty_like(qd)

    def cview(t, n):
        return t[:Lyr * n * C].view(Lyr, n * C, *t.shape[1:])

    def dview(t, n):
        return t[:tau * Lyr * n].view(tau, Lyr, n, *t.shape[1:])

    sids, offered, rows = [], 0, []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall_tick = None
    for tick in range(1, args.max_ticks + 1):
        new = []
        for _ in range(args.arrivals):
            if offered >= args.offered:
                break
            offered += 1
            if ctrl.offer():
                new.append(pool.session_open())
        # arrivals bring their history (untimed); an unbounded pool can run
        # out here too, which is the same wall
        try:
            for p in range(-(-hist // C)) if new else []:
                pool.plan_begin(new, [C] * len(new))
                for l in range(Lyr):
                    pool.frame_append_kv(l, cview(kc, len(new))[l], cview(vc, len(new))[l])
                pool.plan_commit()
        except mtn.MtnError as e:
            wall_tick = tick
            log(f"[admission] tick {tick} (arrivals' history): {e}")
            break
        sids += new
        n = len(sids)
        torch.cuda.synchronize()
        e0.record()
        try:
            pool.frame_step(sids, [C] * n, [tau] * n, cview(qc, n), cview(kc, n), cview(vc, n),
                            cview(oc, n), dview(qd, n), dview(kd, n), dview(vd, n), dview(od, n))
        except mtn.MtnError as e:
            wall_tick = tick
            log(f"[admission] tick {tick}: {e}")
            break
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        ctrl.observe(ms)
        st, ps = ctrl.state(), pool.stats()
        rows.append(dict(tick=tick, offered=offered, admitted=st["admitted"], cap=st["cap"],
                         rejected=st["rejected"], tick_ms=round(ms, 3),
                         occupancy=round(ps["assigned"] / ps["capacity"], 4)))
        if tick % 10 == 0:
            log(f"[admission] tick {tick}: {rows[-1]}")
    pool.close()
    last = rows[-20:]
    ticks = np.array([r["tick_ms"] for r in last]) if last else np.array([0.0])
    out = {
        "metric": "open-system admission ramp under AIMD on the per-frame latency",
        "arm": args.admission, "workload": W.name, "offered": args.offered,
        "arrivals_per_tick": args.arrivals, "frame_budget_ms": budget_ms,
        "target_ms": args.target_frac * budget_ms,
        "controller": dict(backoff=0.8, increase=16, initial_cap=16, max_cap=max_cap, hold_ticks=2),
        "ticks_run": len(rows), "pool_exhausted_at_tick": wall_tick,
        "final": rows[-1] if rows else None,
        "last20_admitted_mean": float(np.mean([r["admitted"] for r in last])) if last else None,
        "last20_tick_ms_p50": float(np.median(ticks)), "last20_tick_ms_p99": float(np.percentile(ticks, 99)),
        "max_tick_ms": max(r["tick_ms"] for r in rows) if rows else None,
        "series": rows,
    }
    print(json.dumps(out), flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(json.dumps(out) + "\n")


def run_recycle(args):
    """Application-level recycling (the paper's alternative to the in-engine
    window, at the Qwen3-Omni shapes): the engine keeps every token (no
    window), and the application bounds the context itself -- when a
    session's context would pass S + 2W it closes the session, opens a fresh
    one and re-prefills the sinks plus the last W tokens as one S + W chunk
    (positions start again at 0), in that frame's batch.  Initial lengths are
    staggered over [S + W, S + 2W) so the re-encodes spread over frames.
    Inputs are synthetic draws like the other runs; the re-prefill costs
    what re-encoding the retained context costs this attention path."""
    import numpy as np
    import torch
    import paper_2607_02640_amd as mtn
    from workload import device_bank, QWEN3_OMNI as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bf = torch.bfloat16
    N, Lyr, Hq, Hkv, D = W.n_sessions, W.n_layers, W.n_q_heads, W.n_kv_heads, W.head_dim
    C, tau, S, Wn = W.chunk[1], W.n_decode[1], W.n_sink, W.window
    keep, limit = S + Wn, S + 2 * Wn
    frames = args.frames or W.frames
    max_len = limit + C + tau + 64
    n_blocks = N * -(-max_len // 16)
    kw = dict(n_layers=Lyr, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, n_sink=S, window=None,
              max_chunk=keep, max_sessions=N, n_blocks=n_blocks, dtype="bf16",
              rope_theta=W.rope_theta, max_len=max_len)
    nbytes = mtn.Pool.required(**kw)
    log(f"[recycle] pool {nbytes / 1e9:.1f} GB ({n_blocks} blocks), {frames} frames")
    kv = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    pool = mtn.Pool(**kw, kv=kv)
    sids = [pool.session_open() for _ in range(N)]
    r_max = 4                                   # re-encodes per frame; later ones wait a frame
    rows = Lyr * ((N - r_max) * C + r_max * keep)
    s0 = 1000 * W.workload_id + 700
    qc = device_bank((rows, Hq, D), bf, dev, s0 + 1)
    kc = device_bank((rows, Hkv, D), bf, dev, s0 + 2)
    vc = device_bank((rows, Hkv, D), bf, dev, s0 + 3)
    oc = torch.empty_like(qc)
    qd = device_bank((tau, Lyr, N, Hq, D), bf, dev, s0 + 4)
    kd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, s0 + 5)
    vd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, s0 + 6)
    od = torch.empty_like(qd)

    def cview(t, tc):
        return t[:Lyr * tc].view(Lyr, tc, *t.shape[1:])

    # staggered start: session i at keep + i * W / N tokens (append-only plans)
    target = [keep + (i * Wn) // N for i in range(N)]
    have = [0] * N
    while True:
        idx = [i for i in range(N) if have[i] < target[i]]
        if not idx:
            break
        ntok = [min(C, target[i] - have[i]) for i in idx]
        pool.plan_begin([sids[i] for i in idx], ntok)
        for l in range(Lyr):
            pool.frame_append_kv(l, cview(kc, sum(ntok))[l], cview(vc, sum(ntok))[l])
        pool.plan_commit()
        for i, n in zip(idx, ntok):
            have[i] += n
    length = list(have)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ticks, recycled = [], []
    for f in range(frames):
        due = [i for i in range(N) if length[i] + C + tau > limit][:r_max]
        for i in due:                           # drop the cache; the chunk re-encodes
            pool.session_close(sids[i])
            sids[i] = pool.session_open()
        cl = [keep if i in due else C for i in range(N)]
        tc = sum(cl)
        e0.record()
        pool.frame_step(sids, cl, [tau] * N, cview(qc, tc), cview(kc, tc), cview(vc, tc),
                        cview(oc, tc), qd, kd, vd, od)
        e1.record()
        torch.cuda.synchronize()
        ticks.append(e0.elapsed_time(e1))
        recycled.append(len(due))
        for i in range(N):
            length[i] = (keep if i in due else length[i] + C) + tau
        if (f + 1) % 50 == 0:
            log(f"[recycle] frame {f + 1}/{frames}")
    pool.close()
    t = np.array(ticks)
    rec = np.array(recycled)
    out = {
        "metric": "per-frame tick latency, application-level recycling arm",
        "workload": W.name + "-app-recycle", "sessions": N, "frames_run": len(t),
        "frame_budget_ms": W.frame_period_s * 1e3, "keep_tokens": keep, "recycle_at": limit,
        "tick_ms_p50": round(float(np.median(t)), 3),
        "tick_ms_p90": round(float(np.percentile(t, 90)), 3),
        "tick_ms_p99": round(float(np.percentile(t, 99)), 3),
        "tick_ms_max": round(float(t.max()), 3),
        "tick_ms_mean": round(float(t.mean()), 3),
        "tick_ms_mean_with_reencode": round(float(t[rec > 0].mean()), 3) if (rec > 0).any() else None,
        "tick_ms_mean_without": round(float(t[rec == 0].mean()), 3) if (rec == 0).any() else None,
        "reencodes": int(rec.sum()),
        "tick_ms_p50_per_10_frames": [round(float(np.median(t[i:i + 10])), 3)
                                      for i in range(0, len(t), 10)],
        "tick_ms": [round(float(x), 3) for x in t],
        "reencodes_per_frame": [int(x) for x in rec],
    }
    print(json.dumps(out), flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(json.dumps(out) + "\n")


def _oracle_frames(job):
    """One host worker: the float64 oracle (as it stands) fast-forwards one
    session to steady state (append + prune, no attention), then times
    ``frames`` consecutive session-frames over ``n_layers_sample`` layers."""
    wname, n_layers_sample, frames, uid = job
    from threadpoolctl import threadpool_limits
    from oracle import windowed_attention as wa
    from workload import session_rng, draw_qkv

    w = pick(wname)
    C, tau = w.chunk[1], w.n_decode[1]
    Hq, Hkv, D = w.n_q_heads, w.n_kv_heads, w.head_dim
    with threadpool_limits(limits=1):
        o = wa.OracleSession(Hq, Hkv, D, w.n_sink, w.window, theta=w.rope_theta,
                             n_layers=n_layers_sample)
        rng = session_rng(w.workload_id, uid)
        q, k, v = draw_qkv(rng, n_layers_sample, C, Hq, Hkv, D, w.act_scale)
        for p in range(-(-steady_len(w) // C)):
            o.begin(C)
            for l in range(n_layers_sample):
                o.layer_step(l, q[l], k[l], v[l], attend=False)
            o.commit()
        t0 = time.perf_counter()
        for f in range(frames):
            o.begin(C)
            for l in range(n_layers_sample):
                o.layer_step(l, q[l], k[l], v[l])
            o.commit()
            for j in range(tau):
                o.begin(1)
                for l in range(n_layers_sample):
                    o.layer_step(l, q[l, :1], k[l, :1], v[l, :1])
                o.commit()
        dt = time.perf_counter() - t0
    return frames, dt


def host_cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_workers_default():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def start_cpu_pool(n_workers):
    """Worker processes for the oracle baseline, started from a fork server
    before this process touches the GPU (the workers never use it)."""
    import multiprocessing as mp
    ctx = mp.get_context("forkserver")
    return ctx.Pool(n_workers)


def cpu_baseline(wkey, w, n_layers_sample, pool, n_workers, frames):
    """The float64 oracle timed on the host cores: ``n_workers`` processes of
    one thread each, each timing ``frames`` consecutive steady-state
    session-frames of its own session, restricted to ``n_layers_sample`` layers
    and scaled to the full depth."""
    jobs = [(wkey, n_layers_sample, frames, 1 + i) for i in range(n_workers)]
    t0 = time.perf_counter()
    res = pool.map(_oracle_frames, jobs) if pool is not None else [_oracle_frames(jobs[0])]
    wall = time.perf_counter() - t0
    scale = n_layers_sample / w.n_layers
    rates = [f * scale / dt for f, dt in res]        # session-frames/s per worker
    total = sum(rates)
    dts = [dt for _, dt in res]
    C, tau = w.chunk[1], w.n_decode[1]
    return dict(value=total, unit="session-frames/s", cores=len(res), kind="oracle",
                per_core=total / len(res),
                sample=(f"{len(res)} processes x 1 thread, each {frames} consecutive "
                        f"session-frames ({C}-token chunk + {tau} decodes) x {n_layers_sample} "
                        f"of {w.n_layers} layers of its own session at steady state "
                        f"(S + W = {w.n_sink + w.window} visible keys), float64 numpy on "
                        f"{host_cpu_model()}; timed regions {min(dts):.1f}-{max(dts):.1f}s, "
                        f"scaled by {w.n_layers}/{n_layers_sample}"),
                seconds=max(dts), wall_seconds=wall)


def main():
    args = parse()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the windowed-KV path "
              "shards by session with no exchange, so N GPUs run N independent copies",
              file=sys.stderr)
        sys.exit(2)
    if args.admission:
        run_admission(args)
        return
    if args.recycle:
        run_recycle(args)
        return
    w = pick(args.workload)
    if args.call:
        call_report(args, w, run_call(args, w))
        return
    pool = None
    if not args.no_cpu_baseline:
        n_workers = args.cpu_workers or cpu_workers_default()
        pool = start_cpu_pool(n_workers) if n_workers > 1 else None
    res = run_gpu(args, w)
    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the float64 oracle on the host ({n_workers} processes)")
        cpu = cpu_baseline(args.workload, w, args.cpu_layers, pool, n_workers, args.cpu_frames)
        if pool is not None:
            pool.close()
            pool.join()
        log(f"[bench] oracle {cpu['value']:.4f} session-frames/s "
            f"({cpu['seconds']:.1f}s per worker, {cpu['cores']} workers)")
    out = {
        "metric": "session-frames/sec and decode-attention HBM GB/s (% of peak) at 128 sessions",
        "value": round(res["sfps"], 2),
        "unit": "session-frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name, "sessions": w.n_sessions, "layers": w.n_layers,
            "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
            "sinks": w.n_sink, "window": w.window, "block": 16, "chunk": w.chunk[1],
            "decode_steps": w.n_decode[1], "frame_budget_s": w.frame_period_s,
            "steady_state": "every query sees S + W keys", "parallelism": "single GPU",
            "kv_cache": {"bf16": "bf16", "f32": "fp32",
                         "fp8": "fp8-e4m3, per-token power-of-two scales"}[res["kv_dtype"]],
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("decode attention (k_attn_mfma, fp8 blocks)" if res["kv_dtype"] == "fp8"
                       else "decode attention (k_attn_mfma, bf16 blocks)"
                       if w.n_q_heads == 8 * w.n_kv_heads and w.head_dim == 128
                       else "decode attention (k_attn_valu)"),
            "achieved": round(res["dec_gbps"], 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(res["dec_gbps"] / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(args.workload) if res["kv_dtype"] == w.dtype else None,
            "bytes_per_launch": res["dec_bytes"],
            "avg_launch_ms": round(res["avg_dec_ms"], 4),
            "launches": res["dec_launches"],
        },
        "cpu_baseline": None if cpu is None else {k: cpu[k] for k in
                                                  ("value", "unit", "cores", "kind", "sample")},
        "extra": {
            "cpu_baseline_per_core": None if cpu is None else cpu["per_core"],
            "ms_per_step_with_launch_events": round(res["ms_per_step_ktiming"], 3),
            "decode_plus_merge_GBps": round(res["dec_merge_gbps"], 1),
            "merge_ms_avg": round(res["merge_ms_avg"], 4),
            "append_ms_avg": round(res["append_ms_avg"], 4),
            "prefill_appends_chunk": res["pre_fused"],
            "prefill_GBps": None if res["pre_gbps"] is None else round(res["pre_gbps"], 1),
            "prefill_TFLOPs": None if res["pre_tflops"] is None else round(res["pre_tflops"], 2),
            "prefill_mfma_frac_of_bf16_peak": None if res["pre_tflops"] is None
            else round(res["pre_tflops"] / BF16_MFMA_PEAK_TFLOPS, 4),
            "prefill_ms_avg": round(res["avg_pre_ms"], 4),
            "tick_ms_p50": round(res["tick_p50"], 3),
            "tick_ms_max": round(res["tick_max"], 3),
            "tick_ms": [round(t, 3) for t in res["ticks"]],
            "frame_budget_ms": w.frame_period_s * 1e3,
            "copy_probe_GBps": round(res["copy_gbps"], 1),
            "read_probe_GBps": round(res["read_gbps"], 1),
            "decode_frac_of_read_probe": round(res["dec_gbps"] / res["read_gbps"], 4),
            "read_probe_one_launch": {"bytes": res["read_same_bytes"],
                                      "ms": round(res["read_same_ms"], 4),
                                      "decode_ms_over_it": round(res["avg_dec_ms"] /
                                                                 res["read_same_ms"], 4)},
            "prefill_traffic": (lambda t: None if t is None or res["kv_dtype"] != w.dtype else
                                {"bytes_per_launch": round(t[0]),
                                 "measured_over_algorithmic": round(t[1], 4)})(
                measured_prefill_traffic(args.workload)),
            "pool_GB": round(res["pool_gb"], 2),
        },
    }
    line = json.dumps(out)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")


if __name__ == "__main__":
    main()
