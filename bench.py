#!/usr/bin/env python3
"""Benchmark of the bounded chunk-prefill hot path on one MI355X.

One step = one streaming chunk through the whole path: bounded attention of
the chunk over [sink | W newest history tokens via the ring | causal chunk],
then the ring append of the chunk's K/V.  The history length advances by
the chunk length every step, so each step reads a different window phase
(the ring wraps inside key tiles).  Inputs are resident in HBM before the
timed region.

Default workload: one Qwen2.5-VL-7B-shaped attention layer -- 28 query /
4 KV heads, head_dim 128, sink 64, W = R = 16384, chunk 2048 -- the shape
the >= 50 % of bf16 MFMA peak target is stated on.  `--workload` selects the
others (3b, full, full_bounded, stream, append, and the query-side path:
query = retrieval + attention over the retrieved chunks, decode = one
decode step over them; drop = temporal token dropping of a batch of chunks).

Prints one JSON line.  `value` is algorithmic TFLOP/s over whole steps
(attention + append); `roofline` prices the attention kernel alone from
HIP events on its stream; `cpu_baseline` times the fp64 oracle on a bounded
sample of rows of the same chunk on the host cores.  The short-call
workloads (query, decode, drop, append) and the stream's aggregate rate are
timed over K calls launched back to back, with events only at the two ends;
their per-call event figures are printed beside them.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0


ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = "paper_2606_19849_amd/csrc/"
# sources whose kernels a traffic figure covers (it goes stale when any changes)
KERNEL_SRC = {"attn_fwd_kernel<128>": [CSRC + "attn_fwd.hip", CSRC + "attn_merge.hip", CSRC + "attn_common.h",
                                       CSRC + "vico_internal.h"],
              "attn_gather_kernel<128>": [CSRC + "attn_gather.hip", CSRC + "attn_merge.hip", CSRC + "attn_common.h",
                                          CSRC + "vico_internal.h"],
              "kv_append_kernel": [CSRC + "kv_append.hip"],
              "drop_sim_kernel<4>": [CSRC + "token_drop.hip", CSRC + "token_drop.h"],
              "drop_fused_kernel<4, 7>": [CSRC + "token_drop.hip", CSRC + "token_drop.h"]}


def kernel_source_sha256(kernel):
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SRC[kernel]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 summary of this kernel and
    workload, or None when there is none or the kernel source changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    fields = dict(line.split(":", 1) for line in open(path) if ":" in line and not line.startswith("#"))
    fields = {k.strip(): v.strip() for k, v in fields.items()}
    if fields.get("kernel") != kernel or fields.get("kernel_source_sha256") != kernel_source_sha256(kernel):
        return None
    return float(fields["hbm_bytes_per_launch"])


class Busy:
    """Matrix-core work on every CU (libvico_bench.so, register-only MFMA
    chains) used to hold the GPU under load: ahead of a loop of short calls it
    lets the host enqueue the calls faster than the GPU runs them, so the
    events around each call bracket its kernels rather than Python call
    overhead, and unlike an idle spin it keeps the engine clock where the
    power manager holds it under load (after an idle period the clock takes
    tens of milliseconds to climb back)."""

    def __init__(self, torch):
        import ctypes
        from paper_2606_19849_amd.build import BENCH_LIB
        lib = ctypes.CDLL(BENCH_LIB)
        self.fn = lib.vico_bench_mfma_peak
        self.fn.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
        self.fn.restype = ctypes.c_int32
        self.torch = torch
        self.groups = torch.cuda.get_device_properties(0).multi_processor_count
        self.sink = torch.empty(self.groups * 8, dtype=torch.float32, device="cuda")
        self.ms_per_iter = None

    def launch(self, iters, stream):
        if self.fn(self.groups, int(iters), self.sink.data_ptr(), stream.cuda_stream) != 0:
            raise RuntimeError("vico_bench_mfma_peak failed")

    def hold(self, stream, ms=4.0):
        torch = self.torch
        if self.ms_per_iter is None:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for _ in range(2):
                a.record(stream)
                self.launch(200, stream)
                b.record(stream)
                torch.cuda.synchronize()
            self.ms_per_iter = a.elapsed_time(b) / 200
        self.launch(max(1, ms / self.ms_per_iter), stream)


def back_to_back(torch, busy, stream, call, first, steps, hold_ms):
    """Seconds per call of call(first) .. call(first + steps - 1) launched back
    to back, with an event only before the first and after the last: an
    event recorded between two launches costs the GPU 2-3 us, a tenth of a
    short call.  A hold of `hold_ms` of matrix work first lets the host
    enqueue every call before the GPU reaches them."""
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    busy.hold(stream, ms=hold_ms)
    a.record(stream)
    for j in range(steps):
        call(first + j)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e-3 / steps


def warm_up(torch, call, min_steps, seconds):
    """Run `call(i)` for at least `min_steps` calls and `seconds` of wall time,
    back to back, so the timed loop starts with the GPU at its loaded clock
    (the power manager raises it over tens of milliseconds of work).  Returns
    the number of calls made."""
    i = 0
    t0 = time.perf_counter()
    while i < min_steps or time.perf_counter() - t0 < seconds:
        call(i)
        i += 1
        if i % 64 == 0:
            torch.cuda.synchronize()      # keep the queue short
    return i


def attn_flops(C, S, Wv, Hq, D, rows=None):
    """Algorithmic flops: 4*d per (query row, visible key) per head; masked pairs excluded."""
    r = np.arange(C) if rows is None else np.asarray(rows)
    return float(4 * Hq * D * np.sum(S + Wv + r + 1, dtype=np.float64))


def workload_shape(name):
    from synth import CONFIGS
    table = {"7b": "7b_wrap", "3b": "3b_wrap", "full": "full", "full_bounded": "full_bounded"}
    return CONFIGS[table[name]]


DESCR = {
    "7b": "qwen2.5-vl-7b layer chunk prefill: 28q/4kv heads, d128, sink 64, W=R=16384, chunk 2048",
    "3b": "qwen2.5-vl-3b layer chunk prefill: 16q/2kv heads, d128, sink 64, W=R=8192, chunk 1024",
    "full": "3b heads, full history 65536 + sink 64, chunk 2048 (unbounded control)",
    "full_bounded": "3b heads, history 65536 + sink 64, W=8192, chunk 2048",
    "stream": "3b heads, 64 chunks ragged in [256,1024], sink 64, W=R=8192, attend then append (one call per chunk)",
    "query": "qwen2.5-vl-7b query-side path per layer: mean of a 32-token query, cosine over 256 stored chunk "
             "features (dm 3584), top-32 chunks, attention of 32 query rows over sink 64 + retrieved chunks "
             "(256..1024 tokens each) + causal query; 28q/4kv, d128; 8 queries in rotation",
    "decode": "qwen2.5-vl-7b decode step per layer: 1 query row over sink 64 + 32 retrieved chunks + 64 tail "
              "tokens; 28q/4kv, d128; 8 retrieved sets in rotation",
    "drop": "temporal token dropping, qwen2.5-vl-7b projector output: 16 chunks x 4 frames x 256 tokens x 3584, "
            "tau 0.9, half the positions static; 4 input batches in rotation",
}


def cpu_model():
    """Host CPU model name (from /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(inp, n_rows, seed=0):
    """Time the fp64 oracle on `n_rows` rows (all heads) of the same chunk."""
    import oracle
    from tests._util import to_f64
    try:
        from threadpoolctl import threadpool_info
        cores = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:
        cores = len(os.sched_getaffinity(0))
    sh = inp.shape
    rows = np.linspace(0, sh.chunk_len - 1, n_rows).round().astype(np.int64)
    x = to_f64(inp)
    t0 = time.perf_counter()
    oracle.chunk_prefill_attention(**x, rows=rows)
    dt = time.perf_counter() - t0
    fl = attn_flops(sh.chunk_len, sh.sink_len, sh.visible_window, sh.num_q_heads, sh.head_dim, rows)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{n_rows} evenly spaced rows of the chunk x all {sh.num_q_heads} heads "
                      f"({fl / 1e9:.1f} GFLOP fp64) in {dt:.1f} s",
            "tokens_per_s": n_rows / dt}


def _dev(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def sustained_mfma_tflops(torch, stream, iters=2000, reps=5):
    """bf16 matrix-core rate the GPU sustains with every CU busy (register-only
    MFMA chains, two waves per SIMD; libvico_bench.so), median of `reps` timed
    launches on `stream`, in TFLOP/s.  Context for `roofline.peak`, which is the
    published figure at the 2.4 GHz peak engine clock."""
    import ctypes
    from paper_2606_19849_amd.build import BENCH_LIB
    lib = ctypes.CDLL(BENCH_LIB)
    fn = lib.vico_bench_mfma_peak
    fn.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int32
    groups = torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.empty(groups * 8, dtype=torch.float32, device="cuda")
    ms = []
    for r in range(reps + 2):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        st = fn(groups, iters, sink.data_ptr(), stream.cuda_stream)
        b.record(stream)
        if st != 0:
            raise RuntimeError(f"vico_bench_mfma_peak failed ({st})")
        torch.cuda.synchronize()
        if r >= 2:
            ms.append(a.elapsed_time(b))
    flops = groups * 8 * iters * 32 * 32768
    return flops / (float(np.median(ms)) * 1e-3) / 1e12


FLUSH_BYTES = 512 << 20      # > the 256 MB last-level cache + 8 x 4 MB L2


def run_chunk_workload(args, torch, vico):
    """Chunk prefill + append, timed in four variants: warm caches or flushed
    (a 512 MiB write before every step evicts the L2s and the last-level
    cache), and the wrapped ring phase of the workload (history = 5R + 777:
    the window starts mid-tile and one key tile straddles the ring end) or the
    aligned one (history = 5R: window start and ring end on tile bounds).  The
    history advances by the chunk length every step.  The headline (`value`,
    `roofline`) is the worst of the four."""
    from synth import make_chunk_inputs
    sh = workload_shape(args.workload)
    inp = make_chunk_inputs(sh, seed=0, family="F1")
    q, kc, vc = _dev(torch, inp.q), _dev(torch, inp.k_chunk), _dev(torch, inp.v_chunk)
    sk, sv = _dev(torch, inp.sink_k), _dev(torch, inp.sink_v)
    C, S, R, Hq, Hkv, D, W = (sh.chunk_len, sh.sink_len, sh.ring_slots, sh.num_q_heads, sh.num_kv_heads,
                              sh.head_dim, sh.window)
    # the resident history enters the ring through the library's own append
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    vico.vico_kv_append(_dev(torch, inp.hist_k), _dev(torch, inp.hist_v), rk, rv, inp.hist_first)
    out = torch.empty((C, Hq, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((Hq, C), dtype=torch.float32, device="cuda")
    full = W < 0
    K = args.steps
    # history of step i in each ring phase (the full-history control keeps its history fixed)
    phases = {"wrapped": lambda i: sh.hist_len + i * C} if not full else {"fixed": lambda i: sh.hist_len}
    if not full:
        phases["aligned"] = lambda i: (sh.hist_len // R) * R + i * C
        assert ((phases["aligned"](0) - min(W, phases["aligned"](0))) % R) % 64 == 0
    n_plan = max(K, 4096)
    wb = max(vico.vico_attn_plan(C, S, R, f(i), W, Hq, Hkv, D)[1] for f in phases.values() for i in (0, 1, 7, n_plan))
    splits = vico.vico_attn_plan(C, S, R, phases[next(iter(phases))](0), W, Hq, Hkv, D)[0]
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def step(H, events=None):
        if events:
            events[0].record(stream)
        vico.vico_chunk_prefill_attn(q, kc, vc, sk, sv, rk, rv, H, W, out, lse=lse, workspace=ws, stream=stream)
        if events:
            events[1].record(stream)
        if not full:
            vico.vico_kv_append(kc, vc, rk, rv, H, stream=stream)
        if events:
            events[2].record(stream)

    def flushed_step(H, j, events=None, fevents=None):
        if fevents:
            fevents[0].record(stream)
        flush.fill_(j & 255)
        if fevents:
            fevents[1].record(stream)
        step(H, events)

    fl = attn_flops(C, S, sh.visible_window, Hq, D)
    variants = {}
    n_warm = 0
    for cache in ("warm", "flushed"):
        for phase, H_of in phases.items():
            if args.only_variant and args.only_variant != f"{cache}_{phase}":
                continue
            ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(K)]
            fev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(2)) for _ in range(K)]
            # each variant is warmed up on its own steps right before it is timed: an idle
            # GPU drops its clock, and it takes tens of milliseconds of work to climb back
            if cache == "warm":
                nw = warm_up(torch, lambda i: step(H_of(i)), args.warmup, args.warmup_seconds)
            else:
                nw = warm_up(torch, lambda i: flushed_step(H_of(i), i), args.warmup, args.warmup_seconds)
            n_warm = max(n_warm, nw)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for j in range(K):
                if cache == "flushed":
                    flushed_step(H_of(nw + j), j, ev[j], fev[j])
                else:
                    step(H_of(nw + j), ev[j])
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            attn_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
            app_ms = np.array([e[1].elapsed_time(e[2]) for e in ev])
            flush_s = sum(a.elapsed_time(b) for a, b in fev) * 1e-3 if cache == "flushed" else 0.0
            step_s = (wall - flush_s) / K        # wall clock per step, flush kernels excluded
            variants[f"{cache}_{phase}"] = {
                "attn_us_mean": round(float(attn_ms.mean()) * 1e3, 2),
                "attn_us_median": round(float(np.median(attn_ms)) * 1e3, 2),
                "append_us_mean": round(float(app_ms.mean()) * 1e3, 2) if not full else None,
                "step_ms_wall": round(step_s * 1e3, 4),
                "attn_tflops": round(fl / (attn_ms.mean() * 1e-3) / 1e12, 2),
                "step_tflops": round(fl / step_s / 1e12, 2),
            }
    worst = min(variants, key=lambda k: variants[k]["step_tflops"])
    worst_attn = min(variants, key=lambda k: variants[k]["attn_tflops"])
    achieved = variants[worst_attn]["attn_tflops"]
    w = variants[worst]
    app_bytes = 2 * 2 * C * Hkv * D * 2          # K and V, read + write
    res = {
        "metric": "chunk-prefill attention TFLOP/s (% bf16 MFMA peak) + visual tokens/s per layer",
        "value": w["step_tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": K, "warmup": n_warm,
        "ms_per_step": w["step_ms_wall"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": DESCR[args.workload], "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D,
                   "sink": S, "window": W, "ring_slots": R, "chunk": C, "hist_start": sh.hist_len,
                   "splits": splits, "out_dtype": "bf16", "inputs": "N(0,1)/sqrt(d) bf16, seed 0"},
        "headline_variant": worst,
        "pct_peak": round(100 * w["step_tflops"] / PEAK_BF16_TFLOPS, 2),
        "visual_tokens_per_s": round(C / (w["step_ms_wall"] * 1e-3), 1),
        "attn_ms_mean": round(variants[worst_attn]["attn_us_mean"] * 1e-3, 4),
        "append_GBps": round(app_bytes / (w["append_us_mean"] * 1e-6) / 1e9, 1) if not full else None,
        "variants": variants,
        "warmup_seconds": args.warmup_seconds,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": args.traffic_bytes if args.traffic_bytes is not None
                     else measured_traffic("attn_fwd_kernel<128>", args.workload),
                     "kernel": "attn_fwd_kernel<128>", "variant": worst_attn,
                     "flops_per_launch": fl},
    }
    sustained = sustained_mfma_tflops(torch, stream)
    res["roofline"]["sustained_peak"] = round(sustained, 1)
    res["roofline"]["frac_of_sustained"] = round(achieved / sustained, 4)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_rows)
    return res


def run_ramp_study(args, torch, vico):
    """Chunk attention time against time since the GPU left an idle period:
    the power manager lowers the engine clock when the GPU idles and raises it
    again over tens of milliseconds of work, so a short timed loop that starts
    right after an idle gap (a host synchronisation followed by slow host
    work, or an idle spin kernel queued ahead of the loop) measures part of the
    climb.  Prints per-call times of consecutive batches after (a) 1 s of
    continuous work, (b) a 200 ms host sleep, (c) a 10 ms idle spin kernel."""
    from synth import make_chunk_inputs
    sh = workload_shape(args.workload)
    inp = make_chunk_inputs(sh, seed=0, family="F1")
    q, kc, vc = _dev(torch, inp.q), _dev(torch, inp.k_chunk), _dev(torch, inp.v_chunk)
    sk, sv = _dev(torch, inp.sink_k), _dev(torch, inp.sink_v)
    C, S, R, Hq, Hkv, D, W = (sh.chunk_len, sh.sink_len, sh.ring_slots, sh.num_q_heads, sh.num_kv_heads,
                              sh.head_dim, sh.window)
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    vico.vico_kv_append(_dev(torch, inp.hist_k), _dev(torch, inp.hist_v), rk, rv, inp.hist_first)
    out = torch.empty((C, Hq, D), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(vico.vico_attn_plan(C, S, R, sh.hist_len, W, Hq, Hkv, D)[1], 256), dtype=torch.uint8,
                     device="cuda")
    stream = torch.cuda.current_stream()
    fl = attn_flops(C, S, sh.visible_window, Hq, D)
    call = lambda: vico.vico_chunk_prefill_attn(q, kc, vc, sk, sv, rk, rv, sh.hist_len, W, out, workspace=ws,
                                                stream=stream)

    def batches(n_batches, per=4):
        evs = []
        for b in range(n_batches):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(per):
                call()
            e1.record(stream)
            evs.append((e0, e1))
        torch.cuda.synchronize()
        t = np.cumsum([a.elapsed_time(b) for a, b in evs])
        return [(round(float(tt), 2), round(a.elapsed_time(b) / per * 1e3, 1)) for tt, (a, b) in zip(t, evs)]

    warm_up(torch, lambda i: call(), 10, 1.0)
    res = {"after_continuous_work_ms_us": batches(40)}
    time.sleep(0.2)
    res["after_200ms_host_sleep_ms_us"] = batches(40)
    warm_up(torch, lambda i: call(), 10, 1.0)
    torch.cuda._sleep(20_000_000)
    res["after_10ms_idle_spin_ms_us"] = batches(40)
    steady = np.median([x[1] for x in res["after_continuous_work_ms_us"]])
    return {"metric": "chunk attention time after idle (clock ramp study)", "value": round(float(steady), 1),
            "unit": "us per call, steady", "n_gpus": 1, "steps": 160, "warmup": None, "higher_is_better": False,
            "config": {"workload": DESCR[args.workload]}, "flops_per_call": fl,
            "series": "pairs (ms since the first batch began, us per call of that batch of 4)", **res}


def run_stream_workload(args, torch, vico):
    """64 ragged chunks at the 3B shape: aggregate visual tokens/s, and
    per-chunk latency vs chunk index.  Each repetition replays the stream
    twice: once with events only before the first and after the last chunk
    (the aggregate rate: an event recorded between two launches costs the
    GPU 2-3 us, 5 % of a chunk), and once with one event per chunk boundary
    (the per-chunk latencies and their drift)."""
    from synth import ragged_chunk_lengths, stream_chunk, stream_sink
    dev = lambda bits: _dev(torch, bits)
    Hq, Hkv, D, S, W, R = 16, 2, 128, 64, 8192, 8192
    counts = ragged_chunk_lengths(64, 256, 1024, seed=0)
    res_all = {}
    for mode, window, slots in (("bounded", W, R), ("full", -1, int(counts.sum()))):
        sk_b, sv_b = stream_sink(S, Hkv, D, seed=0)
        sk, sv = dev(sk_b), dev(sv_b)
        rk = torch.zeros((slots, Hkv, D), dtype=torch.bfloat16, device="cuda")
        rv = torch.zeros_like(rk)
        chunks = [tuple(dev(x) for x in stream_chunk(t, int(c), Hq, Hkv, D, seed=0)) for t, c in enumerate(counts)]
        starts = np.concatenate([[0], np.cumsum(counts)])
        wb = max(vico.vico_attn_plan(int(c), S, slots, int(starts[t]), window, Hq, Hkv, D)[1]
                 for t, c in enumerate(counts))
        ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
        outs = [torch.empty((int(c), Hq, D), dtype=torch.bfloat16, device="cuda") for c in counts]
        stream = torch.cuda.current_stream()
        lat = np.zeros((args.steps, len(counts)))
        whole = np.zeros(args.steps)
        busy = Busy(torch)
        t_warm = time.perf_counter()
        rep, n_warm = 0, None

        def chunk(t):
            q, k, v = chunks[t]
            # attend, then append the chunk to the ring, in one call
            vico.vico_chunk_prefill_attn(q, k, v, sk, sv, rk, rv, int(starts[t]), window, outs[t],
                                         workspace=ws, stream=stream, flags=vico.VICO_ATTN_APPEND)

        hold_ms = 6.0
        while n_warm is None or rep < n_warm + args.steps:
            if n_warm is None and rep >= args.warmup and time.perf_counter() - t_warm >= args.warmup_seconds:
                n_warm = rep
            ends = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            busy.hold(stream, ms=hold_ms)
            ends[0].record(stream)
            t_host = time.perf_counter()
            for t in range(len(counts)):
                chunk(t)
            # the hold must outlast the host's enqueueing of the 64 calls, or
            # the GPU would wait for the host inside the timed span
            hold_ms = max(hold_ms, 1.5e3 * (time.perf_counter() - t_host))
            ends[1].record(stream)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(counts) + 1)]
            busy.hold(stream, ms=hold_ms)
            ev[0].record(stream)
            for t in range(len(counts)):
                chunk(t)
                ev[t + 1].record(stream)
            torch.cuda.synchronize()
            if n_warm is not None:
                whole[rep - n_warm] = ends[0].elapsed_time(ends[1])
                lat[rep - n_warm] = [a.elapsed_time(b) for a, b in zip(ev, ev[1:])]
            rep += 1
        med = np.median(lat, axis=0)
        flops = np.array([attn_flops(int(c), S, min(int(starts[t]), W) if window >= 0 else int(starts[t]), Hq, D)
                          for t, c in enumerate(counts)])
        # latency = a + b * flops + c * t over the chunks whose window is full
        t_idx = np.arange(len(counts))
        sel = starts[:-1] >= W if window >= 0 else np.ones(len(counts), bool)
        X = np.stack([np.ones(sel.sum()), flops[sel], t_idx[sel]], 1)
        coef = np.linalg.lstsq(X, med[sel], rcond=None)[0]
        res_all[mode] = {
            "stream_ms": round(float(np.median(whole)), 4),
            "tokens_per_s": round(float(counts.sum() / (np.median(whole) * 1e-3)), 1),
            "per_chunk_ms": [round(float(x), 4) for x in med],
            "tokens_per_s_chunk_events": round(float(counts.sum() / (med.sum() * 1e-3)), 1),
            "tflops_per_chunk": [round(float(f / (m * 1e-3) / 1e12), 1) for f, m in zip(flops, med)],
            "drift_ms_over_64_chunks": round(float(coef[2] * 63), 4),
            "mean_ms": round(float(med.mean()), 4),
        }
    b = res_all["bounded"]
    return {
        "metric": "chunk-prefill attention TFLOP/s (% bf16 MFMA peak) + visual tokens/s per layer",
        "value": b["tokens_per_s"], "unit": "visual tokens/s per layer",
        "n_gpus": 1, "steps": args.steps, "warmup": n_warm,
        "ms_per_step": b["stream_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": DESCR["stream"], "chunks": len(counts), "tokens": int(counts.sum())},
        "stream": res_all,
    }


def run_query_workload(args, torch, vico):
    """Query-side path on the 7B shape: retrieval (query mean, cosine scores,
    top-k with segment table) and attention over the retrieved chunks for one
    layer (`query`), or one decode step over a retrieved set (`decode`).
    The store holds 256 chunks (336 MB of K/V, more than the 256 MB
    last-level cache); 8 queries in rotation read different chunks."""
    import dataclasses
    from synth import QUERY_CONFIGS, make_query_inputs
    decode = args.workload == "decode"
    base = QUERY_CONFIGS["q_7b"]
    if decode:
        base = dataclasses.replace(base, tail_len=64)
    n_q = 8
    qis = [make_query_inputs(base, seed=0, query_seed=j) for j in range(n_q)]
    qi0 = qis[0]
    sh = qi0.shape
    Lq = 1 if decode else sh.q_len
    dev = lambda bits: _dev(torch, bits)
    k_np, v_np = qi0.store_kv()
    gk, gv = dev(k_np), dev(v_np)
    del k_np, v_np
    sk, sv = dev(qi0.sink_k), dev(qi0.sink_v)
    feats = torch.from_numpy(qi0.chunk_feat).cuda()
    cstart = torch.from_numpy(qi0.chunk_start).cuda()
    clen = torch.from_numpy(qi0.chunk_len.astype(np.int32)).cuda()
    qs = [dict(x=dev(qi.query_x), q=dev(qi.q)[-Lq:].contiguous(), tk=dev(qi.tail_k), tv=dev(qi.tail_v),
               ss=torch.empty(sh.top_k, dtype=torch.int64, device="cuda"),
               sl=torch.empty(sh.top_k, dtype=torch.int32, device="cuda")) for qi in qis]
    qf = torch.empty(sh.feat_dim, dtype=torch.float32, device="cuda")
    scores = torch.empty(sh.num_chunks, dtype=torch.float32, device="cuda")
    oc = torch.empty(sh.top_k, dtype=torch.int32, device="cuda")
    osc = torch.empty(sh.top_k, dtype=torch.float32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    hint = sh.top_k * (sh.chunk_lo + sh.chunk_hi) // 2
    parts, wb = vico.vico_gather_plan(Lq, sh.tail_len, sh.sink_len, qi0.store_len, sh.top_k, hint,
                                      sh.num_q_heads, sh.num_kv_heads, sh.head_dim)
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    out = torch.empty((Lq, sh.num_q_heads, sh.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((sh.num_q_heads, Lq), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def retrieve(d):
        vico.vico_token_mean(d["x"], qf, stream=stream)
        vico.vico_chunk_scores(qf, feats, scores, stream=stream)
        vico.vico_topk_chunks(scores, sh.top_k, oc, osc, cnt, chunk_start=cstart, chunk_len=clen,
                              seg_start=d["ss"], seg_len=d["sl"], stream=stream)

    def attend(d):
        vico.vico_gather_attn(d["q"], d["tk"], d["tv"], sk, sv, gk, gv, d["ss"], d["sl"], out, lse=lse,
                              workspace=ws, keys_hint=hint, stream=stream)

    # every query's segment table once (decode steps reuse them)
    for d in qs:
        retrieve(d)
    torch.cuda.synchronize()
    gathered = [int(d["sl"].sum().item()) for d in qs]

    def step(j, events=None):
        d = qs[j % n_q]
        if events:
            events[0].record(stream)
        if not decode:
            retrieve(d)
        if events:
            events[1].record(stream)
        attend(d)
        if events:
            events[2].record(stream)

    n_warm = warm_up(torch, step, args.warmup, args.warmup_seconds)
    busy = Busy(torch)
    # per-call events (retrieval and attention of each step apart)
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    busy.hold(stream)
    for j in range(args.steps):
        step(n_warm + j, ev[j])
    torch.cuda.synchronize()
    host_paced = args.steps / (time.perf_counter() - t0)
    ret_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    att_ms = np.array([e[1].elapsed_time(e[2]) for e in ev])
    # the same K calls with no events between them (the value and the roofline)
    hold_ms = max(4.0, 1.25e3 * args.steps / host_paced)
    lean = lambda call: back_to_back(torch, busy, stream, call, n_warm, args.steps, hold_ms)
    step_s = lean(step)
    attn_s = lean(lambda j: attend(qs[j % n_q]))
    ret_s = None if decode else lean(lambda j: retrieve(qs[j % n_q]))
    Hq, Hkv, D, S, T = sh.num_q_heads, sh.num_kv_heads, sh.head_dim, sh.sink_len, sh.tail_len
    G = np.array([gathered[(n_warm + j) % n_q] for j in range(args.steps)], dtype=np.float64)
    keys = S + G + T
    kv_bytes = keys * Hkv * D * 2 * 2
    bytes_ = kv_bytes + Lq * Hq * D * 2 * 2 + Hq * Lq * 4            # + Q, O (bf16), LSE
    rows = T - Lq + np.arange(Lq) + 1                                   # visible tail keys per query row
    flops = np.array([4.0 * Hq * D * float(np.sum(S + g + rows)) for g in G])
    gbs = float(bytes_.mean() / attn_s / 1e9)
    tfl = float(flops.mean() / attn_s / 1e12)
    t_hbm = bytes_.mean() / (PEAK_HBM_GBS * 1e9)
    t_mfma = flops.mean() / (PEAK_BF16_TFLOPS * 1e12)
    res = {
        "metric": ("decode-step attention per layer" if decode else
                   "query-side retrieval + gathered attention per layer (TTFT building block)"),
        "value": round(1.0 / step_s, 1), "unit": "steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": n_warm, "ms_per_step": round(step_s * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": DESCR[args.workload], "q_rows": Lq, "tail": T, "top_k": sh.top_k,
                   "stored_chunks": sh.num_chunks, "store_tokens": qi0.store_len, "parts": parts,
                   "gathered_keys_mean": float(G.mean())},
        "host_paced_steps_per_s": round(host_paced, 1),
        "retrieval_us_mean": None if decode else round(ret_s * 1e6, 2),
        "attn_us_mean": round(attn_s * 1e6, 2),
        "attn_tflops": round(tfl, 2),
        "per_call_events": {"retrieval_us_mean": None if decode else round(float(ret_ms.mean()) * 1e3, 2),
                            "attn_us_mean": round(float(att_ms.mean()) * 1e3, 2),
                            "attn_us_median": round(float(np.median(att_ms)) * 1e3, 2)},
        "roofline": {"bound": "hbm" if t_hbm >= t_mfma else "mfma",
                     "achieved": round(gbs, 1) if t_hbm >= t_mfma else round(tfl, 2),
                     "peak": PEAK_HBM_GBS if t_hbm >= t_mfma else PEAK_BF16_TFLOPS,
                     "unit": "GB/s" if t_hbm >= t_mfma else "TFLOP/s",
                     "frac": round(gbs / PEAK_HBM_GBS if t_hbm >= t_mfma else tfl / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic("attn_gather_kernel<128>", args.workload),
                     "kernel": "attn_gather_kernel<128> (+ split merge)",
                     "bytes_per_launch_mean": float(bytes_.mean()), "flops_per_launch_mean": float(flops.mean())},
    }
    return res


def run_drop_workload(args, torch, vico):
    """Temporal token dropping of a batch of chunks (HBM bound): algorithmic
    bytes = the frames read once + the retained tokens and their indices
    written once.  --drop-schedule picks the single pass (a workspace given,
    the default) or the two passes (none)."""
    from synth import make_drop_frames
    B, C, n_f, dm, tau = 16, 4, 256, 3584, 0.9
    n_batches = 4
    batches = [_dev(torch, make_drop_frames(B, C, n_f, dm, seed=j)) for j in range(n_batches)]
    keep = torch.empty((B, n_f), dtype=torch.uint8, device="cuda")
    idx = torch.empty(B * C * n_f, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    out = torch.empty((B * C * n_f, dm), dtype=torch.bfloat16, device="cuda")
    single = args.drop_schedule == "single_pass"
    ws = None
    if single:
        nb = vico.vico_temporal_drop_workspace_bytes(B, C, n_f, dm)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def call(fr):
        vico.vico_temporal_drop(fr, tau, keep, idx, cnt, out_tokens=out, workspace=ws, stream=stream)

    kept = []
    for fr in batches:
        call(fr)
        torch.cuda.synchronize()
        kept.append(int(cnt.item()))
        if kept[-1] < 0:
            raise RuntimeError("temporal drop: a bounded wait of the single pass gave up")
    n_warm = warm_up(torch, lambda j: call(batches[j % n_batches]), args.warmup, args.warmup_seconds)
    busy = Busy(torch)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    busy.hold(stream)
    for j in range(args.steps):
        ev[j][0].record(stream)
        call(batches[(n_warm + j) % n_batches])
        ev[j][1].record(stream)
    torch.cuda.synchronize()
    if int(cnt.item()) != kept[(n_warm + args.steps - 1) % n_batches]:
        raise RuntimeError("temporal drop: the last timed call retained a different count")
    host_paced = B * C * n_f * args.steps / (time.perf_counter() - t0)
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    # the same K calls with no events between them (the value and the roofline)
    call_s = back_to_back(torch, busy, stream, lambda j: call(batches[j % n_batches]), n_warm, args.steps,
                          max(4.0, 1.25e3 * args.steps * B * C * n_f / host_paced))
    if int(cnt.item()) != kept[(n_warm + args.steps - 1) % n_batches]:
        raise RuntimeError("temporal drop: the last timed call retained a different count")
    n_keep = np.array([kept[(n_warm + j) % n_batches] for j in range(args.steps)], dtype=np.float64)
    in_bytes = B * C * n_f * dm * 2
    alg = in_bytes + n_keep * (dm * 2 + 4) + B * n_f
    gbs = float(alg.mean() / call_s / 1e9)
    kernel = "drop_fused_kernel<4, 7>" if single else "drop_sim_kernel<4>"
    return {
        "metric": "temporal token dropping throughput (input tokens/s)",
        "value": round(B * C * n_f / call_s, 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": n_warm, "ms_per_step": round(call_s * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": DESCR["drop"], "retention": round(float(n_keep.mean()) / (B * C * n_f), 4),
                   "schedule": args.drop_schedule},
        "call_us_mean": round(call_s * 1e6, 2),
        "per_call_events": {"call_us_mean": round(float(ms.mean()) * 1e3, 2)},
        "host_paced_tokens_per_s": round(host_paced, 1),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": measured_traffic(kernel, "drop" if single else "drop_two_pass"),
                     "kernel": "drop_fused_kernel<4, 7>" if single else "drop_sim_kernel<4> + drop_compact_kernel",
                     "bytes_per_launch_mean": float(alg.mean())},
    }


def run_append_workload(args, torch, vico):
    """Ring append at capacity (chunk = ring = 16384 tokens of the 7B shape): HBM roofline
    of the append kernel, which is also a plain copy of known size."""
    R, Hkv, D = 16384, 4, 128
    C = R
    g = torch.Generator(device="cuda").manual_seed(0)
    k = torch.randn((C, Hkv, D), device="cuda", generator=g).to(torch.bfloat16)
    v = torch.randn((C, Hkv, D), device="cuda", generator=g).to(torch.bfloat16)
    rk = torch.zeros((R, Hkv, D), dtype=torch.bfloat16, device="cuda")
    rv = torch.zeros_like(rk)
    stream = torch.cuda.current_stream()
    n_warm = warm_up(torch, lambda i: vico.vico_kv_append(k, v, rk, rv, 777 + i, stream=stream), args.warmup,
                     args.warmup_seconds)
    busy = Busy(torch)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    busy.hold(stream)
    for i in range(args.steps):
        ev[i][0].record(stream)
        vico.vico_kv_append(k, v, rk, rv, 777 + i * 1000, stream=stream)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    host_paced = 2 * 2 * C * Hkv * D * 2 * args.steps / wall / 1e9
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    nbytes = 2 * 2 * C * Hkv * D * 2
    # the same K calls with no events between them (the value and the roofline)
    call_s = back_to_back(torch, busy, stream, lambda i: vico.vico_kv_append(k, v, rk, rv, 777 + i * 1000,
                                                                             stream=stream),
                          0, args.steps, max(4.0, 1.25e3 * wall))
    gbs = nbytes / call_s / 1e9
    return {
        "metric": "ring append HBM GB/s", "value": round(gbs, 1), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": n_warm, "ms_per_step": round(call_s * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "ring append at capacity: 16384 tokens x 4 kv heads x d128, K and V, ring wraps",
                   "bytes_per_launch": nbytes},
        "per_call_events": {"GBps": round(nbytes / (ms.mean() * 1e-3) / 1e9, 1)},
        "host_paced_GBps": round(host_paced, 1),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": args.traffic_bytes if args.traffic_bytes is not None
                     else measured_traffic("kv_append_kernel", "append"),
                     "kernel": "kv_append_kernel"},
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="warm-up also lasts at least this long, so timing starts at the loaded clock")
    ap.add_argument("--workload", default="7b", choices=["7b", "3b", "full", "full_bounded", "stream", "append", "query", "decode",
                                                          "drop"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--drop-schedule", default="single_pass", choices=["single_pass", "two_pass"],
                    help="drop workload: single pass (workspace given) or two passes")
    ap.add_argument("--only-variant", default=None,
                    help="chunk workloads: time only this variant (e.g. warm_wrapped), for profiling runs")
    ap.add_argument("--ramp", action="store_true",
                    help="instead of the benchmark: chunk attention time against time since an idle period")
    ap.add_argument("--cpu-rows", type=int, default=2048)
    ap.add_argument("--traffic-bytes", type=float, default=None,
                    help="HBM bytes per attention launch from rocprofv3 FETCH_SIZE+WRITE_SIZE, if measured")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the library runs on one GPU only; sharding by KV-head group across GPUs is "
              "a design, not built", file=sys.stderr)
        sys.exit(2)
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import torch
    import paper_2606_19849_amd as vico
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    vico.load_library()
    if args.ramp:
        res = run_ramp_study(args, torch, vico)
    elif args.workload == "stream":
        res = run_stream_workload(args, torch, vico)
    elif args.workload == "append":
        res = run_append_workload(args, torch, vico)
    elif args.workload in ("query", "decode"):
        res = run_query_workload(args, torch, vico)
    elif args.workload == "drop":
        res = run_drop_workload(args, torch, vico)
    else:
        res = run_chunk_workload(args, torch, vico)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
