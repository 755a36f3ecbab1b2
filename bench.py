"""Benchmark of the HERMES streaming step on one MI355X.

A step is one chunk append over every layer (attention, attention mass) plus
the compression (scoring, smoothing, top-k, gather-compaction) of the 28-layer
7B-shaped cache: 8192 cached tokens + 784 new (4 frames x 196 tokens) per
layer, per-layer budgets ramping 2048 -> 6144.  Between steps the context is
rewound on the host to the untouched initial cache (compaction writes the
other buffer of each pair), so every timed step does identical work with no
restore copy.

Prints ONE JSON line:  metric, value (video tokens appended+compressed per
second), ms_per_step, the roofline of the dominant kernel (HIP events around
its launches in the timed region), and the fp64 CPU oracle timed on a bounded
sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "video tokens/s appended+compressed (all layers) at 7B shape; % MFMA / HBM peak"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E

# HBM bytes per attn_fwd launch on the 28-layer workload, from the FETCH_SIZE
# and WRITE_SIZE counter passes in profiles/traffic_c3_7b_28layer.md (fetch
# scaled x2.000, write x1.000 by a 256 MiB copy).  Valid only for the kernel
# source it was measured on: reported as null once attention.hip changes.
ATTN_TRAFFIC = {"bytes": 1.2163e9, "source_sha256_16": "daa91be90110cf74",
                "workload": "c3_7b_28layer"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attention_flops(wl) -> float:
    """Algorithmic FLOPs of the causal chunk attention over all layers:
    4 d per visible (query row, candidate, head) triple (QK^T and PV)."""
    C, T0 = wl.chunk, wl.init_len
    pairs = wl.n_layers * wl.n_q_heads * (C * T0 + C * (C + 1) // 2)
    return 4.0 * wl.head_dim * pairs


def gather_bytes(wl) -> float:
    """Algorithmic bytes of the gather: each kept row of K and V read and
    written once, plus its position (read + write)."""
    row = wl.n_kv_heads * wl.head_dim * 2
    T = wl.init_len + wl.chunk
    kept = sum(min(T, b) for b in wl.budgets if T > b)
    return kept * (4.0 * row + 8.0)


def select_bytes(wl) -> float:
    """Algorithmic bytes of scoring + top-k: W and positions of every
    evicting layer and of the layer above it read once, the kept list
    written (the fp32 keys round trip between the two select launches is
    working memory, not counted)."""
    T = wl.init_len + wl.chunk
    n = 0.0
    for l, b in enumerate(wl.budgets):
        if T > b:
            n += 8.0 * T + (8.0 * T if l + 1 < wl.n_layers else 0.0) + 4.0 * b
    return n


def attn_traffic(wl):
    import hashlib
    src = os.path.join(ROOT, "paper_2601_14724_amd", "csrc", "attention.hip")
    with open(src, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()[:16]
    if sha != ATTN_TRAFFIC["source_sha256_16"] or wl.name != ATTN_TRAFFIC["workload"]:
        return None
    return ATTN_TRAFFIC["bytes"]


def _cpu_model() -> str:
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, n_layers: int) -> dict:
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import hermes_oracle as orc
    from paper_2601_14724_amd import workloads as wk
    f64 = wk.bf16_bits_to_f64
    layers = list(range(n_layers))
    caches = [wk.gen_cache(wl, l) for l in layers]
    chunks = [wk.gen_chunk(wl, 0, l) for l in layers]
    oc = [orc.LayerCache(f64(c["k"]), f64(c["v"]), c["pos"].astype(np.int64)) for c in caches]
    och = [{"q": f64(c["q"]), "k": f64(c["k"]), "v": f64(c["v"]), "pos": c["pos"]} for c in chunks]
    classes = orc.layer_partition(wl.n_layers)[:n_layers]
    cfg = orc.OracleConfig(budgets=list(wl.budgets[:n_layers]), classes=classes,
                           lambdas=orc.smoothing_lambdas(orc.layer_partition(wl.n_layers))[:n_layers])
    # the oracle's BLAS calls run on every core this process may use
    affinity = len(os.sched_getaffinity(0))
    with threadpool_limits(affinity):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        t0 = time.perf_counter()
        orc.stream_step(oc, och, cfg)
        dt = time.perf_counter() - t0
    per_step = dt * wl.n_layers / n_layers
    return {"value": wl.chunk / per_step, "unit": "video tokens/s", "cores": int(min(threads, affinity)),
            "kind": "oracle", "affinity_cores": affinity, "host_cpus": os.cpu_count(),
            "cpu_model": _cpu_model(),
            "sample": f"fp64 oracle step (attention+mass, scoring, smoothing, top-k, gather) on "
                      f"layers 0..{n_layers - 1} of the 28-layer workload, {dt:.1f} s, scaled "
                      f"x{wl.n_layers}/{n_layers} to the whole step; matrix products on "
                      f"{min(threads, affinity)} BLAS threads, element-wise work on one"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c3_7b_28layer")
    ap.add_argument("--cpu-sample-layers", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extensions", action="store_true",
                    help="skip the summary-token / re-indexing / guidance-prompt timings")
    ap.add_argument("--no-c4", action="store_true",
                    help="skip the 64-chunk stream from an empty cache")
    ap.add_argument("--no-c5", action="store_true",
                    help="skip the long-cache configuration (32768 + 3136 tokens, 64-token query)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        log("the streaming step runs on one GPU and is not sharded across GPUs; --gpus must be 1")
        return 2

    import torch

    from paper_2601_14724_amd import hermes as H
    from paper_2601_14724_amd import streaming, workloads as wk

    wl = wk.WORKLOADS[args.workload]
    log(f"[bench] generating inputs for {wl.name}")
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        caches = list(ex.map(lambda l: wk.gen_cache(wl, l), range(wl.n_layers)))
        chunks = list(ex.map(lambda l: wk.gen_chunk(wl, 0, l), range(wl.n_layers)))
    dev = "cuda:0"
    torch.cuda.set_device(0)
    kv = streaming.make_cache(wl, device=dev, caches=caches)
    st = {k: np.stack([c[k] for c in chunks]) for k in ("q", "k", "v")} | {"pos": chunks[0]["pos"]}
    t = streaming.chunk_tensors(st, dev)
    out = torch.empty_like(t["q"])
    del chunks, st

    def step():
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=out)
        kv.compress()

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Every event recorded on the stream leaves the GPU idle for ~10 us, so
    # each figure comes from its own pass with only the events it needs.
    # 1) The headline: K steps back to back, synchronised on both sides.
    log(f"[bench] timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # 2) Spread over steps: one event pair around each step.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for e0, e1 in ev:
        e0.record()
        step()
        e1.record()
    torch.cuda.synchronize()
    step_ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
    # 3) The select + compaction window (scoring, top-k, gather): events
    #    around compress() only.
    cw = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for c0, c1 in cw:
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=out)
        c0.record()
        kv.compress()
        c1.record()
    torch.cuda.synchronize()
    sc_all = sorted(c0.elapsed_time(c1) for c0, c1 in cw)
    # 4) Per-kernel breakdown from the library's own events around each launch.
    kv.profile(True)
    for kid in range(len(H.KERNEL_NAMES)):
        kv.profile_read(kid)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kernels = {}
    for kid, name in enumerate(H.KERNEL_NAMES):
        ms, cnt = kv.profile_read(kid)
        if cnt:   # per step: a group may hold several launches
            kernels[name] = {"avg_ms": ms / args.steps, "launches": cnt}
    kv.profile(False)

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calib_copy_mib} MiB done")

    ms_step = 1e3 * elapsed / args.steps
    value = wl.chunk * args.steps / elapsed
    fl = attention_flops(wl)
    att_ms = kernels["attention"]["avg_ms"]
    achieved = fl / (att_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": attn_traffic(wl),
                "kernel": "attn_fwd", "flops_per_launch": fl}
    gb = gather_bytes(wl)
    extra = {"kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()}}
    if "gather" in kernels:
        g = gb / (kernels["gather"]["avg_ms"] * 1e-3) / 1e9
        extra["gather_GBps"] = round(g, 1)
        extra["gather_hbm_frac"] = round(g / PEAK_HBM_GBS, 4)
    sc_ms = sc_all[len(sc_all) // 2]
    sc = (gb + select_bytes(wl)) / (sc_ms * 1e-3) / 1e9
    extra["select_compaction"] = {"ms": round(sc_ms, 4), "min_ms": round(sc_all[0], 4),
                                  "bytes": gb + select_bytes(wl), "GBps": round(sc, 1),
                                  "hbm_frac": round(sc / PEAK_HBM_GBS, 4),
                                  "window": "compress(): score_keys, select_kept, gather_rows (median)"}
    if "colsum" in kernels:
        sweep = attention_flops(wl) / 2 * _mass_layer_fraction(wl)
        extra["colsum_TFLOPs_executed"] = round(sweep / (kernels["colsum"]["avg_ms"] * 1e-3) / 1e12, 2)
    extra["step_ms"] = {"median": round(step_ms[len(step_ms) // 2], 4), "min": round(step_ms[0], 4)}
    qres = query_bench(wl, kv, args.steps, args.warmup)
    kv.close()
    c4 = None
    if not args.no_c4 and args.workload == "c3_7b_28layer":
        log("[bench] 64-chunk stream from an empty cache (7B shape, budget 6144)")
        c4 = c4_bench()
    c5 = None
    if not args.no_c5 and args.workload == "c3_7b_28layer":
        log("[bench] long cache: 32768 + 3136 tokens per layer, then a 64-token query")
        c5 = c5_bench(min(args.steps, 10), min(args.warmup, 3))
    ext = None
    if not args.no_extensions:
        log("[bench] adjacent rows: summary tokens + eager re-indexing, guidance prompt")
        ext = extension_bench(wl, caches, t, args.steps, args.warmup)
    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] oracle CPU baseline on {args.cpu_sample_layers} layers")
        cpu = cpu_baseline(wl, args.cpu_sample_layers)
    rec = {"metric": METRIC, "value": round(value, 1), "unit": "video tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded Gaussian Q/K/V, low-rank keys, RoPE theta 1e6)",
           "config": {"workload": wl.name, "n_layers": wl.n_layers, "n_q_heads": wl.n_q_heads,
                      "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                      "cached_tokens": wl.init_len, "chunk_tokens": wl.chunk,
                      "budgets": f"{wl.budgets[0]}..{wl.budgets[-1]} (linear ramp)",
                      "parallelism": "single GPU"},
           "roofline": roofline, "cpu_baseline": cpu, **extra}
    rec["query"] = qres
    if c4 is not None:
        rec["c4_stream"] = c4
    if c5 is not None:
        rec["c5_long"] = c5
    if ext is not None:
        rec["extensions"] = ext
    print(json.dumps(rec), flush=True)
    return 0


def c4_bench() -> dict:
    """The 64-chunk stream of the 7B shape from an empty cache, budget 6144 on
    every layer (steps 0-6 fill the cache, steps 7-63 evict): one untimed
    pass, then one timed pass on a fresh context.  Every step's
    inputs are generated and uploaded before timing (12.9 GB of HBM)."""
    import torch

    from paper_2601_14724_amd import streaming, workloads as wk
    wl = wk.WORKLOADS["c4_7b_stream64"]
    cap = max(wl.budgets) + wl.chunk
    kv = streaming.make_cache(wl, device="cuda:0", cap=cap)
    steps = []
    for s in range(wl.n_steps):
        steps.append(streaming.chunk_tensors(wk.stack_chunks(wl, s), "cuda:0"))
    out = torch.empty_like(steps[0]["q"])

    def run():
        for t in steps:
            kv.append(t["q"], t["k"], t["v"], t["pos"], out=out)
            kv.compress()

    run()
    kv.close()   # compaction has overwritten both buffers: a fresh context starts empty
    # the whole stream with events only at its ends (every event leaves the
    # GPU idle for ~10 us), then a second stream with one event per step for
    # the per-step figures
    kv = streaming.make_cache(wl, device="cuda:0", cap=cap)
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    g0.record()
    run()
    g1.record()
    torch.cuda.synchronize()
    total = g0.elapsed_time(g1)
    kv.close()
    kv = streaming.make_cache(wl, device="cuda:0", cap=cap)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(wl.n_steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i, t in enumerate(steps):
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=out)
        kv.compress()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(wl.n_steps)]
    kv.close()
    del steps
    first_evict = next(s for s in range(wl.n_steps) if (s + 1) * wl.chunk > max(wl.budgets))
    ev_steps = sorted(per[first_evict:])
    return {"workload": wl.name, "steps": wl.n_steps, "ms_total": round(total, 3),
            "video_tokens_per_s": round(wl.chunk * wl.n_steps / (total * 1e-3), 1),
            "evicting_step_ms": {"median": round(ev_steps[len(ev_steps) // 2], 4),
                                 "min": round(ev_steps[0], 4)},
            "algorithmic_tflop": round(_stream_flops(wl) / 1e12, 2),
            "attention_tflops_avg": round(_stream_flops(wl) / (total * 1e-3) / 1e12, 1)}


def _stream_flops(wl) -> float:
    """Algorithmic attention FLOPs of a stream from an empty cache: the cache
    before step s holds min(s*C, budget) tokens."""
    C, d, M = wl.chunk, wl.head_dim, max(wl.budgets)
    pairs = 0
    for s in range(wl.n_steps):
        t0 = min(s * C, M)
        pairs += wl.n_layers * wl.n_q_heads * (C * t0 + C * (C + 1) // 2)
    return 4.0 * d * pairs


def c5_bench(steps: int, warmup: int) -> dict:
    """The long-cache configuration of the 7B shape: 32768 cached + 3136 new
    tokens per layer (budgets 4096..16384), one append + compress per step
    with the cache rewound between steps, then the 64-token query over the
    compacted caches."""
    import concurrent.futures as cf

    import torch

    from paper_2601_14724_amd import hermes as H
    from paper_2601_14724_amd import streaming, workloads as wk
    wl = wk.WORKLOADS["c5_7b_long"]
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        caches = list(ex.map(lambda l: wk.gen_cache(wl, l), range(wl.n_layers)))
        chunks = list(ex.map(lambda l: wk.gen_chunk(wl, 0, l), range(wl.n_layers)))
    kv = streaming.make_cache(wl, device="cuda:0", caches=caches)
    st = {k: np.stack([c[k] for c in chunks]) for k in ("q", "k", "v")} | {"pos": chunks[0]["pos"]}
    t = streaming.chunk_tensors(st, "cuda:0")
    out = torch.empty_like(t["q"])
    del caches, chunks, st

    def step():
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=out)
        kv.compress()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kv.profile(True)
    for kid in range(len(H.KERNEL_NAMES)):
        kv.profile_read(kid)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    kernels = {}
    for kid, name in enumerate(H.KERNEL_NAMES):
        ms, cnt = kv.profile_read(kid)
        if cnt:
            kernels[name] = round(ms / steps, 4)
    kv.profile(False)
    fl = attention_flops(wl)
    att_tf = fl / (kernels["attention"] * 1e-3) / 1e12
    res = {"workload": wl.name, "steps": steps, "ms_per_step": round(1e3 * elapsed / steps, 4),
           "video_tokens_per_s": round(wl.chunk * steps / elapsed, 1), "kernels_ms": kernels,
           "attention_TFLOPs": round(att_tf, 2), "attention_mfma_frac": round(att_tf / PEAK_BF16_TFLOPS, 4),
           "query": query_bench(wl, kv, steps, warmup)}
    kv.close()
    return res


def query_bench(wl, kv, steps: int, warmup: int, n_q: int = 64) -> dict:
    """Query-time attention: n_q text tokens over every layer's compacted cache
    (and their own earlier tokens).  Algorithmic work 4 d per visible (row,
    key, head) triple; bytes = the compacted K/V read once + Q and O.  `ms` is
    the mean of back-to-back calls (wall clock over the synchronised run, as
    the headline steps); `ms_with_events` the mean of the library's events
    around each call's launches."""
    import torch

    from paper_2601_14724_amd import hermes as H
    from paper_2601_14724_amd import streaming, workloads as wk
    qw = wk.scaled(wl, query_len=n_q)
    qs = [wk.gen_query(qw, l) for l in range(wl.n_layers)]
    dev = kv.device
    qt = {k: streaming.bf16_tensor(np.stack([q[k] for q in qs]), dev) for k in ("q", "k", "v")}
    o = torch.empty_like(qt["q"])
    lens = [kv.length(l) for l in range(wl.n_layers)]
    for _ in range(warmup):
        kv.query(qt["q"], qt["k"], qt["v"], out=o)
    torch.cuda.synchronize()
    # the library's events around each call's launches
    kv.profile(True)
    kv.profile_read(H.K_QUERY)
    for _ in range(steps):
        kv.query(qt["q"], qt["k"], qt["v"], out=o)
    ms_ev, cnt = kv.profile_read(H.K_QUERY)
    kv.profile(False)
    ms_ev /= max(cnt, 1)
    # queries back to back with no events between them, as the headline
    # steps (each event on the stream idles the GPU for a few microseconds);
    # enough calls that the clock ramp after the synchronisation is noise
    n_rep = max(steps, 500)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n_rep):
        kv.query(qt["q"], qt["k"], qt["v"], out=o)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / n_rep
    pairs = wl.n_q_heads * sum(n_q * T + n_q * (n_q + 1) // 2 for T in lens)
    flops = 4.0 * wl.head_dim * pairs
    row = wl.n_kv_heads * wl.head_dim * 2
    nbytes = sum(lens) * 2 * row + wl.n_layers * n_q * (2 * wl.n_q_heads * wl.head_dim * 2 + 2 * row)
    tf = flops / (ms * 1e-3) / 1e12
    gb = nbytes / (ms * 1e-3) / 1e9
    return {"n_q": n_q, "cache_tokens": sum(lens), "ms": round(ms, 4), "ms_with_events": round(ms_ev, 4),
            "TFLOPs": round(tf, 2), "mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4),
            "GBps": round(gb, 1), "hbm_frac": round(gb / PEAK_HBM_GBS, 4)}


def extension_bench(wl, caches, t, steps: int, warmup: int, prompt_rows: int = 64) -> dict:
    """The adjacent rows on the same workload: (a) summary tokens in the deep
    layers plus eager RoPE re-indexing at every compression, (b) W from a
    guidance prompt of `prompt_rows` tokens per non-shallow layer instead of
    the chunk, (c) eager 3D M-RoPE re-indexing.  Reports step time and
    per-kernel averages."""
    import torch

    from paper_2601_14724_amd import hermes as H
    from paper_2601_14724_amd import streaming, workloads as wk
    out = {}
    dev = t["q"].device

    def timed(kv, step):
        # step time without events on the stream, then a second pass with the
        # library's per-launch events for the breakdown
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        kv.profile(True)
        for kid in range(len(H.KERNEL_NAMES)):
            kv.profile_read(kid)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        ks = {}
        for kid, name in enumerate(H.KERNEL_NAMES):
            ms, cnt = kv.profile_read(kid)
            if cnt:   # per step: a group may hold several launches
                ks[name] = round(ms / steps, 4)
        kv.profile(False)
        return dt, ks

    o = torch.empty_like(t["q"])
    kv = streaming.make_cache(wl, device=dev, caches=caches, summary_mode=1,
                              reindex_mode=H.REINDEX_EAGER, rope_offset=14)

    def step_a():
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=o)
        kv.compress()
    dt, ks = timed(kv, step_a)
    row = wl.n_kv_heads * wl.head_dim * 2
    kept = sum(b + 1 if i >= wl.n_layers - int(np.floor(0.3 * wl.n_layers + 0.5)) else b
               for i, b in enumerate(wl.budgets))
    g = kept * (4.0 * row + 16.0) / (ks["gather"] * 1e-3) / 1e9 if "gather" in ks else None
    out["summary_eager_reindex"] = {"ms_per_step": round(dt * 1e3, 4), "kernels_ms": ks,
                                    "gather_rotate_GBps": round(g, 1) if g else None}
    kv.close()
    del kv

    kv = streaming.make_cache(wl, device=dev, caches=caches, scoring_mode=H.SCORE_GUIDANCE)
    pr = [wk.gen_prompt(wl, l, prompt_rows) for l in range(wl.n_layers)]
    pt = {k: streaming.bf16_tensor(np.stack([p[k] for p in pr]), dev) for k in ("q", "k", "v")}

    def step_b():
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=o)
        kv.guidance(pt["q"], pt["k"], pt["v"])
        kv.compress()
    dt, ks = timed(kv, step_b)
    out["guidance_prompt"] = {"ms_per_step": round(dt * 1e3, 4), "prompt_rows": prompt_rows,
                              "kernels_ms": ks}
    kv.close()
    del kv

    # (c) 3D M-RoPE: frames of 14 x 14 tokens (t step 2, text prefix 14),
    # every axis left-compacted and every key turned at every compression
    n0 = wl.init_len
    s = np.arange(n0 + wl.chunk)
    fr, r = s // 196, s % 196
    grid = np.stack([14 + 2 * fr, 14 + r // 14, 14 + r % 14]).astype(np.int32)   # [3][n]
    caches3 = [dict(c, thw=grid[:, :n0]) for c in caches]
    kv = streaming.make_cache(wl, device=dev, caches=caches3, reindex_mode=H.REINDEX_EAGER,
                              rope_offset=14, rope_axes=3)
    thw = torch.from_numpy(np.ascontiguousarray(grid[:, n0:])).to(dev)

    def step_c():
        kv.rewind()
        kv.append(t["q"], t["k"], t["v"], t["pos"], out=o, rope_thw=thw)
        kv.compress()
    dt, ks = timed(kv, step_c)
    out["mrope_eager_reindex"] = {"ms_per_step": round(dt * 1e3, 4), "kernels_ms": ks}
    kv.close()
    return out


def _mass_layer_fraction(wl) -> float:
    """Fraction of layers whose attention mass the step computes (the
    non-shallow ones under the 10/60/30 partition)."""
    n_sh = int(np.floor(0.1 * wl.n_layers + 0.5))
    return (wl.n_layers - n_sh) / wl.n_layers


if __name__ == "__main__":
    sys.exit(main())
