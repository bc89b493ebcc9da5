"""Benchmark of the DAF per-layer prefill attention on one MI355X.

One step is one pass of the whole hot path over one synthetic layer already
resident in HBM: the important-row gather of the hidden states, then
daf_layer_attn (hybrid KV write-back, stage 2 with its split merge, stage 1;
both stages write their rows into the hidden states in their epilogues). At
least W untimed warmup steps (and at least --warmup-ms of GPU time, so that the
shader clock has reached its level under sustained load), then exactly K timed
steps between device synchronisations. Several copies of the inputs are
used in rotation; together they touch far more than the 256 MB Infinity Cache
(MALL), so consecutive steps do not find their data there.

A second timed loop calls the stages one by one with HIP events around each
call (on the stream the kernels run on) for per-stage times, TFLOP/s, TB/s and
the roofline fraction of the dominant kernel (stage 1). Before each timed call
a 512 MiB scratch buffer is read and written, which evicts the MALL, and a GPU
spin follows so that the events and the call are queued before the GPU reaches
them. HBM traffic and kernel-trace averages come from the committed rocprofv3
summaries when they were taken on the current attention sources (their SHA-256
is recorded there), else they are null. The CPU oracle is timed on the host on
bounded samples of every workload (``cpu_baseline``).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import daf_inputs as di  # noqa: E402

METRIC = "DAF per-layer attention µs at L_d=32k,r=0.15; stage TFLOP/s + HBM TB/s vs peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attn_qwen7b_32k_pmc.md")
TRACE_SUMMARY = os.path.join(ROOT, "profiles", "attn_layer_qwen7b_32k_kernel_trace.md")
EVICT_MIB = 512  # scratch streamed through before each timed stage call (MALL is 256 MB)
# What determines a standalone stage-1 or stage-2 launch: the kernels and their
# grids, the launch structures, the compile flags, and the host functions that
# build the work tables, plan the key splits and launch the merge. A profile
# record taken on other versions of these is not used.
ATTN_SOURCES = [os.path.join(ROOT, "paper_2607_21599_amd", "csrc", f)
                for f in ("attn_bf16.hip", "attn.hip", "daf_internal.h")] + [
    os.path.join(ROOT, "paper_2607_21599_amd", "build.py")]
ATTN_HOST = os.path.join(ROOT, "paper_2607_21599_amd", "csrc", "api.hip")
ATTN_HOST_FUNCTIONS = ("AttnEntry self_entry(", "int entry_groups(", "daf_status_t run_entries(",
                       "void add_self_entries(", "bool packed_qdoc(", "int qdoc_blocks(",
                       "std::vector<Split> plan_splits(", "WsLayout ws_layout(", "AttnEntry qdoc_entry(",
                       "daf_status_t qdoc_entries(", "daf_status_t run_merge(")


def _function_text(src: str, head: str) -> str:
    """The text of the function that starts with `head` up to its closing
    brace at the start of a line."""
    i = src.find(head)
    if i < 0:
        return ""
    j = src.find("\n}\n", i)
    return src[i:j + 3]


def attn_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    with open(ATTN_HOST) as fh:
        src = fh.read()
    for head in ATTN_HOST_FUNCTIONS:
        h.update(_function_text(src, head).encode())
    return h.hexdigest()


def profile_record(path: str, tag: str, workload: str) -> dict:
    """The `tag:` line of a committed profile summary as a dict, or {} if the
    summary is absent, for another workload, or was taken on other attention
    sources."""
    try:
        with open(path) as fh:
            lines = fh.read().splitlines()
    except OSError:
        return {}
    fields = {}
    for ln in lines:
        if ln.startswith(tag + ":"):
            for kv in ln.split(":", 1)[1].split():
                k, _, v = kv.partition("=")
                fields[k] = v
    if fields.get("workload") != workload or fields.get("sources_sha256") != attn_source_hash():
        return {}
    return fields


def record_number(rec: dict, key: str):
    try:
        return float(rec[key])
    except (KeyError, ValueError):
        return None


def work(shapes) -> dict:
    """Algorithmic FLOP and HBM bytes per stage (causal masks counted exactly,
    every operand read once, every output written once)."""
    f1 = f2 = b1 = b2 = bkv = bhid = bgat = 0
    for s in shapes:
        eb = 2 if s.dtype == di.BF16 else 4
        qrow, krow = s.hq * s.d * eb, s.hkv * s.d * eb
        f1 += 4 * s.d * s.hq * s.n * (s.n + 1) // 2
        f2 += 4 * s.d * s.hq * (s.L_q * s.L_d + s.L_q * (s.L_q + 1) // 2)
        b1 += s.n * (2 * qrow + 2 * krow)
        b2 += s.T * 2 * krow + 2 * s.L_q * qrow
        bkv += 2 * (s.n + s.L_q) * 2 * krow
        bhid += 2 * (s.n + s.L_q) * qrow
        bgat += 2 * s.n * qrow
    return dict(stage1_flop=f1, stage2_flop=f2, stage1_bytes=b1, stage2_bytes=b2, fuse_kv_bytes=bkv,
                fuse_hidden_bytes=bhid, gather_bytes=bgat)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_layer_us(batch, stride1: int, stride2: int, requests=None):
    """Oracle time of one layer in µs: the full hybrid-cache build and fusion,
    and the attention of every stride1-th stage-1 row and every stride2-th
    stage-2 row of the chosen requests, each attention time scaled by total
    over sampled rows. Returns (µs, stage-1 rows, stage-2 rows, threads)."""
    import oracle
    orc = oracle.get()
    w = di.raw_to_f32
    t_total = 0.0
    rows_done = [0, 0]
    for b, s in enumerate(batch.shapes):
        if requests is not None and b not in requests:
            continue
        r = batch.request(b)
        sc = oracle.default_scale(s.d)
        rows1 = np.arange(0, s.n, stride1)
        rows2 = np.arange(0, s.L_q, stride2)
        q1, k1, v1 = w(r["q_imp"]), w(r["k_imp"]), w(r["v_imp"])
        t0 = time.perf_counter()
        kh, vh = orc.hybrid_kv(r["k_cache"], r["v_cache"], r["idx"], r["k_imp"], r["v_imp"], r["k_q"],
                               r["v_q"], s.L_d)
        t_hyb = time.perf_counter() - t0
        t0 = time.perf_counter()
        orc.stage1(q1, k1, v1, r["idx"], sc, rows1)
        t_s1 = time.perf_counter() - t0
        kf, vf, qq = w(kh), w(vh), w(r["q_q"])
        t0 = time.perf_counter()
        orc.stage2(qq, kf, vf, s.L_d, sc, rows2)
        t_s2 = time.perf_counter() - t0
        t0 = time.perf_counter()
        orc.fuse_hidden(r["hidden"], r["idx"], r["q_imp"], r["q_q"], s.L_d)
        t_fuse = time.perf_counter() - t0
        t_total += t_hyb + t_fuse + t_s1 * s.n / max(1, len(rows1)) + t_s2 * s.L_q / max(1, len(rows2))
        rows_done[0] += len(rows1)
        rows_done[1] += len(rows2)
    return t_total * 1e6, rows_done[0], rows_done[1], orc.threads


def cpu_baseline(batch, stride1: int, stride2: int) -> dict:
    """The oracle on a row sample of the bench workload, scaled to the layer."""
    us, n1, n2, threads = oracle_layer_us(batch, stride1, stride2)
    return dict(value=us, unit="us", cores=threads, kind="oracle", cpu=cpu_model(),
                sample=(f"stage-1 rows 0::{stride1} ({n1} rows) and stage-2 rows 0::{stride2} "
                        f"({n2} rows) of every request, full hybrid-cache build and fusion; "
                        "attention times scaled by total/sampled rows"))


# The other workloads the oracle is timed on: (workload, stage-1 stride,
# stage-2 stride, sampled requests or None for all). The batched workload is
# timed on three of its eight requests, generated one at a time, and scaled by
# the attention FLOP of all eight over those three.
ORACLE_SAMPLES = [("tiny_f32_1k", 1, 1, None), ("qwen7b_6k", 2, 1, None), ("qwen7b_16k_r05", 4, 2, None),
                  ("qwen7b_16k_r15", 8, 2, None), ("qwen7b_16k_r30", 16, 4, None),
                  ("qwen7b_batch8", 16, 4, (0, 3, 7))]


def cpu_baseline_configs() -> list:
    out = []
    for name, st1, st2, reqs in ORACLE_SAMPLES:
        shapes = di.workload(name)
        if reqs is None:
            us, n1, n2, _ = oracle_layer_us(di.make_batch(shapes), st1, st2)
            sample = f"stage-1 rows 0::{st1} ({n1}), stage-2 rows 0::{st2} ({n2}), scaled by total/sampled rows"
        else:
            us, n1, n2 = 0.0, 0, 0
            for b in reqs:
                u, a, c, _ = oracle_layer_us(di.make_batch([shapes[b]]), st1, st2)
                us, n1, n2 = us + u, n1 + a, n2 + c
            wall = work(shapes)
            part = work([shapes[b] for b in reqs])
            scale = (wall["stage1_flop"] + wall["stage2_flop"]) / (part["stage1_flop"] + part["stage2_flop"])
            us *= scale
            sample = (f"requests {', '.join(str(b) for b in reqs)} of {len(shapes)}: stage-1 rows 0::{st1} ({n1}), "
                      f"stage-2 rows 0::{st2} ({n2}), scaled by total/sampled rows, then by the attention FLOP "
                      f"of all requests over the sampled ones (x{scale:.2f})")
        out.append({"workload": name, "us": us, "sample": sample})
        print(f"[bench] oracle {name}: {us / 1e6:.2f} s per layer (estimated from a sample)", file=sys.stderr,
              flush=True)
    return out


def decoder_layer_section(s0, batch, spin_cycles: int, selection_us, evict) -> dict:
    """One prefill decoder layer with Qwen2.5-7B-shaped synthetic weights:
    DAF (only the important and question rows, DAF attention on the hybrid
    cache) against full recomputation (every row, causal attention), each
    call timed alone behind a MALL eviction (`evict`) and a GPU spin, and a
    28-layer TTFT model from them."""
    import torch

    import paper_2607_21599_amd as daf
    m = di.QWEN7B
    H, I, QW, KW = m.hidden, m.inter, m.hq * m.d, m.hkv * m.d
    g = torch.Generator(device="cuda")
    g.manual_seed(20240607)

    def randn(*shape, std=1.0, mean=0.0):
        return (torch.randn(*shape, generator=g, device="cuda") * std + mean).to(torch.bfloat16)

    wt = dict(w_in=randn(H, std=0.1, mean=1.0), wq=randn(QW, H, std=H ** -0.5), bq=randn(QW, std=0.1),
              wk=randn(KW, H, std=H ** -0.5), bk=randn(KW, std=0.1), wv=randn(KW, H, std=H ** -0.5),
              bv=randn(KW, std=0.1), wo=randn(H, QW, std=QW ** -0.5), w_post=randn(H, std=0.1, mean=1.0),
              wgu=randn(2 * I, H, std=H ** -0.5), wd=randn(H, I, std=I ** -0.5))
    lw = daf.LayerWeights.from_tensors(wt, H, I, m.eps, m.theta)
    cfg = daf.AttnCfg(m.hq, m.hkv, m.d, daf.DAF_BF16)
    L_d, L_q, n, T = s0.L_d, s0.L_q, s0.n, s0.T
    idx = batch.request(0)["idx"].astype(np.int32)
    rows_act = np.concatenate([idx, np.arange(L_d, T, dtype=np.int32)])
    x_all = randn(T, H)
    modes = {
        "daf": dict(mode=daf.DAF_LAYER_DAF, b=daf.Batch.single(L_d, L_q, n), x0=x_all[torch.from_numpy(rows_act).
                    long().cuda()].contiguous(), pos=torch.from_numpy(rows_act).cuda(),
                    idx=torch.from_numpy(idx).cuda(), kc=randn(T, m.hkv, m.d, std=0.5),
                    vc=randn(T, m.hkv, m.d, std=0.5), reps=5),
        "full": dict(mode=daf.DAF_LAYER_FULL, b=daf.Batch.single(L_d, L_q, 0), x0=x_all,
                     pos=torch.arange(T, dtype=torch.int32, device="cuda"), idx=None, kc=None, vc=None, reps=3),
    }
    res = {}
    for name, c in modes.items():
        ws_bytes = daf.daf_decoder_layer_workspace_size(cfg, lw, c["b"], c["mode"])
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        x = c["x0"].clone()

        def run():
            daf.daf_decoder_layer(cfg, lw, c["b"], c["mode"], c["idx"], c["pos"], x, c["kc"], c["vc"], ws,
                                  ws_bytes)
        run()
        torch.cuda.synchronize()
        t = []
        for _ in range(c["reps"]):
            x.copy_(c["x0"])
            evict()
            torch.cuda._sleep(spin_cycles)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            run()
            b.record()
            torch.cuda.synchronize()
            t.append(a.elapsed_time(b) * 1e3)
        rows = c["x0"].shape[0]
        gemm_flop = 2 * rows * H * (QW + 2 * KW + QW + 2 * I + I)
        res[name] = dict(us=float(np.mean(t)), rows=int(rows), gemm_flop=int(gemm_flop))
        del ws
    n_full_layers, n_layers = 4, 28  # layers 1-4 recomputed in full for the selection signal (layers 2-4)
    sel = selection_us or 0.0
    ttft_daf = n_full_layers * res["full"]["us"] + sel + (n_layers - n_full_layers) * res["daf"]["us"]
    ttft_full = n_layers * res["full"]["us"]
    return {
        "model": "Qwen2.5-7B-shaped layer, synthetic bf16 weights (hidden 3584, 28/4 heads, MLP 18944)",
        "daf_layer_us": res["daf"]["us"], "daf_rows": res["daf"]["rows"],
        "full_layer_us": res["full"]["us"], "full_rows": res["full"]["rows"],
        "layer_speedup": res["full"]["us"] / res["daf"]["us"],
        "daf_gemm_flop": res["daf"]["gemm_flop"], "full_gemm_flop": res["full"]["gemm_flop"],
        "ttft_model_ms": {"daf": ttft_daf / 1e3, "full_recompute": ttft_full / 1e3,
                          "speedup": ttft_full / ttft_daf,
                          "recipe": f"{n_full_layers} full layers (selection signal) + selection + "
                                    f"{n_layers - n_full_layers} DAF layers, vs {n_layers} full layers; "
                                    "no embedding, LM head or KV loading"},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--warmup-ms", type=float, default=100.0,
                    help="keep running untimed warmup steps until at least this much GPU time has passed "
                         "(the shader clock ramps up over the first ~10 ms of sustained load)")
    ap.add_argument("--workload", default="qwen7b_32k")
    ap.add_argument("--copies", type=int, default=3, help="input copies used in rotation")
    ap.add_argument("--cpu-stride1", type=int, default=4)
    ap.add_argument("--cpu-stride2", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layer", action="store_true",
                    help="skip the decoder-layer section (projections, norms and MLP around the attention)")
    ap.add_argument("--no-patterns", action="store_true",
                    help="skip the selection call and the comparison patterns (CacheBlend-style and full "
                         "recomputation attention)")
    ap.add_argument("--no-lq32", action="store_true", help="skip stage 2 at L_q = 32")
    ap.add_argument("--no-oracle-configs", action="store_true",
                    help="time the CPU oracle on the bench workload only")
    ap.add_argument("--evict", choices=("read", "write"), default="read",
                    help="how the 512 MiB scratch evicts the MALL before each timed call: read it (the MALL "
                         "then holds clean lines), or read and write it (dirty lines, whose write-back then "
                         "competes with the timed call's reads)")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="before timing, run one plain device copy of this many MiB (a known-size "
                         "kernel that calibrates HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on one GPU only (the DAF layer attention is measured on a "
              "single MI355X); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import LayerBuffers

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    daf.lib()
    shapes = di.workload(args.workload)
    batch = di.make_batch(shapes)
    s0 = shapes[0]
    print(f"[bench] {args.workload}: generated inputs", file=sys.stderr, flush=True)
    bufs = [LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s0.hq, s0.hkv, s0.d)
            for _ in range(max(1, args.copies))]
    tdt = bufs[0]["hidden"].dtype
    gath = [torch.empty((int(batch.cu_imp[-1]), s0.hq * s0.d), dtype=tdt, device="cuda") for _ in bufs]

    def step(i):
        j = i % len(bufs)
        bufs[j].gather_hidden(gath[j])
        bufs[j].layer()

    if args.calib_copy_mb > 0:
        n = args.calib_copy_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # Untimed warmup: at least W steps and at least --warmup-ms of GPU time.
    # Steps timed right after a short warmup run ~20% slower while the clocks
    # ramp up under the sustained load.
    w0 = torch.cuda.Event(enable_timing=True)
    w1 = torch.cuda.Event(enable_timing=True)
    warm_steps, warm_ms = 0, 0.0
    w0.record()
    while warm_steps < args.warmup or warm_ms < args.warmup_ms:
        for _ in range(max(1, args.warmup - warm_steps) if warm_steps < args.warmup else 10):
            step(warm_steps)
            warm_steps += 1
        w1.record()
        torch.cuda.synchronize()
        warm_ms = w0.elapsed_time(w1)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(args.steps):
        step(warm_steps + i)
    t1.record()
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps
    wk0 = work(shapes)
    step_touch = (wk0["gather_bytes"] + wk0["fuse_kv_bytes"] + wk0["stage1_bytes"] + wk0["stage2_bytes"]
                  + wk0["fuse_hidden_bytes"])
    print(f"[bench] timed {args.steps} steps: {ms_per_step * 1e3:.1f} us/step", file=sys.stderr, flush=True)

    # Per-stage times: events around each stage call on the launch stream.
    # Before each timed call a 512 MiB scratch buffer is read and written
    # (evicting the 256 MB MALL, so the call reads its inputs from HBM), then a
    # GPU spin is queued: a host call takes longer than the shorter kernels, and
    # the spin lets the events and the call be enqueued before the GPU reaches
    # them, so the event pair measures the call's GPU time. The calls are
    # idempotent (same inputs, same outputs).
    evict = torch.zeros(EVICT_MIB << 20, dtype=torch.uint8, device="cuda")
    evict_sum = torch.zeros(1, dtype=torch.int64, device="cuda")
    spin_cycles = 400_000  # ~0.2 ms at the MI355X shader clock, longer than a host call

    def evict_mall():
        if args.evict == "write":
            evict.add_(1)
        else:
            torch.sum(evict.view(torch.int64), dim=0, keepdim=True, out=evict_sum)

    def timed_calls(fn, n):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i in range(n):
            evict_mall()
            torch.cuda._sleep(spin_cycles)
            ev[i][0].record()
            fn(i)
            ev[i][1].record()
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev]) * 1e3

    # the floor of this timing: an event pair around nothing
    event_floor = float(np.mean(timed_calls(lambda i: None, args.steps)))
    # the same step, one call at a time, each after a MALL eviction
    t_cold = timed_calls(step, args.steps)
    print(f"[bench] step after MALL eviction: {np.mean(t_cold):.1f} us", file=sys.stderr, flush=True)

    names = ["gather", "fuse_kv", "stage1", "stage2", "fuse_hidden"]
    calls = {
        "gather": lambda j: bufs[j].gather_hidden(gath[j]),
        "fuse_kv": lambda j: bufs[j].fuse_kv(),
        "stage1": lambda j: bufs[j].stage1(),
        "stage2": lambda j: bufs[j].stage2(),
        "fuse_hidden": lambda j: bufs[j].fuse_hidden(),
    }
    stage_us, stage_pct = {}, {}
    for n in names:
        calls[n](0)
        torch.cuda.synchronize()
        t_us = timed_calls(lambda i: calls[n](i % len(bufs)), args.steps)
        stage_us[n] = float(np.mean(t_us))
        stage_pct[n] = [float(x) for x in np.percentile(t_us, [10, 50, 90])]
    # Reference for the row kernels: a plain contiguous device copy moving the
    # same bytes (read + write) as each of them, timed the same way.
    wk = work(shapes)
    copy_ref = {}
    for name, nbytes in (("gather", wk["gather_bytes"]), ("fuse_kv", wk["fuse_kv_bytes"]),
                         ("fuse_hidden", wk["fuse_hidden_bytes"])):
        half = (nbytes // 2 + 15) // 16 * 16
        src = torch.empty(half, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        t_copy = float(np.mean(timed_calls(lambda i: dst.copy_(src), args.steps)))
        copy_ref[name] = {"bytes": 2 * half, "us": t_copy, "GBps": 2 * half / (t_copy * 1e-6) / 1e9}
        del src, dst
    peak_mma = PEAK_BF16_TFLOPS if s0.dtype == di.BF16 else PEAK_F32_TFLOPS

    def tflops(f, us):
        return f / (us * 1e-6) / 1e12

    def gbs(by, us):
        return by / (us * 1e-6) / 1e9

    stages = {
        "gather": dict(us=stage_us["gather"], GBps=gbs(wk["gather_bytes"], stage_us["gather"]),
                       bytes=wk["gather_bytes"]),
        "fuse_kv": dict(us=stage_us["fuse_kv"], GBps=gbs(wk["fuse_kv_bytes"], stage_us["fuse_kv"]),
                        bytes=wk["fuse_kv_bytes"]),
        "stage1_imp_self_attn": dict(us=stage_us["stage1"], TFLOPs=tflops(wk["stage1_flop"], stage_us["stage1"]),
                                     GBps=gbs(wk["stage1_bytes"], stage_us["stage1"]), flop=wk["stage1_flop"],
                                     bytes=wk["stage1_bytes"]),
        "stage2_qdoc_attn": dict(us=stage_us["stage2"], TFLOPs=tflops(wk["stage2_flop"], stage_us["stage2"]),
                                 GBps=gbs(wk["stage2_bytes"], stage_us["stage2"]), flop=wk["stage2_flop"],
                                 bytes=wk["stage2_bytes"]),
        "fuse_hidden": dict(us=stage_us["fuse_hidden"],
                            GBps=gbs(wk["fuse_hidden_bytes"], stage_us["fuse_hidden"]),
                            bytes=wk["fuse_hidden_bytes"]),
    }
    for k, n in zip(stages, names):
        stages[k]["us_p10_p50_p90"] = stage_pct[n]
    for k in ("gather", "fuse_kv", "fuse_hidden"):
        stages[k]["hbm_frac"] = stages[k]["GBps"] / PEAK_HBM_GBS
        stages[k]["plain_copy_same_bytes"] = copy_ref[k]
    for k in ("stage1_imp_self_attn", "stage2_qdoc_attn"):
        st = stages[k]
        st["mfma_frac"] = st["TFLOPs"] / peak_mma
        st["hbm_frac"] = st["GBps"] / PEAK_HBM_GBS
        # roofline time of the bound that applies, over the measured time
        t_floor = max(st["flop"] / (peak_mma * 1e12), st["bytes"] / (PEAK_HBM_GBS * 1e9))
        st["roofline_frac"] = t_floor / (st["us"] * 1e-6)
    # Kernel-trace averages and counter-measured HBM bytes of the standalone
    # launches, from the committed rocprofv3 summaries of this workload (null
    # when those were taken on other attention sources).
    trace = profile_record(TRACE_SUMMARY, "trace-record", args.workload)
    traffic = profile_record(TRAFFIC_SUMMARY, "traffic-record", args.workload)
    s1 = stages["stage1_imp_self_attn"]
    s1_trace_us = record_number(trace, "stage1_avg_us")
    s1_traffic = record_number(traffic, "stage1_hbm_bytes_per_launch")
    roofline = dict(bound="mfma", kernel="attn_bf16_kernel<128,0> (stage 1, daf_imp_self_attn)",
                    achieved=s1["TFLOPs"], peak=peak_mma, unit="TFLOP/s", frac=s1["TFLOPs"] / peak_mma,
                    traffic=int(s1_traffic) if s1_traffic else None,
                    traffic_unit="bytes per launch (HBM, counters)",
                    flop_per_launch=wk["stage1_flop"], launch_us=s1["us"], launch_us_rocprof=s1_trace_us,
                    frac_rocprof=(tflops(wk["stage1_flop"], s1_trace_us) / peak_mma) if s1_trace_us else None,
                    frac_note="frac: HIP-event time of the standalone call in this run; frac_rocprof: the "
                              "kernel's average duration in the committed kernel trace")
    for k, rk in (("gather", "gather"), ("fuse_kv", "fuse_kv"), ("fuse_hidden", "fuse_hidden")):
        t_k = record_number(trace, rk + "_avg_us")
        b_k = record_number(traffic, rk + "_hbm_bytes_per_launch")
        stages[k]["kernel_us_rocprof"] = t_k
        stages[k]["hbm_frac_rocprof"] = gbs(stages[k]["bytes"], t_k) / PEAK_HBM_GBS if t_k else None
        stages[k]["hbm_bytes_counted"] = int(b_k) if b_k else None
    s1["kernel_us_rocprof"] = s1_trace_us
    s1["hbm_bytes_counted"] = int(s1_traffic) if s1_traffic else None
    s2 = stages["stage2_qdoc_attn"]
    s2_trace = [record_number(trace, k) for k in ("stage2_avg_us", "merge_avg_us")]
    s2_bytes = [record_number(traffic, k) for k in ("stage2_hbm_bytes_per_launch", "merge_hbm_bytes_per_launch")]
    s2["kernel_us_rocprof"] = sum(s2_trace) if None not in s2_trace else None
    s2["hbm_bytes_counted"] = int(sum(s2_bytes)) if None not in s2_bytes else None
    s2["counted_over_algorithmic"] = (sum(s2_bytes) / s2["bytes"]) if None not in s2_bytes else None
    s2["hbm_bytes_counted_split"] = ({"attention": int(s2_bytes[0]), "merge": int(s2_bytes[1])}
                                     if None not in s2_bytes else None)

    # Stage 2 in its bandwidth-bound regime: the same layer with a 32-token
    # question (7 query rows per cached K/V byte, below the MFMA/HBM ridge),
    # timed alone like the stage calls above (MALL evicted before each call).
    stage2_lq32 = None
    if not args.no_lq32 and args.workload == "qwen7b_32k":
        print("[bench] stage 2 at L_q = 32", file=sys.stderr, flush=True)
        shp32 = di.workload("qwen7b_32k_lq32")
        b32 = di.make_batch(shp32)
        bufs32 = [LayerBuffers(b32.arrays, b32.cu_doc, b32.cu_q, b32.cu_imp, s0.hq, s0.hkv, s0.d)
                  for _ in range(max(1, args.copies))]
        for bb in bufs32:
            bb.fuse_kv()
        bufs32[0].stage2()
        torch.cuda.synchronize()
        us32 = float(np.mean(timed_calls(lambda i: bufs32[i % len(bufs32)].stage2(), args.steps)))
        wk32 = work(shp32)
        t_hbm = wk32["stage2_bytes"] / (PEAK_HBM_GBS * 1e9)
        t_mma = wk32["stage2_flop"] / (peak_mma * 1e12)
        tr32 = [record_number(trace, k) for k in ("stage2_lq32_avg_us", "merge_lq32_avg_us")]
        by32 = [record_number(traffic, k) for k in ("stage2_lq32_hbm_bytes_per_launch",
                                                     "merge_lq32_hbm_bytes_per_launch")]
        stage2_lq32 = {"workload": "qwen7b_32k_lq32", "L_q": shp32[0].L_q, "us": us32,
                       "bytes": wk32["stage2_bytes"], "GBps": gbs(wk32["stage2_bytes"], us32),
                       "hbm_frac": gbs(wk32["stage2_bytes"], us32) / PEAK_HBM_GBS,
                       "flop": wk32["stage2_flop"], "TFLOPs": tflops(wk32["stage2_flop"], us32),
                       "floor_us": {"hbm": t_hbm * 1e6, "mfma": t_mma * 1e6},
                       "roofline_frac": max(t_hbm, t_mma) / (us32 * 1e-6),
                       "kernel_us_rocprof": sum(tr32) if None not in tr32 else None,
                       "hbm_frac_rocprof": (gbs(wk32["stage2_bytes"], sum(tr32)) / PEAK_HBM_GBS
                                            if None not in tr32 else None),
                       "hbm_bytes_counted": int(sum(by32)) if None not in by32 else None,
                       "counted_over_algorithmic": (sum(by32) / wk32["stage2_bytes"]) if None not in by32 else None}
        del bufs32, b32

    selection = None
    if not args.no_patterns:
        # The step before the path: choosing the important tokens from the KV
        # deviation over three selection layers (same eviction + spin + event timing).
        print("[bench] important-token selection", file=sys.stderr, flush=True)
        import paper_2607_21599_amd as daf_mod
        from paper_2607_21599_amd.tensors import to_device
        n_sel_layers = 3
        pairs = [di.make_selection_inputs(s, n_sel_layers) for s in shapes]
        fresh = [to_device(np.ascontiguousarray(np.concatenate([p[0][l] for p in pairs])))
                 for l in range(n_sel_layers)]
        cached = [to_device(np.ascontiguousarray(np.concatenate([p[1][l] for p in pairs])))
                  for l in range(n_sel_layers)]
        del pairs
        n_doc = int(batch.cu_doc[-1])
        sel_scores = torch.empty(n_doc, dtype=torch.float32, device="cuda")
        sel_idx = torch.empty(int(batch.cu_imp[-1]), dtype=torch.int32, device="cuda")
        b0 = bufs[0]

        def run_sel():
            daf_mod.daf_select_important(b0.cfg, b0.batch, fresh, cached, sel_scores, sel_idx)

        run_sel()
        torch.cuda.synchronize()
        sel_us = float(np.mean(timed_calls(lambda i: run_sel(), 10)))
        eb = 2 if s0.dtype == di.BF16 else 4
        sel_bytes = 2 * n_sel_layers * n_doc * s0.hkv * s0.d * eb + 4 * n_doc + 4 * int(batch.cu_imp[-1])
        selection = {"us": sel_us, "layers": n_sel_layers, "bytes": sel_bytes, "GBps": gbs(sel_bytes, sel_us),
                     "hbm_frac": gbs(sel_bytes, sel_us) / PEAK_HBM_GBS}
        del fresh, cached

    comparison = None
    if not args.no_patterns and len(shapes) == 1:
        # The schemes the Complexity Analysis compares DAF with, as attention on
        # the same GPU: the CacheBlend pattern (important and question rows over
        # the whole hybrid cache, causal by position) and full recomputation
        # (every token over its prefix). Same eviction + spin + event timing.
        print("[bench] comparison patterns", file=sys.stderr, flush=True)
        pb = bufs[0]
        pb.fuse_kv()
        pb.prepare_patterns(di.make_full_queries(s0))
        pat_us = {}
        for n, fn in (("cacheblend", pb.cacheblend), ("full_recompute", pb.full_recompute)):
            fn()
            torch.cuda.synchronize()
            pat_us[n] = float(np.mean(timed_calls(lambda i: fn(), 5)))
        idx = batch.request(0)["idx"].astype(np.int64)
        pos = np.concatenate([idx, s0.L_d + np.arange(s0.L_q)])
        f_cb = 4 * s0.d * s0.hq * int((pos + 1).sum())
        f_full = 4 * s0.d * s0.hq * s0.T * (s0.T + 1) // 2
        daf_us = stage_us["stage1"] + stage_us["stage2"]
        comparison = {
            "daf_attention_us": daf_us, "daf_attention_flop": wk["stage1_flop"] + wk["stage2_flop"],
            "cacheblend_us": pat_us["cacheblend"], "cacheblend_flop": f_cb,
            "cacheblend_TFLOPs": tflops(f_cb, pat_us["cacheblend"]),
            "full_recompute_us": pat_us["full_recompute"], "full_recompute_flop": f_full,
            "full_recompute_TFLOPs": tflops(f_full, pat_us["full_recompute"]),
            "speedup_vs_cacheblend": pat_us["cacheblend"] / daf_us,
            "speedup_vs_full_recompute": pat_us["full_recompute"] / daf_us,
            "note": "attention only (stage 1 + stage 2 vs the same kernels with position masks); "
                    "the paper's Table 1 speedups are end-to-end TTFT on an A100",
        }

    layer = None
    if not args.no_layer and len(shapes) == 1 and s0.dtype == di.BF16:
        print("[bench] decoder layer: DAF vs full recomputation", file=sys.stderr, flush=True)
        layer = decoder_layer_section(s0, batch, spin_cycles, selection["us"] if selection else None, evict_mall)

    out = {
        "metric": METRIC, "value": ms_per_step * 1e3, "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "warmup_steps_run": warm_steps, "warmup_gpu_ms": round(warm_ms, 1),
        "ms_per_step": ms_per_step, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if s0.dtype == di.BF16 else "f32", "data": "synthetic",
        "config": {"workload": args.workload, "L_d": [s.L_d for s in shapes] if len(shapes) > 1 else s0.L_d,
                   "L_q": [s.L_q for s in shapes] if len(shapes) > 1 else s0.L_q,
                   "n_imp": [s.n for s in shapes] if len(shapes) > 1 else s0.n,
                   "q_heads": s0.hq, "kv_heads": s0.hkv, "head_dim": s0.d, "requests": len(shapes),
                   "step": "gather + daf_layer_attn", "input_copies": len(bufs)},
        "mall": {"value": f"{args.steps} steps back to back, {len(bufs)} input copies in rotation; one copy "
                          f"touches {step_touch / 1e6:.0f} MB per step, so consecutive steps sharing a copy are "
                          f"{(len(bufs) - 1) * step_touch / 1e6:.0f} MB of other traffic apart (MALL 256 MB)",
                 "per_call": f"{EVICT_MIB} MiB scratch {'read' if args.evict == 'read' else 'read and written'} "
                             "before each timed call (stages, step_us_mall_evicted, stage2_lq32, selection, "
                             "comparison, decoder_layer), outside the events",
                 "evict": args.evict},
        "event_floor_us": event_floor,
        "step_us_mall_evicted": float(np.mean(t_cold)),
        "layer_attn_us_sum_of_stages": sum(stage_us[n] for n in names[1:]),
        "stages": stages,
        "roofline": roofline,
    }
    if stage2_lq32 is not None:
        out["stage2_lq32"] = stage2_lq32
    if selection is not None:
        out["selection"] = selection
    if comparison is not None:
        out["comparison"] = comparison
    if layer is not None:
        out["decoder_layer"] = layer
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(batch, args.cpu_stride1, args.cpu_stride2)
        if not args.no_oracle_configs:
            out["cpu_baseline"]["other_workloads"] = cpu_baseline_configs()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
