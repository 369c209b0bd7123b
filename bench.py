"""Benchmark: one GPU's share of the pipeline-stage training step.

Workload (default): the 7B-shaped stage — 4 decoder layers, d_model 4096,
32 heads x 128, SwiGLU FFN 11008, causal sequence 4096, microbatch 1, 16
microbatches in the 1F1B Order of stage 0 of an 8-stage pipeline, bf16
compute with fp32 gradient accumulation, then one AdamW step (with the bf16
cast of the updated weights) over the whole stage bucket. A step is one pass
of all of it; inputs are resident in HBM before timing starts.

Reported: algorithmic TFLOP/s of the step (GEMMs 2MNK; causal attention
S(S+1)/2 pairs per head for each of QK^T and PV; backward = 2x forward;
attention recompute excluded), its fraction of the MI355X bf16 dense peak,
the roofline of the dominant kernel measured with HIP events, the AdamW
shard step on a 1.6e9-element shard in GB/s, and the CPU oracle timed on a
bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2516.6   # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 FLOP/clk)
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
METRIC = ("stage fwd+bwd TFLOP/s + MFMA util (7B-shaped 4-layer stage); Adam shard GB/s")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stage_flops_per_mb(cfg) -> float:
    """Algorithmic FLOP of Chunk F + Chunk B of one microbatch: projection
    GEMMs 2MNK (a MoE layer's experts counted over the 2T routed rows, the
    tiny router product excluded), causal attention S(S+1)/2 pairs per head
    for each of QK^T and PV, backward = 2x forward."""
    T, d, f, H, hd, S, b = (cfg.tokens, cfg.d_model, cfg.d_ff, cfg.n_heads, cfg.head_dim,
                            cfg.seq_len, cfg.micro_batch)
    if cfg.moe:
        ffn = 2.0 * (cfg.top_k * T) * d * (3 * cfg.d_ff_expert)
    else:
        ffn = 2.0 * T * d * (3 * f)
    dkv = cfg.kv_heads * hd  # grouped-query attention: narrower k, v projections
    gemm = 2.0 * T * d * (d + 2 * dkv + d) + ffn
    attn = 4.0 * (S * (S + 1) / 2) * hd * H * b
    return 3.0 * cfg.n_layers * (gemm + attn)


def desc_of(cfg, lc):
    return lc.desc_of_config(cfg)


STEP_STATS = {}  # tag -> median and min of the timed steps
WGRAD_TIMES = {}  # tag -> (durations in ms, FLOP) of the timed weight-gradient launches


def time_stage(torch, lc, cfg, stream, steps, warmup, tag, w_delay=None, overlap=False,
               time_wgrad=False):
    # w_delay with overlap: the split Order with each Bi and the next Bw as a pair
    """Time steps of (zero G, the Order, AdamW over the bucket) on `cfg`;
    returns (ms per step, TFLOP/s, outputs finite). With w_delay set the
    Order is 1F1B with split backwards (Bi, then Bw w_delay backwards later);
    with overlap, 1F1B with its steady-state (F, B) pairs nested and run on
    two streams. With time_wgrad, the library brackets every weight-gradient
    product launch of the timed steps with HIP events on its stream
    (lc_stage_timer_enable); the durations land in WGRAD_TIMES[tag]."""
    from paper_2606_11169_amd.runner import random_stage
    M = cfg.num_microbatches
    aux = None
    if overlap and w_delay is not None:
        order = lc.lc_order_1f1b_split_overlap(M, cfg.pp_size, cfg.pp_rank, w_delay)
        wp = min(w_delay + 1, M)
        aux = torch.cuda.Stream()
    elif overlap:
        order = lc.lc_order_1f1b_overlap(M, cfg.pp_size, cfg.pp_rank)
        wp = 0
        aux = torch.cuda.Stream()
    elif w_delay is None:
        order = lc.lc_order_1f1b(M, cfg.pp_size, cfg.pp_rank)
        wp = 0
    else:
        order = lc.lc_order_1f1b_split(M, cfg.pp_size, cfg.pp_rank, w_delay)
        wp = min(w_delay + 1, M)
    st, peak, peak_w = lc.lc_order_validate_split(order, M, M, M)
    assert st == lc.LC_OK
    wp = max(wp, peak_w)
    log(f"[bench] {cfg.name}: {M} microbatches, 1F1B(P={cfg.pp_size}, s={cfg.pp_rank})"
        f"{'' if w_delay is None else f' split, w_delay {w_delay}'}"
        f"{' with overlapped pairs on two streams' if overlap else ''}, {peak} in flight, "
        f"{peak_w} weight passes pending")
    r = random_stage(desc_of(cfg, lc), peak, seed=0, stream=stream, max_w_pending=wp)
    r.alloc_random_microbatches(M, seed=1)
    log(f"[bench] params {r.n_params}, workspace {r.ws_bytes / 2**30:.1f} GiB")

    def step():
        r.zero_grad()
        r.run_order(order, aux)
        r.adam_step(cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.weight_decay)

    for i in range(warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] {tag} warmup {i + 1}/{warmup} done")
    torch.cuda.synchronize()
    # an event before every step (and after the last) on the launch stream:
    # per-step times without any host synchronisation inside the timed region
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    cap = steps * cfg.n_layers * M * 4  # four dense weight-gradient products per layer and B
    if time_wgrad:
        lc.lc_stage_timer_enable(r.stage, cap)
    ev[0].record(stream)
    for i in range(steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    if time_wgrad:
        wms, wfl, wn = lc.lc_stage_timer_read(r.stage, cap)
        assert wn == cap == len(wms), (wn, cap)
        WGRAD_TIMES[tag] = (wms, wfl)
        lc.lc_stage_timer_enable(r.stage, 0)
    ms = ev[0].elapsed_time(ev[steps]) / steps
    per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    STEP_STATS[tag] = {"median_ms": round(per[len(per) // 2], 2), "min_ms": round(per[0], 2)}
    tflops = stage_flops_per_mb(cfg) * M / (ms * 1e-3) / 1e12
    finite = bool(torch.isfinite(r.Y[M - 1].float()).all().item())
    r.close()
    del r
    torch.cuda.empty_cache()
    return ms, tflops, finite


def time_zero(torch, lc, cfg, stream, steps, warmup, level, ranks=8):
    """One data-parallel rank's step of the stage under ZeRO-2 or ZeRO-3 on one
    GPU (rank 0 of `ranks`, collectives left out): zero the gradient shard,
    the 1F1B Order through lc_run_order_zero (each backward into a temporary
    full gradient, then its slice added into the shard; at level 3 the bf16
    weights gathered from `ranks` shards before every entry), AdamW over the
    shard. Returns (ms per step, TFLOP/s, bytes of persistent gradient +
    optimizer state on this rank, bytes of the temporary buffers)."""
    from paper_2606_11169_amd.runner import random_stage
    M = cfg.num_microbatches
    order = lc.lc_order_1f1b(M, cfg.pp_size, cfg.pp_rank)
    r = random_stage(desc_of(cfg, lc), min(cfg.pp_size - cfg.pp_rank, M), seed=0, stream=stream)
    r.alloc_random_microbatches(M, seed=1)
    n = r.n_params
    bounds = [min(n, (n * i // ranks) // 4 * 4) for i in range(ranks)] + [n]
    off, end = bounds[0], bounds[1]
    shard = torch.zeros(end - off, dtype=torch.float32, device=r.device)
    full = torch.empty(n, dtype=torch.float32, device=r.device)
    master = r.master[off:end].clone()
    m = torch.zeros_like(master)
    v = torch.zeros_like(master)
    w_shards, w_full = (), None
    if level == 3:
        w_shards = [r.w[bounds[i]:bounds[i + 1]].clone() for i in range(ranks)]
        w_full = torch.empty_like(r.w)
    out = w_shards[0] if level == 3 else r.w[off:end]
    log(f"[bench] {cfg.name}: ZeRO-{level}, rank 0 of {ranks}: shard of {end - off} elements")

    def step(t):
        lc.lc_zero_fill_f32(shard, shard.numel(), stream)
        r.run_order_zero(order, level, shard, off, full, w_shards, w_full)
        lc.shard_adam_step(master, m, v, shard, lc.LC_FP32, out, end - off, cfg.lr, cfg.beta1,
                           cfg.beta2, cfg.adam_eps, cfg.weight_decay, t, stream)

    for i in range(warmup):
        step(i + 1)
        torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(steps):
        step(warmup + i + 1)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    tflops = stage_flops_per_mb(cfg) * M / (ms * 1e-3) / 1e12
    persistent = (end - off) * 4 * 4 + (sum(x.numel() for x in w_shards[:1]) * 2 if level == 3
                                        else n * 2)
    temporary = n * 4 + (n * 2 if level == 3 else 0)
    r.close()
    del r
    torch.cuda.empty_cache()
    return ms, tflops, persistent, temporary


def time_launches(torch, stream, fns):
    """Per-launch HIP event timing on `stream`; returns the durations (ms)."""
    out = []
    for fn in fns:
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record(stream)
        fn()
        e.record(stream)
        e.synchronize()
        out.append(s.elapsed_time(e))
    return out


def wgrad_roofline(times):
    """Roofline entry of the weight-gradient GEMM (both operands token-major,
    fp32 accumulate into the bucket; the kernel with the largest share of the
    step's time), from its launches inside the timed steps: achieved =
    average algorithmic FLOP per launch / average launch duration, both over
    every timed launch (the four per-layer shapes dW_qkv = dqkv^T n1,
    dW_o = dh^T o, dW_13 = [dg|du]^T n2, dW_2 = dy^T act, each B)."""
    wms, wfl = times
    n = len(wms)
    avg_ms = sum(wms) / n
    avg_flops = sum(wfl) / n
    achieved = avg_flops / (avg_ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": "gemm_bf16_kernel<false,false,LC_EPI_ACCUM_F32>",
            "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic(),
            "launches": n, "avg_launch_ms": round(avg_ms, 4), "flop_per_launch": avg_flops,
            "timing": "HIP events around each launch inside the timed steps"}


GEMM_SRC = os.path.join(ROOT, "paper_2606_11169_amd", "csrc", "k_gemm.hip")
TRAFFIC_MD = os.path.join(ROOT, "profiles", "gemm_wgrad_traffic.md")
CAL_N = 1 << 26  # calibration: accumulate of 2^26 fp32 elements reads 8 B and writes 4 B each


def gemm_source_hash() -> str:
    import hashlib
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the roofline kernel from the committed PMC
    summary, if it was taken on the current GEMM source (else None)."""
    try:
        lines = open(TRAFFIC_MD).read().splitlines()
    except OSError:
        return None
    vals = {}
    for ln in lines:
        if ln.startswith("traffic_bytes_per_launch:") or ln.startswith("k_gemm_sha256_16:"):
            k, v = ln.split(":", 1)
            vals[k] = v.strip().split()[0]
    if vals.get("k_gemm_sha256_16") != gemm_source_hash():
        return None
    return float(vals["traffic_bytes_per_launch"]) if "traffic_bytes_per_launch" in vals else None


MFMA_MD = os.path.join(ROOT, "profiles", "stage7b_mfma_busy.md")


def csrc_hash() -> str:
    """Digest of every HIP source of the library (the counters depend on all kernels)."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2606_11169_amd", "csrc")
    for name in sorted(os.listdir(d)):
        if name.endswith(".hip"):
            with open(os.path.join(d, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def measured_mfma_busy():
    """Matrix-core busy fraction of the 7B-shaped step from the committed PMC
    summary (SQ_VALU_MFMA_BUSY_CYCLES over the SIMD-cycles its kernels had).
    Not measured by this run: reported with its source file and the source
    digest it was taken on, and only while that digest matches the current
    sources (else None)."""
    try:
        lines = open(MFMA_MD).read().splitlines()
    except OSError:
        return None
    vals = {}
    for ln in lines:
        for key in ("mfma_busy_step:", "csrc_sha256_16:"):
            if ln.startswith(key):
                vals[key[:-1]] = ln.split(":", 1)[1].strip().split()[0]
    if vals.get("csrc_sha256_16") != csrc_hash() or "mfma_busy_step" not in vals:
        return None
    return {"value": float(vals["mfma_busy_step"]),
            "source": os.path.relpath(MFMA_MD, ROOT), "csrc_sha256_16": vals["csrc_sha256_16"],
            "measured": "a separate rocprofv3 --pmc run of one 7B-shaped step (see the source "
                        "file for its command), not this run"}


def calibration_copy(torch, lc, stream):
    """A plain streaming kernel of known HBM traffic (for scaling PMC byte counters)."""
    a = torch.zeros(CAL_N, dtype=torch.float32, device="cuda")
    g = torch.ones(CAL_N, dtype=torch.float32, device="cuda")
    for _ in range(3):
        lc.chunk_accumulate_grad(a, g, lc.LC_FP32, CAL_N, stream=stream)
    torch.cuda.synchronize()
    del a, g


ADAM_MD = os.path.join(ROOT, "profiles", "adam_shard_traffic.md")
OPTIM_SRC = os.path.join(ROOT, "paper_2606_11169_amd", "csrc", "k_optim.hip")


def adam_traffic():
    """HBM bytes per AdamW launch from the committed PMC summary, if it was
    taken on the current k_optim.hip (else None)."""
    import hashlib
    try:
        lines = open(ADAM_MD).read().splitlines()
        h = hashlib.sha256(open(OPTIM_SRC, "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    vals = {}
    for ln in lines:
        for key in ("traffic_bytes_per_launch:", "k_optim_sha256_16:"):
            if ln.startswith(key):
                vals[key[:-1]] = ln.split(":", 1)[1].strip().split()[0]
    if vals.get("k_optim_sha256_16") != h or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def gemm_compare(torch, lc, stream, reps=20, n=4096):
    """Diagnostic: the library's GEMM and hipBLASLt (torch.matmul; the library never calls
    it) on one n^3 product C = A B^T of N(0, 1) bf16 operands, both k-major (the layout of
    the stage's forward products), bf16 output; `reps` launches back to back between two
    HIP events (per-launch events would add each call's host-side launch gap)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    a = torch.randn(n, n, generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn(n, n, generator=g, device="cuda").to(torch.bfloat16)
    c = torch.empty(n, n, dtype=torch.bfloat16, device="cuda")

    def lib():
        lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE, n, n, n, a, n, 1, b, n, 1, c, n, stream=stream)

    def blas():
        torch.matmul(a, b.t(), out=c)

    out = {"workload": f"gemm_nt_{n}^3_bf16", "flop": 2 * n ** 3}
    with torch.cuda.stream(stream):
        for name, fn in (("lc_gemm", lib), ("hipblaslt", blas)):
            for _ in range(3):
                fn()
            stream.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            e1.synchronize()
            ms = e0.elapsed_time(e1) / reps
            out[name] = {"us": round(ms * 1e3, 1), "tflops": round(2 * n ** 3 / (ms * 1e-3) / 1e12, 1)}
    return out


def gemm_compare_shapes(torch, lc, cfg, stream, reps=10):
    """Diagnostic: the library's GEMM main loop (plain bf16 store; the stage's fused
    epilogues left out so both sides do the same work) and hipBLASLt (torch.matmul; the
    library never calls it) at the stage's twelve product shapes and layouts, N(0, 1)
    bf16 operands; `reps` launches back to back between two HIP events per side.
    Layouts as C = A B^T: NT = both operands k-major (forward projections), NN = B
    m/n-major (input gradients), TN = both m/n-major (weight gradients)."""
    T, d, f = cfg.tokens, cfg.d_model, cfg.d_ff
    q = cfg.n_heads * cfg.head_dim + 2 * cfg.kv_heads * cfg.head_dim
    shapes = [("qkv", "NT", T, q, d), ("o", "NT", T, d, d), ("gate_up", "NT", T, 2 * f, d),
              ("down", "NT", T, d, f), ("dn2", "NN", T, d, 2 * f), ("do", "NN", T, d, d),
              ("dn1", "NN", T, d, q), ("dh", "NN", T, f, d), ("dW_qkv", "TN", q, d, T),
              ("dW_o", "TN", d, d, T), ("dW_13", "TN", 2 * f, d, T), ("dW_2", "TN", d, f, T)]
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    out = []
    for name, lay, M, N, K in shapes:
        if lay == "NT":
            a = torch.randn(M, K, generator=g, device="cuda").to(torch.bfloat16)
            b = torch.randn(N, K, generator=g, device="cuda").to(torch.bfloat16)
            args, blas_ab = (a, K, 1, b, K, 1), (a, b.t())
        elif lay == "NN":
            a = torch.randn(M, K, generator=g, device="cuda").to(torch.bfloat16)
            b = torch.randn(K, N, generator=g, device="cuda").to(torch.bfloat16)
            args, blas_ab = (a, K, 1, b, N, 0), (a, b)
        else:
            a = torch.randn(K, M, generator=g, device="cuda").to(torch.bfloat16)
            b = torch.randn(K, N, generator=g, device="cuda").to(torch.bfloat16)
            args, blas_ab = (a, M, 0, b, N, 0), (a.t(), b)
        c = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")

        def lib():
            lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE, M, N, K, *args, c, N, stream=stream)

        def blas():
            torch.matmul(*blas_ab, out=c)
        row = {"product": name, "layout": lay, "M": M, "N": N, "K": K}
        with torch.cuda.stream(stream):
            for side, fn in (("lc_gemm", lib), ("hipblaslt", blas)):
                for _ in range(3):
                    fn()
                stream.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(reps):
                    fn()
                e1.record(stream)
                e1.synchronize()
                ms = e0.elapsed_time(e1) / reps
                row[side] = {"us": round(ms * 1e3, 1), "tflops": round(2 * M * N * K / (ms * 1e-3) / 1e12, 1)}
        row["ratio"] = round(row["hipblaslt"]["us"] / row["lc_gemm"]["us"], 3)
        print(f"[bench] {name} {lay} {M}x{N}x{K}: lc {row['lc_gemm']['us']} us, hipBLASLt "
              f"{row['hipblaslt']['us']} us", file=sys.stderr, flush=True)
        out.append(row)
        del a, b, c
    return {"workload": cfg.name, "timing": f"{reps} launches back to back between HIP events",
            "shapes": out}


def adam_shard(torch, lc, shard, stream, reps=20):
    n = shard.n
    dev = "cuda"
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    p = torch.randn(n, generator=g, device=dev).mul_(shard.p_std)
    m = torch.zeros_like(p)
    v = torch.zeros_like(p)
    gr = torch.randn(n, generator=g, device=dev).mul_(shard.g_std).to(torch.bfloat16)
    out = torch.empty(n, dtype=torch.bfloat16, device=dev)

    def step(t):
        lc.shard_adam_step(p, m, v, gr, lc.LC_BF16, out, n, shard.lr, shard.beta1, shard.beta2,
                           shard.eps, shard.weight_decay, t, stream=stream)
    step(1)
    step(2)
    torch.cuda.synchronize()
    per = sorted(time_launches(torch, stream, [lambda i=i: step(3 + i) for i in range(reps)]))
    med = per[len(per) // 2]
    gbs = 28.0 * n / (med * 1e-3) / 1e9
    del p, m, v, gr, out
    torch.cuda.empty_cache()
    return {"workload": shard.name, "n": n, "bytes_per_elem": 28, "launches": reps,
            "ms": round(med, 3), "ms_min": round(per[0], 3),
            "ms_mean": round(sum(per) / len(per), 3), "value": round(gbs, 1), "unit": "GB/s",
            "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "timing": "median of per-launch HIP events",
            "traffic": adam_traffic(), "algorithmic_bytes": 28 * n}


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, tokens: int, adam_sample: int = 20_000_000):
    """The oracle, as it stands, on one layer of the workload truncated to
    `tokens` positions of one sequence (Chunk F then Chunk B), and its AdamW
    on a slice of the bucket; the full step's oracle time is extrapolated
    from them (every layer and microbatch does the same work)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import optim as OP
    from oracle import stage as OS
    sample = synth.scaled(cfg, n_layers=1, seq_len=tokens, micro_batch=1, bf16=False)
    flat = synth.stage_params(sample, 0)
    X = synth.activation(sample, 0, 0, "x")
    dY = synth.activation(sample, 0, 0, "dy")
    layers = OS.layer_params(sample, flat)
    t0 = time.perf_counter()
    Y, caches = OS.stage_forward(sample, layers, X)
    dX, G = OS.stage_backward(sample, layers, caches, dY)
    dt = time.perf_counter() - t0
    del Y, caches, dX, G, layers, flat
    p, m, v, g = synth.adam_inputs(adam_sample, seed=0)
    t0 = time.perf_counter()
    OP.adamw(p, m, v, g, cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.weight_decay, 1)
    dta = time.perf_counter() - t0
    n_params = synth.param_count(cfg)
    flops = stage_flops_per_mb(sample)
    ratio = stage_flops_per_mb(cfg) * cfg.num_microbatches / flops
    step_s = dt * ratio + dta * n_params / adam_sample
    threads = max([i.get("num_threads", 1) for i in threadpool_info()
                   if i.get("internal_api") == "openblas"] or [1])
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"value": round(flops / dt / 1e12, 4), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"1 of {cfg.n_layers} layers, first {tokens} of {cfg.seq_len} tokens of one "
                      f"microbatch, Chunk F + Chunk B in float64 numpy ({flops / 1e12:.3f} TFLOP; "
                      f"matrix products on {threads} BLAS threads, the rest on one), and AdamW "
                      f"on {adam_sample} elements in {dta:.2f} s",
            "nproc": os.cpu_count(), "affinity_cpus": affinity, "cpu_model": cpu_model(),
            "extrapolated_step_seconds": round(step_s, 1),
            "extrapolation": f"sample time x {ratio:g} (the step's algorithmic FLOP over the "
                             f"sample's) + AdamW time scaled to the {n_params}-element bucket "
                             "(not measured)"}


def streaming_kernels(torch, lc, cfg, stream, reps=20):
    """Achieved HBM GB/s of the stage's bandwidth-bound kernels, each timed
    alone (median of per-launch HIP events) at the 7B-shaped stage's own shapes
    and element types: RMSNorm forward (fp32 residual rows -> bf16 normalised
    rows + fp32 rstd) and backward (fp32 dn, x, dres -> fp32 dx + its bf16
    copy, gain partial sums) over T = 4096 rows of d = 4096, and gradient
    accumulation of an fp32 gradient into the stage's 809.5 M-element fp32
    bucket. Bytes are the algorithmic minimum (each operand read or written
    once)."""
    T, d = cfg.tokens, cfg.d_model
    F32, BF16 = lc.LC_FP32, lc.LC_BF16
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    x = torch.randn((T, d), generator=g, device="cuda")
    dn = torch.randn((T, d), generator=g, device="cuda")
    dres = torch.randn((T, d), generator=g, device="cuda")
    gain = torch.ones(d, dtype=torch.bfloat16, device="cuda")
    n = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    rstd = torch.empty(T, dtype=torch.float32, device="cuda")
    dx = torch.empty((T, d), dtype=torch.float32, device="cuda")
    cp = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    dg = torch.zeros(d, dtype=torch.float32, device="cuda")
    sb = lc.lc_rmsnorm_scratch_bytes(T, d)
    scratch = torch.empty(sb, dtype=torch.uint8, device="cuda")

    def fwd():
        lc.lc_rmsnorm_forward(T, d, x, gain, cfg.rms_eps, n, rstd, F32, BF16, BF16, stream=stream)

    def bwd():
        lc.lc_rmsnorm_backward(T, d, dn, x, rstd, gain, dres, dx, dg, scratch, sb, F32, F32, BF16,
                               F32, F32, dx_copy=cp, stream=stream)
    out = {}
    for name, fn, nbytes in (("rmsnorm_forward", fwd, T * d * (4 + 2) + T * 4),
                             ("rmsnorm_backward", bwd, T * d * (4 * 4 + 2) + T * 4)):
        fn()
        torch.cuda.synchronize()
        per = sorted(time_launches(torch, stream, [fn] * reps))
        med = per[len(per) // 2]
        out[name] = {"value": round(nbytes / (med * 1e-3) / 1e9, 1), "unit": "GB/s",
                     "us": round(med * 1e3, 1), "bytes": nbytes,
                     "frac_hbm": round(nbytes / (med * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del x, dn, dres, n, dx, cp, scratch
    nacc = synth_param_count(cfg)
    acc = torch.zeros(nacc, dtype=torch.float32, device="cuda")
    gr = torch.ones(nacc, dtype=torch.float32, device="cuda")

    def accum():
        lc.chunk_accumulate_grad(acc, gr, F32, nacc, stream=stream)
    accum()
    torch.cuda.synchronize()
    per = sorted(time_launches(torch, stream, [accum] * reps))
    med = per[len(per) // 2]
    out["accumulate"] = {"value": round(12.0 * nacc / (med * 1e-3) / 1e9, 1), "unit": "GB/s",
                         "us": round(med * 1e3, 1), "bytes": 12 * nacc, "n": nacc,
                         "frac_hbm": round(12.0 * nacc / (med * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del acc, gr
    torch.cuda.empty_cache()
    out["timing"] = ("each kernel alone at the 7B-shaped stage's shapes and types, median of "
                     f"{reps} launches timed with HIP events on the launch stream")
    return out


def synth_param_count(cfg):
    import synth
    return synth.param_count(cfg)


MOE_W_DELAY = 1


def moe_schedule(args):
    """The MoE line's schedule: 1F1B with split backwards, each Bi and the
    next microbatch's Bw run as an overlapped pair (fastest measured; the
    flat plain Order with --moe-flat)."""
    return {} if args.moe_flat else {"w_delay": MOE_W_DELAY, "overlap": True}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-adam-shard", action="store_true")
    ap.add_argument("--no-moe", action="store_true")
    ap.add_argument("--moe-only", action="store_true",
                    help="only the MoE stage timing (kernel profiles of that workload)")
    ap.add_argument("--roofline-only", action="store_true",
                    help="only the calibration copy and the 7B-shaped stage with its weight-gradient "
                         "launches timed (PMC runs)")
    ap.add_argument("--split-only", type=int, default=None, metavar="W_DELAY",
                    help="only the 7B-shaped and MoE stages with split backwards (Bw W_DELAY "
                         "backwards after its Bi)")
    ap.add_argument("--qwen3-only", action="store_true",
                    help="only the Qwen3-8B-shaped stage (q/k norm, 8 key/value heads), flat "
                         "and with overlapped pairs")
    ap.add_argument("--overlap", action="store_true",
                    help="7B-shaped stage: run the steady-state (F, B) pairs of the 1F1B Order "
                         "overlapped on two streams (no gain measured there)")
    ap.add_argument("--moe-flat", action="store_true",
                    help="MoE stage: the flat 1F1B Order instead of split backwards with "
                         "overlapped (Bi, Bw) pairs")
    ap.add_argument("--flat", action="store_true",
                    help="with --qwen3-only: the flat Order only (per-kernel profiles)")
    ap.add_argument("--zero-only", action="store_true",
                    help="only the 7B-shaped stage as rank 0 of 8 under ZeRO-2 and ZeRO-3")
    ap.add_argument("--overlap-only", action="store_true",
                    help="only the 7B-shaped and MoE stages with overlapped (F, B) pairs on "
                         "two streams")
    ap.add_argument("--adam-only", action="store_true",
                    help="only the calibration copy and the AdamW shard (PMC runs)")
    ap.add_argument("--streaming-only", action="store_true",
                    help="only the calibration accumulate and the RMSNorm / accumulate kernels at the 7B shapes")
    ap.add_argument("--gemm-shapes", action="store_true",
                    help="diagnostic: the library's GEMM beside hipBLASLt at the 7B stage's twelve product shapes")
    ap.add_argument("--gemm-compare", action="store_true",
                    help="only the library's GEMM beside hipBLASLt on a 4096^3 NT product "
                         "(a diagnostic for the matrix cores' sustained rate)")
    ap.add_argument("--no-streaming", action="store_true",
                    help="skip the RMSNorm / accumulate bandwidth lines")
    ap.add_argument("--cpu-tokens", type=int, default=4096)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the stage; --gpus {args.gpus} is not "
              "supported (no collectives across GPUs are implemented).", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2606_11169_amd import libchunk as lc
    from paper_2606_11169_amd.runner import random_stage, require_gpu

    require_gpu()
    cfg = synth.STAGE_7B
    M = cfg.num_microbatches
    stream = torch.cuda.current_stream()
    if args.moe_only:
        mcfg = synth.MOE_2K
        mms, mtf, _ = time_stage(torch, lc, mcfg, stream, args.steps, args.warmup, "moe",
                                 **moe_schedule(args))
        print(json.dumps({"moe_stage": {"workload": mcfg.name, "value": round(mtf, 2),
                                        "unit": "TFLOP/s", "ms_per_step": round(mms, 2)}}))
        return
    if args.split_only is not None:
        res = {}
        for c in (cfg, synth.MOE_2K):
            sms, stf, sfin = time_stage(torch, lc, c, stream, args.steps, args.warmup, "split",
                                        w_delay=args.split_only)
            res[c.name] = {"w_delay": args.split_only, "value": round(stf, 2),
                           "unit": "TFLOP/s", "ms_per_step": round(sms, 2),
                           "step_ms": STEP_STATS.get("split"), "outputs_finite": sfin}
        print(json.dumps({"split_stage": res}))
        return
    if args.qwen3_only:
        qc = synth.QWEN3_STAGE
        res = {}
        for ov in ((False,) if args.flat else (False, True)):
            qms, qtf, qfin = time_stage(torch, lc, qc, stream, args.steps, args.warmup, "qwen3",
                                        overlap=ov)
            res["overlap" if ov else "flat"] = {
                "value": round(qtf, 2), "unit": "TFLOP/s", "ms_per_step": round(qms, 2),
                "frac": round(qtf / BF16_PEAK_TFLOPS, 4), "outputs_finite": qfin}
        print(json.dumps({"qwen3_stage": {
            "workload": qc.name,
            "algorithmic_tflop_per_step": round(stage_flops_per_mb(qc) * qc.num_microbatches / 1e12, 2),
            **res}}))
        return
    if args.zero_only:
        res = {}
        for level in (2, 3):
            zms, ztf, pers, tmp = time_zero(torch, lc, cfg, stream, args.steps, args.warmup,
                                            level)
            res[f"zero{level}"] = {"value": round(ztf, 2), "unit": "TFLOP/s",
                                   "ms_per_step": round(zms, 2),
                                   "persistent_gib": round(pers / 2**30, 3),
                                   "temporary_gib": round(tmp / 2**30, 3)}
        print(json.dumps({"zero_stage": {"workload": cfg.name, "rank": "0 of 8", **res}}))
        return
    if args.overlap_only:
        res = {}
        for c in (cfg, synth.MOE_2K):
            oms, otf, ofin = time_stage(torch, lc, c, stream, args.steps, args.warmup,
                                        "overlap", overlap=True)
            res[c.name] = {"value": round(otf, 2), "unit": "TFLOP/s",
                           "ms_per_step": round(oms, 2), "outputs_finite": ofin}
        print(json.dumps({"overlap_stage": res}))
        return
    if args.streaming_only:
        calibration_copy(torch, lc, stream)
        print(json.dumps({"streaming": streaming_kernels(torch, lc, cfg, stream, reps=args.steps)}),
              flush=True)
        return
    if args.gemm_shapes:
        print(json.dumps({"gemm_shapes": gemm_compare_shapes(torch, lc, cfg, stream, reps=args.steps)}),
              flush=True)
        return
    if args.gemm_compare:
        print(json.dumps({"gemm_compare": gemm_compare(torch, lc, stream, reps=args.steps)}),
              flush=True)
        return
    if args.adam_only:
        calibration_copy(torch, lc, stream)
        print(json.dumps({"adam_shard": adam_shard(torch, lc, synth.ADAM_1P6B, stream,
                                                   reps=args.steps)}), flush=True)
        return
    if args.roofline_only:
        calibration_copy(torch, lc, stream)
        time_stage(torch, lc, cfg, stream, args.steps, args.warmup, "7b", time_wgrad=True)
        print(json.dumps({"roofline": wgrad_roofline(WGRAD_TIMES["7b"])}), flush=True)
        return
    ms, tflops, finite = time_stage(torch, lc, cfg, stream, args.steps, args.warmup, "7b",
                                    overlap=args.overlap, time_wgrad=True)
    flops = stage_flops_per_mb(cfg) * M
    log(f"[bench] {ms:.1f} ms/step, {tflops:.1f} TFLOP/s ({100 * tflops / BF16_PEAK_TFLOPS:.1f}% of bf16 peak)")

    roof = wgrad_roofline(WGRAD_TIMES["7b"])
    log(f"[bench] roofline {roof}")
    moe = None
    if not args.no_moe:
        mcfg = synth.MOE_2K
        mover = not args.moe_flat
        mms, mtf, mfin = time_stage(torch, lc, mcfg, stream, args.steps, args.warmup, "moe",
                                    **moe_schedule(args))
        moe = {"workload": mcfg.name, "value": round(mtf, 2), "unit": "TFLOP/s",
               "order": f"1F1B(P={mcfg.pp_size},s={mcfg.pp_rank})"
                        + (f" with split backwards (w_delay {MOE_W_DELAY}), each Bi and the "
                           "next Bw overlapped on two streams" if mover else ""),
               "ms_per_step": round(mms, 2), "step_ms": STEP_STATS.get("moe"),
               "frac": round(mtf / BF16_PEAK_TFLOPS, 4),
               "algorithmic_tflop_per_step":
                   round(stage_flops_per_mb(mcfg) * mcfg.num_microbatches / 1e12, 3),
               "outputs_finite": mfin}
        log(f"[bench] moe stage {moe}")
    adam = None if args.no_adam_shard else adam_shard(torch, lc, synth.ADAM_1P6B, stream)
    if adam:
        log(f"[bench] adam shard {adam}")
    streaming = None if args.no_streaming else streaming_kernels(torch, lc, cfg, stream)
    if streaming:
        log(f"[bench] streaming kernels {streaming}")
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, args.cpu_tokens)
        log(f"[bench] cpu baseline {cpu}")

    out = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 2),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg.name, "layers": cfg.n_layers, "d_model": cfg.d_model,
                   "heads": cfg.n_heads, "head_dim": cfg.head_dim, "d_ff": cfg.d_ff,
                   "seq_len": cfg.seq_len, "micro_batch": cfg.micro_batch,
                   "num_microbatches": M,
                   "order": f"1F1B(P={cfg.pp_size},s={cfg.pp_rank})"
                            + (", (F, B) pairs overlapped on two streams" if args.overlap else ""),
                   "optimizer": "AdamW over the stage bucket + bf16 cast",
                   "parallelism": "one GPU's share (no collectives)",
                   "algorithmic_tflop_per_step": round(flops / 1e12, 2)},
        "mfma_util": round(tflops / BF16_PEAK_TFLOPS, 4),
        "mfma_busy_counters": measured_mfma_busy(),
        "step_ms": STEP_STATS.get("7b"),
        "roofline": roof,
        "adam_shard": adam,
        "streaming": streaming,
        "moe_stage": moe,
        "cpu_baseline": cpu,
        "outputs_finite": finite,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
