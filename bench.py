#!/usr/bin/env python3
"""Throughput of one fine-tuning step on one MI355X, as one JSON line.

Default workload: the GPT-J-shaped step (28 layers, d 4096, 16 heads of 256
with rotary on 64 dims, parallel attention + MLP block, MLP 16384, vocab
50400, seq 2048, batch 2; bf16 compute, fp32 master weights, AdamW lr 1e-5,
nothing frozen) on seeded uniform-random tokens that stand in for WikiText-2.
A step is forward + backward + AdamW over all 6.05 B parameters; inputs are
resident in HBM before the timed region.  The AdamW step of every weight
matrix whose weight-gradient product runs in the 256 x 256 GEMM kernel is
applied in that product's epilogue (--separate-adamw: all in the separate
pass); the diagnostics report the optimizer's share of the step and the
bandwidth of the separate pass over all parameters.

Reported beside the throughput:
  roofline      the dominant kernel by time: the weight-gradient product of
                the fused QKV + fc1 weight (28672 x 4096 x 4096 tokens), whose
                epilogue also applies that weight's AdamW step (28 B per
                weight element: read p, m, v; write p, m, v, the bf16 copy and
                its transpose).  Timed with HIP events on the model's stream
                around each of its launches inside the timed region; achieved
                = algorithmic FLOPs per launch / mean launch time, against the
                dense bf16 MFMA peak, and beside it the fraction of the serial
                bound (FLOPs at MFMA peak plus the update's bytes at HBM peak).
                traffic = HBM bytes per launch from rocprofv3 FETCH_SIZE /
                WRITE_SIZE counters scaled by the same counters of a 1 GiB
                device copy (bench.py --copy-calibration), read from
                profiles/ when they were taken on the current GEMM source
                (else null).  roofline_qkv_fwd: the same for the fused QKV +
                fc1 forward product (timed in a diagnostic step).
  step_ms       median, p10 and p90 of the timed steps (HIP events between
                consecutive steps on the model's stream).
  cpu_baseline  the float64 oracle timed on this host on a bounded sample
                (two GPT-J-shaped blocks plus embedding and head, one sequence
                of 2048 tokens; AdamW over one block's tensors), scaled to the
                full step by algorithmic FLOPs (forward + backward) and by
                parameter count (AdamW), with the CPU model, the BLAS library
                and its thread count.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU (published: 2.5 PF)
PEAK_HBM_GBS = 8000.0
METRIC = "training tokens/sec + % bf16 MFMA peak, GPT-J-shaped step, 1 MI355X"

WORKLOADS = {
    "gptj": "GPT-J-shaped fine-tuning step: 28 layers, d_model 4096, 16 heads (dh 256, rotary 64), "
            "parallel attn+MLP, MLP 16384, vocab 50400, seq 2048, batch 2, AdamW on all 6.05B params",
    "gpt2s": "GPT-2-small-shaped fine-tuning step: 12 layers, d_model 768, 12 heads, MLP 3072, "
             "vocab 50257, seq 1024, batch 8, AdamW on all params",
    "vith": "ViT-H/14-shaped fine-tuning step: 32 layers, d_model 1280, 16 heads, MLP 5120, "
            "224x224x3 images, 257 tokens, 1000 classes, batch 64, AdamW on all params",
    "gpt2m": "GPT-2-medium-shaped fine-tuning step: 24 layers, d_model 1024, 16 heads, MLP 4096, "
             "vocab 50257, seq 512, batch 8",
    "tiny": "tiny GPT-2-style decoder: 2 layers, d_model 64, 4 heads, MLP 256, vocab 512, seq 32, batch 2",
    "resnet": "ResNet (200M) fine-tuning step: bottleneck ResNet-152 depth (3, 8, 36, 3) at twice the width "
              "(stem 128, 236 M parameters), batch norm in training mode, 224x224x3 images, 1000 classes, "
              "batch 64, AdamW on all params",
    "grid": "model-selection grid: 8 GPT-2-medium-shaped decoders (24 layers, d_model 1024, 16 heads, "
            "MLP 4096, vocab 50257, seq 512), lr {1e-5,3e-5,1e-4,3e-4} x batch {8,16}, bottom 12 blocks "
            "frozen where (lr index + batch index) is odd, one HIP stream each, one shared seed",
}


def step_flops(kw):
    """Algorithmic FLOPs of one step (same formula as the library's
    sat_model_stats): 2 FLOPs per multiply-add of every forward product, twice
    that again for the input- and weight-gradient products of blocks >= k and
    the head, causal attention counted as half the square."""
    d, m, L, k = kw["d_model"], kw["d_mlp"], kw["n_layers"], kw.get("frozen_layers", 0)
    dh = d // kw["n_heads"]
    if kw["arch"] == "vit":
        g = kw["img_size"] // kw["patch"]
        S, npch, pd = g * g + 1, g * g, kw.get("channels", 3) * kw["patch"] ** 2
    else:
        S, npch, pd = kw["seq_len"], 0, 0
    B = kw["batch"]
    T = B * S
    gemm = 2.0 * T * (4 * d * d + 2 * d * m)
    attn = 4.0 * B * kw["n_heads"] * S * S * dh * (1.0 if kw["arch"] == "vit" else 0.5)
    f = L * (gemm + attn) + (L - k) * 2.0 * (gemm + attn)
    rows = B if kw["arch"] == "vit" else T
    f += 3.0 * 2.0 * rows * d * kw["vocab"]
    if kw["arch"] == "vit":
        pe = 2.0 * B * npch * pd * d
        f += pe + (pe if k == 0 else 0.0)
    return f


def _resnet_cfg(kw, **over):
    from oracle import resnet as OR
    c = dict(blocks=tuple(kw["res_blocks"]), width=kw["res_width"], classes=kw["vocab"],
             img_size=kw["img_size"], channels=kw.get("channels", 3), batch=kw["batch"],
             frozen_layers=kw.get("frozen_layers", 0), lr=kw["lr"])
    c.update(over)
    return OR.ResNetConfig(**c)


def n_params(kw):
    import numpy as np
    if kw["arch"] == "resnet":
        from oracle import resnet as OR
        return sum(int(np.prod(s)) for _, s, _ in OR.param_spec(_resnet_cfg(kw)))
    import oracle
    cfg = oracle.Config(**{k: v for k, v in kw.items() if k in oracle.Config.__dataclass_fields__})
    return sum(int(np.prod(s)) for _, s, _ in oracle.param_spec(cfg))


def cpu_baseline_resnet(kw, seed):
    """Oracle fwd+bwd of one image through one block per stage at the full
    width (the stem, every stage's projection block and the head), and AdamW
    over that sample's tensors; scaled to the full step by algorithmic FLOPs
    (forward + backward) and by parameter count (AdamW)."""
    import numpy as np

    from oracle import resnet as OR
    from paper_2309_01226_amd.inputs import batch_for
    cpu_model, blas, threads = _cpu_info()
    scfg = _resnet_cfg(kw, blocks=(1, 1, 1, 1), batch=1)
    full = _resnet_cfg(kw)
    rng = np.random.default_rng(seed)
    P = OR.init_params(scfg, rng)
    x, y = batch_for(dict(kw, batch=1), seed=seed, step=0)
    t0 = time.perf_counter()
    _, cache = OR.forward(scfg, P, x, y)
    G = OR.backward(scfg, P, cache)
    t_fb = time.perf_counter() - t0
    del cache
    t0 = time.perf_counter()
    for n in G:
        z = np.zeros_like(P[n])
        OR.adamw_update(scfg, P[n], G[n], z, z, 1)
    t_opt = time.perf_counter() - t0
    p_s = sum(P[n].size for n in G)
    f_s, f_full = OR.step_flops(scfg), OR.step_flops(full)
    p_full = n_params(kw)
    est = t_fb * f_full / f_s + t_opt * p_full / p_s
    return {
        "value": kw["batch"] / est,
        "unit": "images/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"float64 numpy oracle, one 224x224 image through one block per stage at the full width "
                   f"plus stem and head: fwd+bwd {t_fb:.2f} s scaled by FLOPs x{f_full / f_s:.1f} "
                   f"(extrapolated to {full.n_blocks} blocks and batch {kw['batch']}); AdamW over the "
                   f"sample's {p_s / 1e6:.0f} M params {t_opt:.2f} s scaled by params x{p_full / p_s:.1f}; "
                   f"estimated full step {est:.1f} s"),
        "sample_seconds": round(t_fb + t_opt, 2),
        "extrapolated": True,
        "cpu_model": cpu_model,
        "blas": blas,
        "blas_threads": threads,
        "host_cpus": os.cpu_count(),
    }


def _cpu_info():
    """CPU model name (from /proc/cpuinfo) and the BLAS library numpy uses."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas, threads = "unknown", os.cpu_count()
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = ", ".join(f"{i.get('internal_api')} {i.get('version')} ({os.path.basename(i.get('filepath', ''))})"
                             for i in info)
            threads = max(i.get("num_threads", 1) for i in info)
    except Exception:
        pass
    return model, blas, threads


def cpu_baseline(kw, seed):
    """Oracle fwd+bwd and AdamW on a bounded sample of the same workload: two
    blocks of the real per-layer shapes, one row of the batch (ViT: four
    images), the full embedding and head; the full step's time is
    extrapolated by FLOPs and parameter count."""
    import numpy as np

    import oracle
    from paper_2309_01226_amd.inputs import batch_for
    cpu_model, blas, threads = _cpu_info()
    L_s = min(2, kw["n_layers"])
    sample = dict(kw, n_layers=L_s, frozen_layers=0)
    if kw["arch"] == "vit":
        sample["batch"] = 4
    else:
        sample.update(batch=1)
    fields = oracle.Config.__dataclass_fields__
    cfg = oracle.Config(**{k: v for k, v in sample.items() if k in fields})
    rng = np.random.default_rng(seed)
    P = oracle.init_params(cfg, rng)
    x, y = batch_for(sample, seed=seed, step=0)
    t0 = time.perf_counter()
    loss, cache = oracle.forward(cfg, P, x, y)
    G = oracle.backward(cfg, P, cache)
    t_fb = time.perf_counter() - t0
    del cache
    # AdamW timed on the first block's tensors only (bounded work), scaled by count
    t0 = time.perf_counter()
    p_s = 0
    for n in G:
        if not n.startswith("h0."):
            continue
        z = np.zeros_like(P[n])
        oracle.adamw_update(cfg, P[n], G[n], z, z, 1)
        p_s += P[n].size
    t_opt = time.perf_counter() - t0
    f_s, f_full = step_flops(sample), step_flops(kw)
    p_full = n_params(kw)
    est = t_fb * f_full / f_s + t_opt * p_full / p_s
    rows = kw["batch"] * (kw["seq_len"] if kw["arch"] != "vit" else 1)
    if kw["arch"] == "vit":
        rows = kw["batch"] * ((kw["img_size"] // kw["patch"]) ** 2 + 1)
    srows = sample["batch"] * (sample.get("seq_len", 0) if kw["arch"] != "vit" else
                               (kw["img_size"] // kw["patch"]) ** 2 + 1)
    return {
        "value": rows / est,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"float64 numpy oracle, {L_s} blocks of the same shapes with batch {sample['batch']} x "
                   f"{srows // sample['batch']} tokens ({srows} tokens) plus the full embedding/head: "
                   f"fwd+bwd {t_fb:.2f} s scaled by FLOPs x{f_full / f_s:.1f} (extrapolated to "
                   f"{kw['n_layers']} blocks and the full batch); AdamW over one block's "
                   f"{p_s / 1e6:.0f} M params {t_opt:.2f} s scaled by params x{p_full / p_s:.1f}; "
                   f"estimated full step {est:.1f} s"),
        "sample_seconds": round(t_fb + t_opt, 2),
        "extrapolated": True,
        "cpu_model": cpu_model,
        "blas": blas,
        "blas_threads": threads,
        "host_cpus": os.cpu_count(),
    }


# What the paper reports (end-to-end model-selection makespans of its
# planner, not a per-step figure): context for the measurement, not its target.
PAPER_CONTEXT = {
    "model_selection_runtime_reduction": "39-49 % vs current practice (Abstract, Sec. 5.1)",
    "breakdown": "single node 39-40 %, two homogeneous nodes 43-48 %, two heterogeneous nodes "
                 "(8 + 4 GPUs) 41-45 % (Sec. 5.1)",
    "hardware": "AWS p4d instances: one 8-GPU node, two 8-GPU nodes, or an 8-GPU and a 4-GPU node "
                "(Sec. 5); the GPU model is not named for them (the motivating example in Sec. 1 "
                "uses an 8-GPU A100 instance); PyTorch 2.0, Ray 2.2, Gurobi 10.0",
    "workloads": "TXT: GPT-2 1.5B and GPT-J 6B on WikiText-2; IMG: ViT-G 1.8B and ResNet 200M on ImageNet",
}


def bandwidth_summary(diag, sep_ms, sep_bytes, n_trainable):
    """Achieved HBM GB/s of the bandwidth-bound kernels inside one step
    (algorithmic bytes over the HIP-event durations of their launches), with
    the fraction of the 8 TB/s peak.  The separate AdamW pass is the one over
    all parameters (fusion off), at 30 B per parameter.  LayerNorm tensors of one call (25-300 MB)
    may partly hit the 256 MB Infinity Cache, as they do in the step."""
    out = {}
    for name in ("ln_fwd", "ln_bwd", "xent"):
        ms, n, nbytes = diag.get(name, (0.0, 0, 0.0))
        if n and ms > 0:
            gbs = nbytes / (ms * 1e-3) / 1e9
            out[name] = {"launches": n, "us_per_launch": ms / n * 1e3, "bytes_per_launch": nbytes / n,
                         "gbs": gbs, "frac_hbm": gbs / PEAK_HBM_GBS}
    if sep_ms:
        # 30 B per trainable parameter: read p, g, m, v (16 B); write p, m, v
        # and the bf16 shadow (14 B).  The pass also writes the transposed bf16
        # copy of each weight matrix (2 B per element), counted in bytes_moved.
        b30 = 30.0 * n_trainable
        gbs = b30 / (sep_ms * 1e-3) / 1e9
        out["adamw_all_params"] = {"ms": sep_ms, "bytes_30_per_param": b30, "gbs": gbs,
                                   "frac_hbm": gbs / PEAK_HBM_GBS, "bytes_moved": sep_bytes,
                                   "gbs_moved": sep_bytes / (sep_ms * 1e-3) / 1e9}
    return out


def bandwidth_cold(kw, calls=8):
    """LayerNorm forward and backward and the softmax cross-entropy at the
    workload's shapes, each called `calls` times back to back through the
    kernel-level ABI on input sets that together exceed the 256 MB Infinity
    Cache by rotating over them, so no call finds its operands cached; one
    HIP-event pair around the calls (no per-call event overhead), queued
    behind a spin kernel so that host launch time is not measured.  Bytes are
    algorithmic: LN forward reads 4 and writes 2 B per element (+ 8 B per row
    of statistics); LN backward reads dy, x and the residual gradient and
    writes the residual gradient (16 B per element) plus the statistics; the
    cross-entropy reads 4 and writes 2 B per logit."""
    import torch

    from paper_2309_01226_amd import ops
    T = kw["batch"] * kw["seq_len"]
    d, V = kw["d_model"], kw["vocab"]
    dev = "cuda"
    out = {}

    def timed(fn, n):
        fn(0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # a bounded spin kernel ahead of the calls keeps the GPU behind the host,
        # so the calls run back to back and the Python launch path is not timed
        # (without it, the figure includes the host's launch time)
        spin = getattr(torch.cuda, "_sleep", None)
        if spin is not None:
            spin(20_000_000)
        e0.record()
        for i in range(1, n + 1):  # set 0 was just warmed: start past it
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3  # us per call

    def report(name, us, nbytes):
        out[name] = {"us_per_call": us, "bytes_per_call": nbytes, "gbs": nbytes / us / 1e3,
                     "frac_hbm": nbytes / us / 1e3 / PEAK_HBM_GBS}

    g = torch.ones(d, device=dev)
    b = torch.zeros(d, device=dev)
    nset = max(2, -(-600_000_000 // (T * d * 6)))  # sets of x, y: more than 600 MB in all
    xs = [torch.randn(T, d, device=dev) for _ in range(nset)]
    ys = [torch.empty(T, d, device=dev, dtype=torch.bfloat16) for _ in range(nset)]
    mean = torch.empty(T, device=dev)
    rstd = torch.empty(T, device=dev)
    us = timed(lambda i: ops.layernorm_fwd(xs[i % nset], g, b, ys[i % nset], mean, rstd, T, d, 1e-5),
               calls)
    report("ln_fwd", us, T * d * 6.0 + T * 8.0 + d * 8.0)
    del ys
    dys = [torch.randn(T, d, device=dev) for _ in range(nset)]
    dres = [torch.zeros(T, d, device=dev) for _ in range(nset)]
    dg = torch.empty(d, device=dev)
    db = torch.empty(d, device=dev)
    us = timed(lambda i: ops.layernorm_bwd(dys[i % nset], xs[i % nset], g, mean, rstd, dres[i % nset],
                                           dg, db, T, d), calls)
    report("ln_bwd", us, T * d * 16.0 + T * 8.0 + d * 8.0)
    del xs, dys, dres
    torch.cuda.empty_cache()
    z = torch.randn(T, V, device=dev)  # T x V fp32: larger than the Infinity Cache on its own
    labels = torch.randint(0, V, (T,), device=dev, dtype=torch.int32)
    row_loss = torch.empty(T, device=dev)
    dz = torch.empty(T, V, device=dev, dtype=torch.bfloat16)
    inv_n = torch.full((1,), 1.0 / T, device=dev)
    us = timed(lambda i: ops.cross_entropy(z, labels, row_loss, dz, inv_n, T, V), max(2, calls // 4))
    report("xent", us, T * V * 6.0 + T * 8.0)
    del z, dz
    torch.cuda.empty_cache()
    out["note"] = ("isolated calls through the kernel-level ABI, operands evicted from the Infinity "
                   "Cache between uses; LN backward includes its two column-sum launches")
    return out


def traffic_from_profiles(name):
    """HBM bytes per launch of a GEMM from the committed counter summary
    profiles/<name>, if it was taken on the current GEMM source (else None)."""
    path = os.path.join(ROOT, "profiles", name)
    src = os.path.join(ROOT, "paper_2309_01226_amd", "csrc", "gemm256.hip")
    try:
        rec = {}
        for line in open(path):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
        cur = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if rec.get("gemm_source_sha256") != cur:
            return None
        return float(rec["hbm_bytes_per_launch"])
    except Exception:
        return None


def copy_calibration(nbytes=1 << 30, reps=3):
    """A plain device copy of known size, for scaling the FETCH_SIZE /
    WRITE_SIZE counters of other kernels (run under rocprofv3 --pmc)."""
    import torch
    x = torch.ones(nbytes // 4, device="cuda", dtype=torch.float32)
    y = torch.empty_like(x)
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def bench_grid(args):
    """All grid members advance one step per round, each on its own stream;
    the round is timed from the first enqueue to the last member's end."""
    import torch

    from paper_2309_01226_amd.configs import grid_members
    from paper_2309_01226_amd.inputs import decoder_batch
    from paper_2309_01226_amd.model import Model

    torch.cuda.set_device(0)
    kws = grid_members()
    streams = [torch.cuda.Stream() for _ in kws]
    models = [Model(kw, stream=st) for kw, st in zip(kws, streams)]
    # the members' own streams already overlap their steps; a second stream per
    # member measured 1.5 % slower on this grid
    for m in models:
        if args.separate_adamw:
            m.set_option("fused_adamw", 0)
        m.set_option("overlap_wgrad", 0)
    rows = max(kw["batch"] for kw in kws)
    K, W = args.steps, args.warmup
    batches = []
    for t in range(W + K):
        per = []
        for kw in kws:
            x, y = decoder_batch(kw["batch"], kw["seq_len"], kw["vocab"], seed=args.seed, step=t,
                                 rows=rows)
            per.append((torch.as_tensor(x).cuda(), torch.as_tensor(y).cuda()))
        batches.append(per)
    torch.cuda.synchronize()

    def round_(t):
        for m, (x, y) in zip(models, batches[t]):
            m.train_step(x, y, sync=False)

    for t in range(W):
        round_(t)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(K):
        round_(W + t)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    flops = sum(m.stats()[2] for m in models)
    tokens = sum(kw["batch"] * kw["seq_len"] for kw in kws)
    losses = [m.eval_loss(*batches[0][i]) for i, m in enumerate(models)]
    out = {
        "metric": "model-selection grid training tokens/sec, 8 GPT-2-medium-shaped members, 1 MI355X",
        "value": tokens * K / dt, "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": dt / K * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": WORKLOADS["grid"], "name": "grid", "tokens_per_round": tokens,
                   "overlap_wgrad": False,
                   "members": [{"lr": kw["lr"], "batch": kw["batch"], "frozen_layers": kw["frozen_layers"]}
                               for kw in kws]},
        "round_tflop": flops / 1e12,
        "achieved_tflops": flops / (dt / K) / 1e12,
        "mfu": flops / (dt / K) / 1e12 / PEAK_BF16_TFLOPS,
        "loss_after": losses,
    }
    for m in models:
        m.close()
    print(json.dumps(out), flush=True)


def bench_grid_plan(args):
    """The grid as a planned run: every member profiled alone (sat_profile),
    the concurrency slowdown measured on one member, the lane count and LPT
    assignment with the smallest estimated makespan chosen (schedule.plan),
    then the plan executed for K steps per member and its makespan timed, next
    to the estimate and to all members at once on their own streams."""
    import torch

    from paper_2309_01226_amd import schedule
    from paper_2309_01226_amd.configs import grid_members

    torch.cuda.set_device(0)
    kws = grid_members()
    K = args.steps
    prof = [schedule.profile(kw, warmup=args.warmup, steps=K) for kw in kws]
    costs = [p["step_ms_mean"] * K for p in prof]
    mem = [p["arena_bytes"] for p in prof]
    slow = schedule.measure_slowdown(kws[0], [1, 2, 4, 8], steps=max(K, 5))
    pl = schedule.plan(costs, mem, slow, mem_budget=int(0.8 * torch.cuda.get_device_properties(0).total_memory))

    def timed(lanes):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        schedule.run_plan([(kw, K) for kw in kws], lanes, seed=args.seed, keep_params=False)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3

    tokens = sum(kw["batch"] * kw["seq_len"] for kw in kws) * K
    ms_plan = timed(pl["lanes"])
    ms_all = timed([[i] for i in range(len(kws))])
    print(json.dumps({
        "metric": "model-selection grid makespan, planned on one MI355X (profile -> plan -> run)",
        "value": tokens / (ms_plan * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "higher_is_better": True, "data": "synthetic",
        "config": {"workload": WORKLOADS["grid"], "name": "grid-plan"},
        "profiles_step_ms": [p["step_ms_mean"] for p in prof],
        "slowdown": slow, "n_lanes": pl["n_lanes"], "lanes": pl["lanes"],
        "est_makespan_ms": pl["est_makespan"], "makespan_ms": ms_plan,
        "makespan_all_concurrent_ms": ms_all,
        "note": "measured makespans include creating each member (arena, init) and its final eval",
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="gptj", choices=sorted(WORKLOADS))
    ap.add_argument("--plan", action="store_true",
                    help="with --config grid: profile, plan and run the grid (stream packing)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--checkpoint", action="store_true",
                    help="activation checkpointing: recompute each block's activations in the backward")
    ap.add_argument("--separate-adamw", action="store_true",
                    help="update every tensor in the separate AdamW pass (SAT_OPT_FUSED_ADAMW 0) "
                         "instead of fusing eligible weights' steps into their weight-gradient products")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run the blocks' weight-gradient products on the model's stream "
                         "(SAT_OPT_OVERLAP_WGRAD 0) instead of the weight-gradient stream")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path; run it with "
              "--gpus 1 (the default).", file=sys.stderr, flush=True)
        sys.exit(2)

    if args.config == "grid":
        bench_grid_plan(args) if args.plan else bench_grid(args)
        return

    import torch

    from paper_2309_01226_amd.configs import preset
    from paper_2309_01226_amd.model import TIMING, Model, device_batch

    kw = preset(args.config)
    if args.checkpoint:
        kw["checkpoint"] = 1
    torch.cuda.set_device(0)
    m = Model(kw)
    if args.separate_adamw:
        m.set_option("fused_adamw", 0)
    overlap = not args.no_overlap
    m.set_option("overlap_wgrad", int(overlap))
    n_all, n_train, flops = m.stats()
    resnet = kw["arch"] == "resnet"
    if not resnet:
        assert abs(flops - step_flops(kw)) <= 1e-9 * flops, (flops, step_flops(kw))
    K, W = args.steps, args.warmup
    batches = [device_batch(kw, seed=args.seed, step=t) for t in range(W + K)]
    tokens = m.rows() if kw["arch"] != "vit" else m.rows()
    for t in range(W):
        m.train_step(*batches[t], sync=False)
    torch.cuda.synchronize()
    per_step = kw["n_layers"] - kw.get("frozen_layers", 0)
    # the dominant kernel class: the fused QKV (+ fc1) weight-gradient product
    # with its AdamW epilogue; for the ResNet, the 3x3 convolution forward products
    dominant = "qkv_fwd_gemm" if resnet else "qkv_wgrad_gemm"
    m.set_timing(TIMING[dominant], (kw["n_layers"] if resnet else per_step) * K + 8)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(m.stream)
    for t in range(K):
        m.train_step(*batches[W + t], sync=False)
        ev[t + 1].record(m.stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    w_ms, w_n, w_fl = m.timing_read()
    step_ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(K))

    # diagnostics outside the timed region: one step per kernel class, as
    # timed (AdamW of the eligible weights fused into their weight-gradient
    # products), then with every tensor in the separate AdamW pass: that pass
    # over all parameters is the optimizer's bandwidth kernel, and the GEMM
    # time without the fused epilogues gives the optimizer's share of the step
    # Per-launch durations are those of kernels running alone: the
    # diagnostic steps keep every launch on the model's stream.
    m.set_option("overlap_wgrad", 0)
    diag = {}
    diag_kinds = ("adamw", "all_gemm", "xent") if resnet else \
        ("qkv_fwd_gemm", "qkv_wgrad_gemm", "adamw", "all_gemm", "attn_fwd", "attn_bwd", "ln_fwd", "ln_bwd",
         "xent")
    for name in diag_kinds:
        m.set_timing(TIMING[name], 4096)
        m.train_step(*batches[0], sync=False)
        diag[name] = m.timing_read()
    if not args.separate_adamw:
        m.set_option("fused_adamw", 0)
    for name in ("adamw", "all_gemm"):
        m.set_timing(TIMING[name], 4096)
        m.train_step(*batches[0], sync=False)
        diag[name + "_separate"] = m.timing_read()
    m.set_option("fused_adamw", 0 if args.separate_adamw else 1)
    m.set_option("overlap_wgrad", int(overlap))
    m.set_timing(0, 0)
    loss = m.train_step(*batches[0])

    ms_step = dt / K * 1e3
    step_tflops = flops / (dt / K) / 1e12
    adamw_ms = diag["adamw"][0]
    sep_ms, _, sep_bytes = diag["adamw_separate"]
    # optimizer time inside the step: the separate pass that remains, plus
    # what the fused epilogues add to the GEMMs
    opt_ms = adamw_ms + max(diag["all_gemm"][0] - diag["all_gemm_separate"][0], 0.0)
    out = {
        "metric": ("training images/sec + % bf16 MFMA peak, ResNet (200M) step, 1 MI355X" if resnet
                   else METRIC),
        "value": tokens * K / dt,
        "unit": "images/s" if resnet else "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_step,
        "step_ms": {"median": step_ms[len(step_ms) // 2] if K % 2 else
                    0.5 * (step_ms[K // 2 - 1] + step_ms[K // 2]),
                    "p10": step_ms[int(0.1 * (K - 1))], "p90": step_ms[int(round(0.9 * (K - 1)))],
                    "min": step_ms[0], "max": step_ms[-1]},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "name": args.config,
                   "global_batch": kw["batch"], "seq_len": 1 if resnet else m.rows() // kw["batch"],
                   "tokens_per_step": tokens, "params": n_all, "trainable_params": n_train,
                   "frozen_layers": kw.get("frozen_layers", 0), "checkpoint": kw.get("checkpoint", 0),
                   "overlap_wgrad": overlap,
                   "arena_gb": m.nbytes / 1e9},
        "step_tflop": flops / 1e12,
        "achieved_tflops": step_tflops,
        "mfu_step": step_tflops / PEAK_BF16_TFLOPS,
        "mfu_fwd_bwd": flops / ((dt / K) - opt_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "optimizer": {
            "fused_into_wgrad_gemms": not args.separate_adamw,
            "in_step_ms": opt_ms,
            "separate_pass_in_step_ms": adamw_ms,
            "separate_pass_all_params": {
                "ms": sep_ms, "gbs": sep_bytes / (sep_ms * 1e-3) / 1e9 if sep_ms else None,
                "frac_hbm": sep_bytes / (sep_ms * 1e-3) / 1e9 / PEAK_HBM_GBS if sep_ms else None},
        },
        "all_gemm": {"ms": diag["all_gemm"][0], "launches": diag["all_gemm"][1],
                     "tflops": diag["all_gemm"][2] / (diag["all_gemm"][0] * 1e-3) / 1e12,
                     "ms_without_fused_optimizer": diag["all_gemm_separate"][0],
                     "tflops_without_fused_optimizer":
                         diag["all_gemm_separate"][2] / (diag["all_gemm_separate"][0] * 1e-3) / 1e12},
        "bandwidth_kernels": bandwidth_summary(diag, sep_ms, sep_bytes, n_train),
        "loss_after": loss,
        "paper_context": PAPER_CONTEXT,
    }
    if not resnet:
        out["attention"] = {"fwd_ms": diag["attn_fwd"][0], "bwd_ms": diag["attn_bwd"][0],
                            "fwd_tflops": diag["attn_fwd"][2] / max(diag["attn_fwd"][0], 1e-9) / 1e9,
                            "bwd_tflops": diag["attn_bwd"][2] / max(diag["attn_bwd"][0], 1e-9) / 1e9}
    ncols = 3 * kw.get("d_model", 0) + kw.get("d_mlp", 0) if kw["arch"] == "gptj" else 3 * kw.get("d_model", 0)
    if w_n and resnet:
        achieved = w_fl / w_n / (w_ms / w_n * 1e-3) / 1e12
        out["roofline"] = {
            "kernel": "3x3 convolution forward products (im2col operand x weight, fp32 out), "
                      "mean over the 50 per step",
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
            "launches": w_n, "avg_ms": w_ms / w_n, "flop_per_launch": w_fl / w_n,
        }
    elif w_n:
        fused = not args.separate_adamw
        achieved = w_fl / w_n / (w_ms / w_n * 1e-3) / 1e12
        opt_bytes = 28.0 * ncols * kw["d_model"] if fused else 0.0
        serial_us = (w_fl / w_n / (PEAK_BF16_TFLOPS * 1e12) + opt_bytes / (PEAK_HBM_GBS * 1e9)) * 1e6
        out["roofline"] = {
            "kernel": (f"gemm256_kernel<4, 0> (AdamW epilogue): weight gradient of the fused QKV + fc1 weight "
                       f"({ncols} x {kw['d_model']} x {m.rows()} tokens) with that weight's AdamW step"
                       if fused else
                       f"gemm256_kernel<0, 0>: weight gradient of the fused QKV + fc1 weight "
                       f"({ncols} x {kw['d_model']} x {m.rows()} tokens)"),
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic_from_profiles("gemm_qkv_wgrad_adamw_gptj_traffic.txt") if fused else None,
            "launches": w_n, "avg_ms": w_ms / w_n, "flop_per_launch": w_fl / w_n,
            "optimizer_bytes_per_launch": opt_bytes,
            "optimizer_bytes_per_element": 28 if fused else 0,
            "serial_bound_us": serial_us,
            "frac_of_serial_bound": serial_us / (w_ms / w_n * 1e3),
            "note": "dominant kernel by time per step; serial bound = FLOPs at the MFMA peak plus the "
                    "fused AdamW bytes at the 8 TB/s HBM peak",
        }
        i_ms, i_n, i_fl = diag["qkv_wgrad_gemm"]
        if i_n:
            # the same launches in a diagnostic step with every launch on the model's stream: with the
            # weight-gradient stream on, the timed launches share the chip with the input-gradient chain
            out["roofline"]["alone"] = {
                "avg_ms": i_ms / i_n, "achieved": i_fl / i_ms * 1e-9,
                "frac": i_fl / i_ms * 1e-9 / PEAK_BF16_TFLOPS,
                "frac_of_serial_bound": serial_us / (i_ms / i_n * 1e3)}
    q_ms, q_n, q_fl = diag["qkv_fwd_gemm"] if "qkv_fwd_gemm" in diag else (0.0, 0, 0.0)
    if q_n:
        achieved = q_fl / q_n / (q_ms / q_n * 1e-3) / 1e12
        out["roofline_qkv_fwd"] = {
            "kernel": "gemm256_kernel<2, 0> (bf16 epilogue, GELU on the fc1 columns): fused QKV + fc1 forward "
                      f"({m.rows()} x {ncols} x {kw['d_model']})",
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic_from_profiles("gemm_qkv_fc1_fwd_gptj_traffic.txt"),
            "launches": q_n, "avg_ms": q_ms / q_n, "flop_per_launch": q_fl / q_n,
        }
    if "seq_len" in kw:  # token workloads: LayerNorm and vocabulary cross-entropy shapes
        out["bandwidth_kernels_cold"] = bandwidth_cold(kw)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_resnet(kw, args.seed) if resnet else cpu_baseline(kw, args.seed)
    m.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
