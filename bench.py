#!/usr/bin/env python3
"""Throughput of the BCMT token-mixing layer (forward + backward) on one MI355X.

One step = bcmt_layer_forward + bcmt_layer_backward (input gradient and all
weight and decay gradients) over one batch of synthetic inputs already
resident in HBM.  The workload is the GPT-2-small-shaped layer at the paper's
maximum context: B=8, T=1024, D=768, H=12 heads of 64, block L=128, bf16
storage with float32 accumulation, activations N(0,1), weights N(0, 0.02^2).

Prints one JSON line.  `value` is layer tokens/s = B*T / (time per step).
`roofline` describes the stage with the largest GPU time, measured with HIP
events around each launch in a second pass of the same steps (library stage
tracing).  `cpu_baseline` is the float64 CPU oracle timed on a bounded sample
of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = dict(B=8, T=1024, D=768, H=12, L=128, gamma=0.8, dtype="bf16")
PEAK = {"mfma_bf16_tflops": 2500.0, "mfma_f32_tflops": 157.3, "hbm_gbs": 8000.0}


def stage_work(name, B, T, D, H, L, es):
    """Algorithmic work of one launch of a stage: (bound, amount, unit).

    Matrix stages count 2 flops per multiply-add of the defining product;
    attention counts only the causal pairs of each block; bandwidth stages
    count the bytes each must read and write once."""
    nb = -(-T // L)
    BT = B * T
    pairs = 0
    for s in range(0, T, L):
        n = min(L, T - s)
        pairs += n * (n + 1) // 2
    pairs *= B
    gemm = {
        "fwd.qkv_gemm": 6 * BT * D * D, "fwd.wo_gemm": 2 * BT * D * D,
        "fwd.gate_gemm": 2 * BT * D * D,
        "bwd.wg_wgrad_gemm": 2 * BT * D * D,
        "bwd.wm_wgrad_gemm": 2 * B * nb * D * D, "bwd.wg_dgrad_gemm": 2 * BT * D * D,
        "bwd.wo_dgrad_gemm": 2 * BT * D * D, "bwd.wo_wgrad_gemm": 2 * BT * D * D,
        "bwd.qkv_dgrad_gemm": 6 * BT * D * D, "bwd.qkv_wgrad_gemm": 6 * BT * D * D,
        # long sequences: the memory projections as products of their own
        # (Q = S W_m; dM = dP W_m^T with dP as a bf16 hi + lo pair)
        "fwd.wm_gemm": 2 * B * nb * D * D,
        "bwd.wm_dgrad_gemm": (4 if es == 2 else 2) * B * nb * D * D,
        # QK^T and PV over causal pairs (forward); the backward recomputes
        # QK^T twice and forms dP twice, dV, dK and dQ.
        "fwd.attention": 4 * 64 * H * pairs,
        "bwd.attention_dq": 6 * 64 * H * pairs,
        "bwd.attention_dkdv": 8 * 64 * H * pairs,
        # fused backward: dV, dP, dQ and dK over the causal pairs (the
        # recomputed scores are not credited)
        "bwd.attention_block": 8 * 64 * H * pairs,
    }
    if name in gemm:
        return "mfma", gemm[name], "flop"
    if name.endswith("_reduce"):
        return "hbm", 0, "byte"  # split-K reductions: size depends on the split plan
    act = BT * D * es
    # dw_p partial rows: one per pooling-backward workgroup of 8 row
    # segments of R rows (R a multiple of the rows in flight, for about 1024
    # workgroups, 8 to 64 rows, at most a block)
    nvj = next(n for n in (1, 2, 4, 8) if n * 64 >= D // (16 // es) or n == 8)
    tb = 1 if nvj >= 4 else 4 // nvj
    lb = min(L, T)
    rseg = min(max(-(-(BT // 8192) // tb) * tb, 8), 64, -(-lb // tb) * tb)
    pool_rows = -(-(B * nb * -(-lb // rseg)) // 8)
    fused = nb <= 32  # the single-kernel memory path (projection + scan)
    hbm = {
        "fwd.pool": act + BT * 4 + B * nb * D * 4 + B * nb * 8,
        # single kernel: read S (float32 and compute type) and W_m, write M
        # (both types) and P; long path, the scans alone: read S and Q = S W_m
        # (float32), write M (both types) and P, each once (the two-pass scan
        # reads S and Q twice)
        "fwd.memory_scan": (B * nb * D * (4 + es + 4 + es + 4) + D * D * es) if fused
                           else B * nb * D * (4 + 4 + 4 + es + 4),
        "bwd.gate": 3 * act + B * nb * D * (4 + es),
        # single kernel: read dP (bf16: a hi + lo pair), W_m and M, write dS;
        # long path, the reverse scans alone: read dM and M, write dS
        "bwd.memory_scan": (B * nb * D * ((2 * es if es == 2 else es) + 4 + 4) + D * D * es)
                           if fused else B * nb * D * (4 + 4 + 4),
        # read H, s, dS and S; write a, ds and the dw_p partial rows
        "bwd.pool": act + BT * 12 + B * nb * D * 8 + pool_rows * D * 4,
        "bwd.pool_dwp": pool_rows * D * 4,
        "bwd.zero_grads": (D + 1) * 4,
    }
    return "hbm", hbm.get(name, 0), "byte"


def layer_flops(B, T, D, H, L):
    """Algorithmic forward flops of one layer (projections + causal pairs)."""
    nb = -(-T // L)
    pairs = sum(min(L, T - s) * (min(L, T - s) + 1) // 2 for s in range(0, T, L)) * B
    return 10 * B * T * D * D + 2 * B * (nb - 1) * D * D + 4 * 64 * H * pairs


# Source files whose kernels a stage runs (for matching stored counters).
STAGE_SOURCES = {"attention": ["attention.hip"], "gemm": ["gemm.hip"],
                 "other": ["memory.hip"]}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_sha(stage):
    kind = "attention" if "attention" in stage else ("gemm" if "gemm" in stage else "other")
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_13578_amd", "csrc")
    for f in STAGE_SOURCES[kind] + ["common.h", "kernels.h"]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(stage):
    """HBM bytes per launch from the committed counter summary, or None when
    absent or taken on a different version of the stage's kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(stage)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != source_sha(stage):
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(seconds_target=12.0):
    """The float64 oracle on a bounded sample of the workload (host cores)."""
    import numpy as np
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad, to_f64
    w = WORKLOAD
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max(i.get("num_threads", 0) for i in threadpool_info()) or None
    except Exception:
        pass
    cores = threads or len(os.sched_getaffinity(0))

    def run(bs):
        X, [W] = make_layer_inputs(bs, w["T"], w["D"], seed=0, bf16=True)
        dY = make_upstream_grad(bs, w["T"], w["D"], seed=1, bf16=True)
        t0 = time.perf_counter()
        Y, cache = orc.forward(X.astype(np.float64), to_f64(W), w["L"], w["H"], w["gamma"])
        orc.backward(cache, dY.astype(np.float64))
        return time.perf_counter() - t0

    t1 = run(1)
    bs = max(1, min(w["B"], int(seconds_target / max(t1, 1e-3))))
    # Repeated until at least seconds_target of CPU work (capped at 4x that
    # many repetitions of the estimate, so a slow host stays bounded).
    reps, t = 0, 0.0
    max_reps = max(1, int(4 * seconds_target / max(t1 * bs, 1e-3)))
    while t < seconds_target and reps < max_reps:
        t += run(bs)
        reps += 1
    return {"value": round(reps * bs * w["T"] / t, 1), "unit": "tokens/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{reps} x {bs} of the {w['B']} sequences (T={w['T']}, D={w['D']}, "
                      f"H={w['H']}, L={w['L']}), float64 forward+backward, {t:.1f} s",
            "host": host_info()}


def host_info():
    """The host the oracle ran on: logical CPUs, this process's affinity,
    CPU model and the BLAS NumPy calls (vendor, version, threads)."""
    info = {"cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            info["blas"] = {"vendor": blas[0].get("internal_api"),
                            "version": blas[0].get("version"),
                            "threads": blas[0].get("num_threads")}
    except Exception:
        pass
    return info


# Long-context shape for the bandwidth-bound kernels: at the measured layer
# they move 13-40 MB per launch, too little for a bandwidth figure to mean
# much beside launch latency; here each moves 16x more.
LONG = {"B": 2, "T": 65536, "D": 1024, "H": 16, "L": 256, "gamma": 0.8}


def long_context(make_step, torch, abi, dt, steps=10, warmup=3, make_chunked=None, chunks=4):
    """Layer throughput at the long-context shape and, per bandwidth-bound
    stage (and the attention kernels), bytes moved / stage time against the
    HBM peak.  Stage times come from the library's per-stage tracer (every
    stage alone on one stream).  With make_chunked, the same sequence also
    runs as `chunks` consecutive calls of the chunked entry points (the
    memory state handed from chunk to chunk, the backward in reverse)."""
    g = LONG
    B, T, D, H, L = g["B"], g["T"], g["D"], g["H"], g["L"]
    es = 2 if dt == "bf16" else 4
    step, keep = make_step(B, T, D, H, L, g["gamma"])
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    abi.bcmt_trace_read()
    abi.bcmt_trace_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    stages = abi.bcmt_trace_read()
    abi.bcmt_trace_enable(False)
    print(f"long context B={B} T={T} D={D} H={H} L={L}: {ms * 1e3:.1f} us per step", file=sys.stderr)
    for name, calls, total in stages:
        print(f"  {name:24s} {total / calls * 1e3:10.1f} us", file=sys.stderr)
    act = B * T * D * es
    # attention: Q, K, V read and O written (forward); the fused backward
    # reads Q, K, V, O, dO and writes dQ, dK, dV; the two-kernel backward
    # (blocks over 128 tokens) reads Q, K, V, O, dO and writes dQ, then reads
    # Q, K, V, dO and writes dK, dV
    attn_bytes = {"fwd.attention": 4 * act, "bwd.attention_block": 8 * act,
                  "bwd.attention_dq": 6 * act, "bwd.attention_dkdv": 6 * act}
    res = {}
    for name, calls, total in stages:
        bound, amount, unit = stage_work(name, B, T, D, H, L, es)
        if name in attn_bytes:
            amount, bound = attn_bytes[name], "hbm"
        if bound != "hbm" or amount <= 0:
            continue
        avg_s = total / calls / 1e3
        gbs = amount / avg_s / 1e9
        res[name] = {"us": round(avg_s * 1e6, 1), "bytes": amount, "GB/s": round(gbs, 1),
                     "frac": round(gbs / PEAK["hbm_gbs"], 3)}
    out = {"workload": f"bcmt-layer fwd+bwd B={B} T={T} D={D} H={H}x64 L={L} {dt}",
           "tokens_per_s": round(B * T / (ms / 1e3), 1), "ms_per_step": round(ms, 3),
           "hbm_stages": res}
    if make_chunked is not None:
        del step, keep
        torch.cuda.empty_cache()
        cstep, ckeep = make_chunked(B, T, D, H, L, g["gamma"], chunks)
        for _ in range(warmup):
            cstep()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            cstep()
        e1.record()
        torch.cuda.synchronize()
        cms = e0.elapsed_time(e1) / steps
        print(f"  as {chunks} chunks of {T // chunks} tokens: {cms * 1e3:.1f} us per step",
              file=sys.stderr)
        out["chunked"] = {"chunks": chunks, "tokens_per_chunk": T // chunks,
                          "tokens_per_s": round(B * T / (cms / 1e3), 1),
                          "ms_per_step": round(cms, 3),
                          "time_vs_one_call": round(cms / ms, 3)}
        del cstep, ckeep
    return out


PAPER_SHAPE = {"B": 16, "T": 1024, "D": 128, "H": 8, "Ls": [64, 128, 256, 512, 1024],
               "gamma": 0.8}


def paper_shape(make_step, torch, abi, steps=100, warmup=100):
    """The layer at the paper's model width (d_model 128, 8 heads of 16
    dimensions) over the block sizes it sweeps; L = T is the dense limit
    (one block: plain causal attention, no memory).  Reports fwd+bwd
    tokens/s per L, its ratio to the dense limit, and the layer's device
    buffers (saved activations + the larger workspace)."""
    g = PAPER_SHAPE
    B, T, D, H = g["B"], g["T"], g["D"], g["H"]
    out = {"workload": f"bcmt-layer fwd+bwd B={B} T={T} D={D} H={H}x{D // H} bf16", "by_L": {}}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for L in g["Ls"]:
        step, keep = make_step(B, T, D, H, L, g["gamma"])
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        cfg = keep[0].cfg
        mem = abi.bcmt_saved_bytes(cfg) + max(abi.bcmt_workspace_bytes(cfg, abi.BCMT_PASS_FORWARD),
                                              abi.bcmt_workspace_bytes(cfg, abi.BCMT_PASS_BACKWARD))
        out["by_L"][str(L)] = {"us_per_step": round(ms * 1e3, 1),
                               "tokens_per_s": round(B * T / (ms / 1e3), 1),
                               "device_bytes": int(mem)}
        del step, keep
    dense = out["by_L"][str(T)]["tokens_per_s"]
    for L, r in out["by_L"].items():
        r["vs_dense"] = round(r["tokens_per_s"] / dense, 3)
        print(f"paper shape L={L:>5s}: {r['us_per_step']:8.1f} us per step, "
              f"{r['tokens_per_s'] / 1e6:7.2f} M tokens/s, x{r['vs_dense']:.2f} of dense",
              file=sys.stderr)
    return out


def decay_variants(make_step, torch, steps=100, warmup=100):
    """The measured layer with the decays the paper's sensitivity remark
    spans (0.7, 0.8, 0.9), with one decay per channel (drawn in [0.7, 0.9])
    and with a multi-scale memory (four channel groups decaying at 0.5, 0.8,
    0.95, 0.99): tokens/s fwd+bwd for each."""
    import numpy as np
    w = WORKLOAD
    B, T, D, H, L = w["B"], w["T"], w["D"], w["H"], w["L"]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {"workload": f"bcmt-layer fwd+bwd B={B} T={T} D={D} H={H}x64 L={L} bf16"}
    per_ch = np.random.default_rng(5).uniform(0.7, 0.9, D).astype(np.float32)
    # a multi-scale memory: four channel groups, each with its own decay
    multi = np.repeat(np.array([0.5, 0.8, 0.95, 0.99], np.float32), D // 4)
    for name, gamma in (("gamma=0.7", 0.7), ("gamma=0.8", 0.8), ("gamma=0.9", 0.9),
                        ("per-channel", per_ch), ("multi-scale", multi)):
        step, keep = make_step(B, T, D, H, L, gamma)
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        out[name] = {"us_per_step": round(ms * 1e3, 1), "tokens_per_s": round(B * T / (ms / 1e3), 1)}
        print(f"decay {name:12s}: {ms * 1e3:7.1f} us per step", file=sys.stderr)
        del step, keep
    return out


# The language model of the paper's experiments (Sec. 4.1: d_model 128, 6
# layers, 8 heads, batch 16) with a GPT-2-sized vocabulary; Phase I compares
# the Dense model with BCMT-128 over context lengths, Phase II the block
# sizes at T = 1024 (the paper's two throughput tables).
MODEL = {"V": 50257, "d": 128, "H": 8, "layers": 6, "B": 16, "gamma": 0.8,
         "phase1": {"Ts": [128, 256, 512, 1024], "L": 128},
         "phase2": {"T": 1024, "Ls": [64, 128, 256, 512]}}


def model_bench(torch, abi, steps=20, warmup=20, only=None):
    """Training step (forward, backward, AdamW) of the language model on
    synthetic token ids: tokens/s, device bytes (workspace plus the float32
    parameter, gradient and moment vectors and the bf16 copy) and the ratio
    to the Dense model (L = T) at the same context length."""
    import numpy as np
    from paper_2608_13578_amd.model import ModelBuffers
    m = MODEL
    rng = np.random.default_rng(0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cache = {}

    def run(T, L):
        if (T, L) in cache:
            return cache[(T, L)]
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        mb = ModelBuffers(m["V"], m["d"], m["H"], m["layers"], m["B"], T, L, m["gamma"])
        p = torch.randn(mb.n, device="cuda") * 0.02
        for name, (off, cnt) in zip(mb.names, mb.layout):
            if name.endswith("_g"):
                p[off:off + cnt] = 1.0
            elif name.endswith("_b"):
                p[off:off + cnt] = 0.0
        mb.params.copy_(p)
        del p
        abi.bcmt_model_cast(mb.cfg, mb.params, mb.params_bf16)
        tok = torch.from_numpy(rng.integers(0, m["V"], (m["B"], T)).astype(np.int32)).cuda()
        tgt = torch.roll(tok, -1, 1).contiguous()
        opt = {"lr": 1e-4}
        for _ in range(warmup):
            mb.step(tok, tgt, opt)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        e0.record()
        for _ in range(steps):
            mb.step(tok, tgt, opt)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        # peak device memory of the step, measured: every buffer of the model
        # (workspace, parameters, gradients, moments, tokens) is a torch
        # allocation, and the step allocates nothing of its own
        peak = torch.cuda.max_memory_allocated() - base
        r = {"ms_per_step": round(ms, 3), "tokens_per_s": round(m["B"] * T / (ms / 1e3), 1),
             "device_bytes": int(peak)}
        del mb, tok, tgt
        torch.cuda.empty_cache()
        cache[(T, L)] = r
        return r

    if only is not None:  # one (T, L) configuration, for the profiler
        return run(*only)

    out = {"workload": f"bcmt-lm train step (fwd+bwd+AdamW) V={m['V']} d={m['d']} "
                       f"layers={m['layers']} H={m['H']}x{m['d'] // m['H']} B={m['B']} bf16",
           "phase1": {}, "phase2": {}}
    L1 = m["phase1"]["L"]
    for T in m["phase1"]["Ts"]:
        dense, bc = run(T, T), run(T, L1)
        out["phase1"][str(T)] = {"dense": dense, f"bcmt-{L1}": bc,
                                 "speedup": round(bc["tokens_per_s"] / dense["tokens_per_s"], 3),
                                 "memory_ratio": round(bc["device_bytes"] / dense["device_bytes"], 3)}
    T2 = m["phase2"]["T"]
    dense = run(T2, T2)
    out["phase2"]["dense"] = dense
    for L in m["phase2"]["Ls"]:
        r = dict(run(T2, L))
        r["speedup"] = round(r["tokens_per_s"] / dense["tokens_per_s"], 3)
        r["memory_ratio"] = round(r["device_bytes"] / dense["device_bytes"], 3)
        out["phase2"][f"bcmt-{L}"] = r
    for T, r in out["phase1"].items():
        print(f"model T={T:>5s}: dense {r['dense']['tokens_per_s'] / 1e6:6.2f} M tok/s, "
              f"bcmt-{L1} {r[f'bcmt-{L1}']['tokens_per_s'] / 1e6:6.2f} M tok/s "
              f"(x{r['speedup']:.2f}, memory x{r['memory_ratio']:.2f})", file=sys.stderr)
    return out


DECODE = [{"B": 8, "D": 768, "H": 12, "L": 128, "gamma": 0.8},
          {"B": 2, "D": 1024, "H": 16, "L": 256, "gamma": 0.8}]


def decode_bench(torch, abi, dt, g, blocks=2, warmup_blocks=1):
    """Incremental decoding: time per decode step (one token for each of B
    sequences) over `blocks` whole blocks, and the per-stage times.  The
    weights a step must read (Wq, Wk, Wv, Wo, Wg; Wm once per block) set its
    bandwidth floor."""
    from paper_2608_13578_amd.inputs import make_layer_inputs
    from paper_2608_13578_amd.layer import DecodeBuffers, to_device
    B, D, H, L = g["B"], g["D"], g["H"], g["L"]
    es = 2 if dt == "bf16" else 4
    X, [W] = make_layer_inputs(B, L, D, seed=0, bf16=True)
    db = DecodeBuffers(B, D, H, L, gamma=g["gamma"], dtype=dt)
    db.set_params(W)
    xs = [to_device(X[:, t], dt) for t in range(L)]
    y = torch.empty((B, D), dtype=xs[0].dtype, device="cuda")
    db.reset()
    t = 0
    for _ in range(warmup_blocks * L):
        db.step(t, xs[t % L], y)
        t += 1
    torch.cuda.synchronize()
    n = blocks * L
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        db.step(t, xs[t % L], y)
        t += 1
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / n
    abi.bcmt_trace_read()
    abi.bcmt_trace_enable(True)
    for _ in range(n):
        db.step(t, xs[t % L], y)
        t += 1
    torch.cuda.synchronize()
    stages = abi.bcmt_trace_read()
    abi.bcmt_trace_enable(False)
    wbytes = (5 * D * D + D * D / L) * es
    print(f"decode B={B} D={D} H={H} L={L}: {us:.1f} us per step", file=sys.stderr)
    per = {}
    for name, calls, total in stages:
        per[name] = round(total / calls * 1e3, 2)
        print(f"  {name:24s} {total / calls * 1e3:10.2f} us  x{calls / n:.3f} per step",
              file=sys.stderr)
    return {"workload": f"bcmt-layer decode B={B} D={D} H={H}x64 L={L} {dt}",
            "us_per_step": round(us, 2), "tokens_per_s": round(B / (us * 1e-6), 1),
            "weight_bytes_per_step": int(wbytes),
            "weight_GB/s": round(wbytes / (us * 1e-6) / 1e9, 1), "stage_us": per}


def timed(torch, step, steps, warmup):
    """ms per call of step() over `steps` calls after `warmup` untimed ones."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


# The block-size sweep of the benchmark configurations (B = 16, T = 1024,
# D = 768, 12 heads); L = T is one block, the dense causal baseline.
SWEEP = {"B": 16, "T": 1024, "D": 768, "H": 12, "Ls": [32, 64, 128, 256, 1024], "gamma": 0.8}


def block_size_sweep(make_step, torch, steps=50, warmup=50):
    g = SWEEP
    B, T, D, H = g["B"], g["T"], g["D"], g["H"]
    out = {"workload": f"bcmt-layer fwd+bwd B={B} T={T} D={D} H={H}x64 bf16", "by_L": {}}
    for L in g["Ls"]:
        step, keep = make_step(B, T, D, H, L, g["gamma"])
        ms = timed(torch, step, steps, warmup)
        fl = 3 * layer_flops(B, T, D, H, L)
        out["by_L"][str(L)] = {"us_per_step": round(ms * 1e3, 1),
                               "tokens_per_s": round(B * T / (ms / 1e3), 1),
                               "mfma_frac": round(fl / (ms / 1e3) / 1e12 / PEAK["mfma_bf16_tflops"], 4)}
        print(f"block-size sweep L={L:5d}: {ms * 1e3:8.1f} us per step, "
              f"{B * T / (ms / 1e3) / 1e6:6.2f} M tokens/s", file=sys.stderr)
        del step, keep
    dense = out["by_L"][str(T)]["tokens_per_s"]
    for r in out["by_L"].values():
        r["vs_dense"] = round(r["tokens_per_s"] / dense, 3)
    return out


def long_t_sweep(make_step, torch, Ts=(4096, 16384, 65536), steps=8, warmup=3):
    """The long-context shape at growing T: time per step and tokens/s, and
    the time per token relative to the shortest T (1.0 = linear in T)."""
    g = LONG
    B, D, H, L = g["B"], g["D"], g["H"], g["L"]
    out = {"workload": f"bcmt-layer fwd+bwd B={B} D={D} H={H}x64 L={L} bf16", "by_T": {}}
    base = None
    for T in Ts:
        step, keep = make_step(B, T, D, H, L, g["gamma"])
        ms = timed(torch, step, steps, warmup)
        per_tok = ms / (B * T)
        base = base or per_tok
        out["by_T"][str(T)] = {"ms_per_step": round(ms, 3),
                               "tokens_per_s": round(B * T / (ms / 1e3), 1),
                               "time_per_token_vs_T4096": round(per_tok / base, 3)}
        print(f"long context T={T:6d}: {ms:7.3f} ms per step, "
              f"{B * T / (ms / 1e3) / 1e6:6.2f} M tokens/s", file=sys.stderr)
        del step, keep
        torch.cuda.empty_cache()
    return out


def stack_bench(torch, steps=10, warmup=5, layers=12):
    """Forward then backward through a stack of residual BCMT layers at the
    measured shape: stack time and tokens/s per layer (layers * B * T / t)."""
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad
    from paper_2608_13578_amd.layer import LayerBuffers, SideStream, to_device
    w = WORKLOAD
    B, T, D, H, L = w["B"], w["T"], w["D"], w["H"], w["L"]
    X, Ws = make_layer_inputs(B, T, D, seed=0, bf16=True, n_layers=layers)
    dY = make_upstream_grad(B, T, D, seed=1, bf16=True)
    side = SideStream()
    lbs = []
    for W in Ws:
        lb = LayerBuffers(B, T, D, H, L, gamma=w["gamma"], dtype="bf16", residual=True,
                          side=side)
        lb.set_params(W)
        lbs.append(lb)
    xs = [to_device(X, "bf16")] + [lbs[0].new_activation() for _ in range(layers)]
    dys = [to_device(dY, "bf16")] + [lbs[0].new_activation() for _ in range(layers)]
    grads = [lb.new_grads() for lb in lbs]

    def step():
        for i, lb in enumerate(lbs):
            lb.forward(xs[i], xs[i + 1])
        for i in reversed(range(layers)):
            j = layers - 1 - i
            lbs[i].backward(xs[i], dys[j], dys[j + 1], grads[i])
    ms = timed(torch, step, steps, warmup)
    print(f"{layers}-layer stack: {ms:.3f} ms per step, "
          f"{layers * B * T / (ms / 1e3) / 1e6:.2f} M layer-tokens/s", file=sys.stderr)
    return {"workload": f"{layers} residual bcmt-layers fwd+bwd B={B} T={T} D={D} H={H}x64 L={L} bf16",
            "ms_per_step": round(ms, 3), "tokens_per_s_per_layer": round(layers * B * T / (ms / 1e3), 1),
            "tokens_per_s": round(B * T / (ms / 1e3), 1)}


# The memory path's stress shape: B = 16 sequences of 65536 tokens in
# blocks of 32 (2048 blocks each), D = 1024 (the long-context width).
STRESS = {"B": 16, "T": 65536, "D": 1024, "H": 16, "L": 32, "gamma": 0.8}


def stress_shape(make_step, torch, abi, steps=2, warmup=1):
    """Per-stage times of the bandwidth-bound memory stages at the stress
    shape (every stage alone on one stream), with bytes moved per launch
    against the HBM peak."""
    g = STRESS
    B, T, D, H, L = g["B"], g["T"], g["D"], g["H"], g["L"]
    step, keep = make_step(B, T, D, H, L, g["gamma"])
    timed(torch, step, 1, warmup)
    abi.bcmt_trace_read()
    abi.bcmt_trace_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    stages = abi.bcmt_trace_read()
    abi.bcmt_trace_enable(False)
    res = {}
    for name, calls, total in stages:
        if not any(k in name for k in ("pool", "memory_scan", "bwd.gate")):
            continue
        bound, amount, unit = stage_work(name, B, T, D, H, L, 2)
        avg_s = total / calls / 1e3
        gbs = amount / avg_s / 1e9
        res[name] = {"us": round(avg_s * 1e6, 1), "bytes": amount, "GB/s": round(gbs, 1),
                     "frac": round(gbs / PEAK["hbm_gbs"], 3)}
        print(f"stress {name:22s} {avg_s * 1e6:9.1f} us {gbs:8.1f} GB/s", file=sys.stderr)
    del step, keep
    torch.cuda.empty_cache()
    return {"workload": f"bcmt-layer memory stages B={B} T={T} D={D} L={L} ({T // L} blocks) bf16",
            "hbm_stages": res}


def event_overhead_ms(torch, n=200):
    """Interval of an empty pair of timing events on one stream (what the
    stage tracer adds to each launch it brackets)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for a, b in evs:
        a.record()
        b.record()
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) for a, b in evs)
    return t[len(t) // 2]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # The GPU's clocks take some tens of milliseconds of load to settle: 200
    # warm-up steps (about 70 ms here) reach the steady state that 10 do not.
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-long-context", action="store_true",
                    help="skip the long-context pass (bandwidth kernels at T=65536)")
    ap.add_argument("--no-decode", action="store_true", help="skip the incremental decoding pass")
    ap.add_argument("--no-decay-variants", action="store_true",
                    help="skip the pass over decay values and the per-channel decay")
    ap.add_argument("--no-model", action="store_true",
                    help="skip the language-model pass (paper-shape training step)")
    ap.add_argument("--no-paper-shape", action="store_true",
                    help="skip the pass at the paper's model width (D=128, 16-dim heads)")
    ap.add_argument("--no-sweeps", action="store_true",
                    help="skip the block-size sweep (B=16), the long-context T sweep, the "
                         "12-layer stack and the memory path's stress shape")
    ap.add_argument("--profile-model", action="store_true",
                    help="for rocprofv3: only the language-model training step at T=1024, "
                         "L=128 (--warmup untimed steps, then --steps)")
    ap.add_argument("--profile-run", action="store_true",
                    help="for rocprofv3: a 256 MiB calibration copy, then steps with the "
                         "library's stage tracing on (every stage serialised on one stream, "
                         "as in the per-stage pass of the normal run)")
    ap.add_argument("--shape", default=None,
                    help="with --profile-run: B,T,D,H,L of the layer to profile instead of the "
                         "measured workload (e.g. 16,65536,1024,16,32 for the memory path's "
                         "stress shape)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the layer's multi-GPU sharding is a design, not an implementation)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_13578_amd import bcmt as abi
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad
    from paper_2608_13578_amd.layer import LayerBuffers, to_device

    if not os.path.exists(abi.LIB_PATH):
        from paper_2608_13578_amd.build import build
        build()
    w = WORKLOAD
    B, T, D, H, L = w["B"], w["T"], w["D"], w["H"], w["L"]
    dt = w["dtype"]
    torch.cuda.set_device(0)
    if args.profile_model:
        r = model_bench(torch, abi, steps=args.steps, warmup=args.warmup,
                        only=(1024, MODEL["phase1"]["L"]))
        print(json.dumps({"profile_model": True, "T": 1024, "L": MODEL["phase1"]["L"], **r}))
        return

    def make_step(B, T, D, H, L, gamma):
        X, [W] = make_layer_inputs(B, T, D, seed=0, bf16=True)
        dY = make_upstream_grad(B, T, D, seed=1, bf16=True)
        lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype=dt)
        lb.set_params(W)
        Xd, dYd = to_device(X, dt), to_device(dY, dt)
        del X, dY
        Yd, dXd = lb.new_activation(), lb.new_activation()
        grads = lb.new_grads()

        def step():
            lb.forward(Xd, Yd)
            lb.backward(Xd, dYd, dXd, grads)
        return step, (lb, Xd, dYd, Yd, dXd, grads)

    def make_chunked(B, T, D, H, L, gamma, n):
        """Forward over n consecutive chunks (state handed on), then the
        backward from the last chunk to the first (state gradient handed
        back), weight gradients accumulated."""
        X, [W] = make_layer_inputs(B, T, D, seed=0, bf16=True)
        dY = make_upstream_grad(B, T, D, seed=1, bf16=True)
        tc = T // n
        runs = []
        grads = None
        for k in range(n):
            lb = LayerBuffers(B, tc, D, H, L, gamma=gamma, dtype=dt, accumulate=True)
            lb.set_params(W)
            Xd = to_device(X[:, k * tc:(k + 1) * tc], dt)
            dYd = to_device(dY[:, k * tc:(k + 1) * tc], dt)
            if grads is None:
                grads = lb.new_grads()
            runs.append((lb, Xd, dYd, lb.new_activation(), lb.new_activation(), lb.new_carry(),
                         lb.new_carry()))
        del X, dY

        def step():
            cin = None
            for lb, Xd, dYd, Yd, dXd, cout, dcin in runs:
                lb.forward_chunk(Xd, Yd, cin, cout)
                cin = cout
            dcout = None
            for lb, Xd, dYd, Yd, dXd, cout, dcin in reversed(runs):
                lb.backward_chunk(Xd, dYd, dcout, dXd, dcin, grads)
                dcout = dcin
        return step, (runs, grads)

    if args.shape:
        if not args.profile_run:
            print("bench.py: --shape needs --profile-run", file=sys.stderr)
            sys.exit(2)
        B, T, D, H, L = (int(v) for v in args.shape.split(","))
    step, keep = make_step(B, T, D, H, L, w["gamma"])
    # The GPU's clocks settle after some tens of milliseconds of load: steps
    # for 0.25 s of wall time first, then the requested warm-up steps.
    t_end = time.time() + 0.25
    while time.time() < t_end:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.profile_run:
        # A plain copy of known size: its counter readings calibrate the
        # FETCH_SIZE / WRITE_SIZE counters of the layer's kernels.
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        dst.copy_(src)
        torch.cuda.synchronize()
        abi.bcmt_trace_enable(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        abi.bcmt_trace_read()
        abi.bcmt_trace_enable(False)
        print(json.dumps({"profile_run": True, "steps": args.steps, "shape": [B, T, D, H, L],
                          "calibration_copy_bytes": 256 << 20}))
        return
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    tokens = B * T
    value = tokens / (ms / 1e3)

    # Second pass with per-launch events: per-stage GPU time, each stage
    # alone (tracing keeps the backward's side-stream products on the
    # caller's stream).
    abi.bcmt_trace_read()
    abi.bcmt_trace_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    stages = abi.bcmt_trace_read()
    abi.bcmt_trace_enable(False)
    es = 2 if dt == "bf16" else 4
    rows = []
    for name, calls, total in stages:
        bound, amount, unit = stage_work(name, B, T, D, H, L, es)
        avg_ms = total / calls
        rate = amount / (avg_ms / 1e3)
        rows.append((name, calls // args.steps, avg_ms, total / args.steps, bound, amount, rate))
    traced_ms = sum(r[3] for r in rows)
    print(f"{'stage':24s} {'launch/step':>11s} {'avg us':>9s} {'share':>6s}  achieved", file=sys.stderr)
    for name, per, avg_ms, per_step, bound, amount, rate in rows:
        ach = f"{rate / 1e12:8.1f} TFLOP/s" if bound == "mfma" else f"{rate / 1e9:8.1f} GB/s"
        print(f"{name:24s} {per:11d} {avg_ms * 1e3:9.2f} {per_step / traced_ms:6.1%}  {ach}",
              file=sys.stderr)
    print(f"untraced step {ms * 1e3:.1f} us; traced sum of stages {traced_ms * 1e3:.1f} us",
          file=sys.stderr)
    dom = max(rows, key=lambda r: r[3])
    name, per, avg_ms, per_step, bound, amount, rate = dom
    traffic = stored_traffic(name)
    # The tracer's two events bracket each launch; an empty pair of events
    # takes `ovh` on its own, which the kernel's duration excludes.
    ovh = event_overhead_ms(torch)
    kern_ms = max(avg_ms - ovh, 1e-6)
    rate = amount / (kern_ms / 1e3)
    if bound == "mfma":
        peak = PEAK["mfma_bf16_tflops"] if dt == "bf16" else PEAK["mfma_f32_tflops"]
        roof = {"bound": "mfma", "kernel": name, "achieved": round(rate / 1e12, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(rate / 1e12 / peak, 4), "traffic": traffic}
    else:
        roof = {"bound": "hbm", "kernel": name, "achieved": round(rate / 1e9, 1),
                "peak": PEAK["hbm_gbs"], "unit": "GB/s",
                "frac": round(rate / 1e9 / PEAK["hbm_gbs"], 4), "traffic": traffic}
    roof["avg_launch_us"] = round(kern_ms * 1e3, 2)
    roof["timing"] = (f"per-launch HIP events on the launch stream, {avg_ms * 1e3:.2f} us, "
                      f"minus the {ovh * 1e3:.2f} us of an empty event pair")
    roof["work_per_launch"] = amount
    fl = 3 * layer_flops(B, T, D, H, L)

    out = {
        "metric": "BCMT layer tokens/s (fwd+bwd) at T=1024 bf16",
        "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dt, "data": "synthetic",
        "config": {"workload": "bcmt-layer fwd+bwd B=8 T=1024 D=768 H=12x64 L=128 bf16",
                   "B": B, "T": T, "D": D, "H": H, "L": L, "gamma": w["gamma"]},
        "layer_mfma_frac": round(fl / (ms / 1e3) / 1e12 / PEAK["mfma_bf16_tflops"], 4),
        "roofline": roof,
    }
    del keep, step
    torch.cuda.empty_cache()
    if not args.no_sweeps:
        out["block_size_sweep"] = block_size_sweep(make_step, torch)
        out["stack"] = stack_bench(torch)
        torch.cuda.empty_cache()
    if not args.no_long_context:
        out["long_context"] = long_context(make_step, torch, abi, dt, make_chunked=make_chunked)
        torch.cuda.empty_cache()
    if not args.no_sweeps:
        out["long_context_T"] = long_t_sweep(make_step, torch)
        out["stress_shape"] = stress_shape(make_step, torch, abi)
    if not args.no_decode:
        out["decode"] = [decode_bench(torch, abi, dt, g) for g in DECODE]
    if not args.no_paper_shape:
        out["paper_shape"] = paper_shape(make_step, torch, abi)
    if not args.no_model:
        out["model"] = model_bench(torch, abi)
    if not args.no_decay_variants:
        out["decay_variants"] = decay_variants(make_step, torch)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
