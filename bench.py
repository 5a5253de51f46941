"""Throughput of the GPT-2 124M training step on one MI355X.

One step = forward (embedding, 12 blocks, final LN, tied LM head, softmax
cross-entropy) + backward + global-norm clip + AdamW, on a micro-batch of
16 x 1024 synthetic Zipf(1.1) tokens already resident in HBM. Prints one JSON
line with tokens/s, model-FLOPs utilisation against the bf16 MFMA peak, a
roofline entry for the dominant kernel (its launches in the last timed step
timed with HIP events on the library's stream) and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def flops_per_token(w: dict) -> float:
    """Algorithmic training FLOPs per token: 6 per matmul parameter (counting
    the LM head on the real vocabulary) plus causal attention (q.k and p.v
    over the unmasked half, three times for forward and backward)."""
    L, C, V, T = w["n_layer"], w["d_model"], w["vocab"], w["T"]
    n_mm = 12 * L * C * C + C * V
    return 6.0 * n_mm + 6.0 * L * C * (T + 1)


def flops_per_token_palm(w: dict, n_params: int) -> float:
    return 6.0 * n_params + 12.0 * w["n_layer"] * w["d_model"] * w["T"]


def qwen3_flops_per_token(w: dict) -> float:
    """Algorithmic FLOPs per token of the adapter step, as the library
    computes it: the frozen projections forward and their input gradients
    (no weight gradients; the first layer's q|k|v input gradient, which would
    only reach the frozen token table, is not computed), the LM head forward
    and input gradient on the positions that carry loss only, causal
    attention (q.k and p.v over the unmasked half, forward and backward),
    and the adapters at their true rank (x A^T, u B^T, dy B, du A and the two
    adapter gradients; du A skipped for the first layer's q|k|v)."""
    L, C, F, V, T, r = w["n_layer"], w["d_model"], w["d_ff"], w["vocab"], w["T"], w["lora_rank"]
    qd, kvd = w["n_head"] * w["head_dim"], w["n_kv_head"] * w["head_dim"]
    qkvd = qd + 2 * kvd
    n_layer_mm = L * (C * qkvd + qd * C + 2 * F * C + F * C)
    loss_frac = (T - int(np.floor(w["loss_from"] * T))) / T
    dense = 4.0 * n_layer_mm - 2.0 * C * qkvd + 4.0 * V * C * loss_frac
    attn = 6.0 * L * qd * (T + 1)
    groups = {"q": ("qkv", C, qd), "k": ("qkv", C, kvd), "v": ("qkv", C, kvd), "o": ("o", qd, C),
              "gate": ("gu", C, F), "up": ("gu", C, F), "down": ("down", F, C)}
    adapter = 0.0
    for t in w["lora_targets"]:
        _, i, o = groups[t]
        adapter += L * 6.0 * r * (i + o) - (2.0 * r * i if t in ("q", "k", "v") else 0.0)
    return dense + attn + adapter


def qwen3_cpu_baseline(w: dict, base: dict, lora: dict, ids, tgt) -> dict:
    """The oracle's adapter step (forward, masked loss, backward, clip, AdamW)
    on the first sequence of the batch through the full model."""
    from oracle import qwen3 as q3
    from threadpoolctl import threadpool_info
    from paper_2609_28568_amd import synth
    ws = dict(w)
    ws["B"] = 1
    cfg = q3.Qwen3Config.from_dict({**ws, **synth.QWEN3_OPTIM})
    lo = {k: v.copy() for k, v in lora.items()}
    m = {k: np.zeros_like(v) for k, v in lo.items()}
    v = {k: np.zeros_like(v) for k, v in lo.items()}
    t0 = time.perf_counter()
    q3.train_step(base, lo, m, v, 0, ids[:1], tgt[:1], cfg)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": round(ws["T"] / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_count": os.cpu_count(),
            "sample": f"one adapter step (fwd+masked loss+bwd+clip+AdamW) on 1 sequence x {ws['T']} tokens of the "
                      f"same model and token stream, numpy fp32, {dt:.1f} s"}


def qwen3_bench(args) -> None:
    """Throughput of the Qwen3-0.6B-shaped adapter step: forward, masked loss,
    backward to the adapters through the frozen base, clip and AdamW on the
    adapters, on B x T synthetic Zipf(1.1) tokens resident in HBM."""
    import torch
    from paper_2609_28568_amd import qwen3_binding as qb, synth

    w = dict(synth.QWEN3_WORKLOADS[args.workload])
    print(f"bench: {args.workload} B={w['B']} T={w['T']} on {torch.cuda.get_device_name(0)}",
          file=sys.stderr, flush=True)
    base, lora = synth.init_qwen3(w)
    ids, tgt = synth.token_batch(w)
    m = qb.Qwen3(qb.make_config(w, synth.QWEN3_OPTIM))
    m.set_fusion("swiglu", args.swiglu)
    m.set_base(base)
    m.set_lora(lora)
    dev_ids, dev_tgt = torch.from_numpy(ids).cuda(), torch.from_numpy(tgt).cuda()
    torch.cuda.synchronize()
    probe = args.probe if args.probe in qb.KCLASS else "attn_bwd"

    def step(i):
        m.forward(dev_ids, dev_tgt)
        m.backward()
        m.adamw_step(i)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"bench: warmup done, loss {m.loss():.4f}", file=sys.stderr, flush=True)
    m.probe_reset()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        if i == args.steps - 1:
            m.probe_enable([probe])
        step(args.warmup + i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    pr = m.probe_read(probe)
    m.probe_enable([])
    loss = m.loss()
    print(f"bench: timed {args.steps} steps, wall {wall:.3f} s, loss {loss:.4f}", file=sys.stderr, flush=True)

    extra = {}
    if args.classes:
        m.probe_reset()
        m.probe_enable(list(qb.KCLASS))
        for i in range(3):
            step(args.warmup + args.steps + i)
        torch.cuda.synchronize()
        for c in qb.KCLASS:
            r = m.probe_read(c)
            if r["launches"]:
                extra[c] = {"ms_per_step": round(r["ms"] / 3, 4), "launches_per_step": r["launches"] // 3,
                            "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 1) if r["flops"] else None,
                            "gbs": round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 1) if r["bytes"] else None}
        m.probe_enable([])
        print("bench: per-class " + json.dumps(extra), file=sys.stderr, flush=True)

    tokens = w["B"] * w["T"]
    tok_s = tokens / (wall / args.steps)
    f_tok = qwen3_flops_per_token(w)
    achieved = pr["flops"] / (pr["ms"] * 1e-3) / 1e12 if pr["ms"] else 0.0
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_from_profiles(probe, args.workload),
                "kernel": probe, "launches": pr["launches"],
                "avg_launch_ms": round(pr["ms"] / max(pr["launches"], 1), 4),
                "flops_per_launch": pr["flops"] / max(pr["launches"], 1)}
    if args.calibration_copy:
        calibration_copy()
    cpu = None
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle on a 1-sequence sample", file=sys.stderr, flush=True)
        cpu = qwen3_cpu_baseline(w, base, lora, ids, tgt)
    out = {
        "metric": "adapter fine-tuning tokens/sec on 1 MI355X, Qwen3-0.6B-shaped, rank-16 adapters; "
                  "bf16 MFMA model-FLOPs util",
        "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"Qwen3-0.6B-shaped adapter step (fwd+masked loss+bwd+clip+AdamW), {args.workload}",
                   "n_layer": w["n_layer"], "d_model": w["d_model"], "n_head": w["n_head"],
                   "n_kv_head": w["n_kv_head"], "head_dim": w["head_dim"], "d_ff": w["d_ff"], "vocab": w["vocab"],
                   "global_batch": w["B"], "seq_len": w["T"], "lora_rank": w["lora_rank"],
                   "lora_targets": list(w["lora_targets"]), "loss_from": w["loss_from"],
                   "tokens_per_step": tokens, "token_dist": "zipf(1.1)", "parallelism": "none",
                   "swiglu_fused": args.swiglu},
        "mfu": round(tok_s * f_tok / (PEAK_BF16_TFLOPS * 1e12), 4),
        "flops_per_token": f_tok,
        "peak_tflops": PEAK_BF16_TFLOPS,
        "gpu_event_ms_per_step": round(gpu_ms / args.steps, 3),
        "final_loss": round(loss, 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if extra:
        out["classes"] = extra
    print(json.dumps(out), flush=True)
    m.close()


def cpu_baseline(w: dict, params, ids, tgt) -> dict:
    """The oracle's step (fwd + bwd + clip + AdamW) on the first four
    sequences of the batch: 4 x 1024 tokens through the full model (about
    20 s on 16 host threads)."""
    import numpy as np
    import oracle
    from threadpoolctl import threadpool_info
    ws = dict(w)
    nb = min(4, len(ids))
    ws["B"] = nb
    cfg = oracle.Config.from_dict({**ws, "lr_min": 6e-5})
    p = {k: v.copy() for k, v in params.items()}
    m = oracle.zero_grads(p)
    v = oracle.zero_grads(p)
    t0 = time.perf_counter()
    oracle.train_step(p, m, v, 0, [(ids[:nb], tgt[:nb])], cfg)
    dt = time.perf_counter() - t0
    info = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    return {"value": round(nb * ws["T"] / dt, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_count": os.cpu_count(), "blas": sorted({i.get("internal_api", "?") for i in info}),
            "sample": f"one optimizer step (fwd+bwd+clip+AdamW) on {nb} sequence(s) x {ws['T']} tokens of the same "
                      f"model and token stream, numpy fp32 with {threads} BLAS threads, {dt:.1f} s"}


def accum_measure(steps: int = 20) -> dict:
    """The accumulation configuration: GPT-2 124M with 32 micro-batches of
    16 x 1024 tokens per optimizer step (524,288 tokens; forward and backward
    accumulating into the fp32 gradients, then clip and AdamW on the
    scheduled rate), one untimed optimizer step, then `steps` consecutive ones
    between two synchronised points, on Zipf-distributed synthetic tokens."""
    import torch
    from paper_2609_28568_amd import binding, synth
    w = dict(synth.WORKLOADS["gpt2_124m_accum32"])
    accum = w["grad_accum"]
    m = binding.GPT2(binding.make_config(w, synth.OPTIM))
    m.set_params(synth.init_params(w))
    dev = [tuple(torch.from_numpy(a).cuda() for a in synth.token_batch(w, micro=i)) for i in range(4)]

    def opt_step(i):
        for k in range(accum):
            ids, tgt = dev[(i * accum + k) % len(dev)]
            m.forward(ids, tgt)
            m.backward(accumulate=k > 0)
        m.adamw_step(i)

    opt_step(0)
    first = m.loss()
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(steps):
        opt_step(1 + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    last = m.loss()
    m.close()
    tokens = w["B"] * w["T"] * accum
    tok_s = tokens * steps / wall
    return {"workload": "GPT-2 124M, 32 micro-batches of 16 x 1024 tokens per optimizer step (gpt2_124m_accum32)",
            "optimizer_steps": steps, "tokens_per_step": tokens, "ms_per_step": round(wall * 1e3 / steps, 2),
            "tokens_per_s": round(tok_s, 1),
            "mfu": round(tok_s * flops_per_token(w) / (PEAK_BF16_TFLOPS * 1e12), 4),
            "gpu_event_ms_step_stats": {"median": round(float(np.median(per_step)), 2),
                                        "min": round(min(per_step), 2), "max": round(max(per_step), 2)},
            "loss_after_first_step": round(first, 4), "loss_last": round(last, 4)}


def device_info() -> dict:
    """The GPU the run used: name, architecture, compute units and peak
    shader clock (hipDeviceGetAttribute), beside the peaks the roofline uses."""
    import ctypes
    import torch
    props = torch.cuda.get_device_properties(0)
    out = {"name": props.name, "arch": getattr(props, "gcnArchName", ""), "compute_units": props.multi_processor_count,
           "peak_bf16_tflops_used": PEAK_BF16_TFLOPS, "peak_hbm_gbs_used": 8000.0}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        v = ctypes.c_int()
        # hipDeviceAttributeClockRate (5): peak clock in kHz
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 5, 0) == 0:
            out["clock_mhz_max"] = v.value / 1000.0
    except OSError:
        pass
    return out


def block_measure(with_cpu: bool) -> dict:
    """The single-block configuration: one GPT-2 124M block on 16 sequences of
    1024 tokens (bf16 input ~ N(0,1), upstream gradient ~ N(0, 1e-3)), forward
    and then backward to the block's weight gradients and its input gradient.
    GPU: 20 passes after 3 untimed ones, timed with HIP events on the stream;
    with_cpu, the oracle's block forward and backward over the same 16
    sequences on the host."""
    import torch
    from paper_2609_28568_amd import binding, synth
    w = dict(synth.WORKLOADS["block124m"])
    B, T, C, F, H = w["B"], w["T"], w["d_model"], w["d_ff"], w["n_head"]
    p = synth.init_params(w)
    x, dy = synth.block_inputs(w)
    m = binding.GPT2(binding.make_config(w, synth.OPTIM))
    m.set_params(p)
    tx = torch.from_numpy(x).cuda().to(torch.bfloat16)
    tdy = torch.from_numpy(dy).cuda().to(torch.bfloat16)
    out, dxin = torch.empty_like(tx), torch.empty_like(tx)

    def one():
        m.block_forward(0, tx, out)
        m.block_backward(0, tdy, dxin)

    for _ in range(3):
        one()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n = 20
    e0.record(stream)
    for _ in range(n):
        one()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    m.close()
    # forward: the four products 2 BT (4 C^2 + 2 C F) and causal attention
    # 4 hd T(T+1)/2 per (sequence, head); the backward twice the forward
    fwd = 2.0 * B * T * (4 * C * C + 2 * C * F) + 4.0 * (C // H) * T * (T + 1) / 2 * B * H
    res = {"workload": "one GPT-2 124M block, 16 x 1024 tokens: forward, then backward to its weight and input "
                       "gradients (block124m)",
           "gpu_ms": round(ms, 3), "gpu_tokens_per_s": round(B * T / (ms * 1e-3), 1),
           "gpu_tflops": round(3 * fwd / (ms * 1e-3) / 1e12, 1), "flops_per_pass": 3 * fwd, "passes": n}
    if with_cpu:
        import oracle
        print("bench: timing the CPU oracle on the single block", file=sys.stderr, flush=True)
        ocfg = oracle.Config.from_dict({**w, "lr_min": 6e-5})
        t0 = time.perf_counter()
        _, cache = oracle.block_forward(x.reshape(B, T, C), p, 0, ocfg)
        grads = oracle.zero_grads(p)
        oracle.block_backward(dy.reshape(B, T, C), cache, p, 0, ocfg, grads)
        dt = time.perf_counter() - t0
        res["cpu_oracle"] = {"value": round(B * T / dt, 1), "unit": "tokens/s", "seconds": round(dt, 2),
                             "kind": "oracle", "cpu_count": os.cpu_count(),
                             "sample": "the same 16 x 1024 tokens through the block, numpy fp32"}
    return res


# Kernel classes with counter-derived traffic: the sources their kernels are
# built from, the pattern of their kernel names in rocprofv3 output, and how
# many kernels one launch of the class runs (the attention backward is the
# dQ kernel and then the dK/dV kernel). The host file that plans the launches
# (shapes, splits, tile configurations) is added per workload.
KERNEL_CLASSES = {
    "gemm_fwd": (("gemm.hip", "common.h", "lds_dma.h", "kernels.h"),
                 r"gemm_kernel<\d+, \d+, \d+, \d+, false, false, 0(, (false|true))*>", 1),
    "gemm_dw": (("gemm.hip", "common.h", "lds_dma.h", "kernels.h"),
                r"gemm_kernel<\d+, \d+, \d+, \d+, true, true, [35](, false)?(, false)?>", 1),
    "gemm_dw_grouped": (("gemm.hip", "common.h", "lds_dma.h", "kernels.h"),
                        r"gemm_kernel<\d+, \d+, \d+, \d+, true, true, [35], false, true>", 1),
    "attn_bwd": (("attention.hip", "common.h", "lds_dma.h", "kernels.h"), r"attn_bwd", 2),
}


def calibration_copy() -> None:
    """A device-to-device copy of CALIBRATION_BYTES, whose counter readings
    scale the kernels' FETCH_SIZE and WRITE_SIZE to bytes."""
    import torch
    src = torch.empty(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def plan_source(workload: str) -> str:
    return "qwen3.cpp" if workload.startswith("qwen3") else "gpt2.cpp"


CALIBRATION_BYTES = 1 << 30


def kernel_source_hash(kernel_tag: str, workload: str) -> str:
    """Hash of the sources the kernel class is built from and of the file that
    plans its launches, so that stored counter readings go stale when either
    changes."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_28568_amd", "csrc")
    for f in KERNEL_CLASSES[kernel_tag][0] + (plan_source(workload),):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def traffic_path(kernel_tag: str, workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"{kernel_tag}_{workload}_traffic.json")


def traffic_from_profiles(kernel_tag: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the kernel's current source."""
    path = traffic_path(kernel_tag, workload)
    if kernel_tag not in KERNEL_CLASSES or not os.path.exists(path):
        return None
    d = json.load(open(path))
    if d.get("source_sha256") != kernel_source_hash(kernel_tag, workload):
        return None
    return d.get("bytes_per_launch")


def pmc_summary(kernel_tag: str, workload: str, fetch_csv: str, write_csv: str, command: str) -> dict:
    """Turn two rocprofv3 counter passes (FETCH_SIZE, WRITE_SIZE; KiB per
    dispatch) into HBM bytes per launch of one kernel class (the class's
    kernels per launch summed), each counter scaled by its reading on a
    device-to-device copy of CALIBRATION_BYTES."""
    import csv
    import re
    pat = re.compile(KERNEL_CLASSES[kernel_tag][1])
    per_launch = KERNEL_CLASSES[kernel_tag][2]

    def read(path, counter):
        kern, copy = [], []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"]) * 1024.0
            if pat.search(r["Kernel_Name"]):
                kern.append(v)
            elif "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) >= 1 << 16:
                copy.append(v)
        if not kern or not copy:
            raise SystemExit(f"{path}: no {counter} rows for {kernel_tag} or for the calibration copy")
        return sum(kern) / len(kern), max(copy), len(kern)

    fk, fc, n = read(fetch_csv, "FETCH_SIZE")
    wk, wc, _ = read(write_csv, "WRITE_SIZE")
    f_scale, w_scale = CALIBRATION_BYTES / fc, CALIBRATION_BYTES / wc
    # read() averages over dispatches; a launch of the class runs per_launch kernels
    return {"kernel": kernel_tag, "dispatches": n, "kernels_per_launch": per_launch,
            "fetch_bytes_raw": fk * per_launch, "write_bytes_raw": wk * per_launch,
            "copy_fetch_bytes_raw": fc, "copy_write_bytes_raw": wc, "fetch_scale": f_scale,
            "write_scale": w_scale, "bytes_per_launch": (fk * f_scale + wk * w_scale) * per_launch,
            "source_sha256": kernel_source_hash(kernel_tag, workload), "command": command}


def pmc_report(workload: str, stats_csv: str, fetch_csv: str, write_csv: str, mfma_csv: str, command: str) -> None:
    """Per-kernel counter summary of one benchmark command: average duration
    (kernel-statistics run), HBM bytes per dispatch from FETCH_SIZE and
    WRITE_SIZE (each scaled by its reading for a device-to-device copy of
    CALIBRATION_BYTES), the bandwidth they make over the average duration,
    and the MFMA busy fraction (rocprofv3's MfmaUtil: MFMA-busy cycles over
    active cycles times SIMDs), written to profiles/<workload>_kernel_counters.md."""
    import csv
    from collections import defaultdict

    def counters(path, name):
        vals, copy = defaultdict(list), []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != name:
                continue
            v = float(r["Counter_Value"])
            if "copyBuffer" in r["Kernel_Name"]:
                if int(r["Grid_Size"]) >= 1 << 16:
                    copy.append(v)
            else:
                vals[r["Kernel_Name"]].append(v)
        return vals, (max(copy) if copy else None)

    stats = {}
    for r in csv.DictReader(open(stats_csv)):
        stats[r["Name"]] = (int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["TotalDurationNs"]) / 1e6)
    fetch, fcopy = counters(fetch_csv, "FETCH_SIZE")
    write, wcopy = counters(write_csv, "WRITE_SIZE")
    mfma, _ = counters(mfma_csv, "MfmaUtil")
    fs = CALIBRATION_BYTES / (fcopy * 1024.0) if fcopy else None
    ws = CALIBRATION_BYTES / (wcopy * 1024.0) if wcopy else None
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_28568_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        h.update(open(os.path.join(csrc, f), "rb").read())
    total = sum(t for _, _, t in stats.values())
    lines = [f"# rocprofv3 kernel counters: {workload}", "",
             "Commands (from the repository root, `R` = its absolute path, each after "
             "`cd /tmp && export TMPDIR=/tmp`):", "", "```", command, "```", "",
             f"Source hash (all of `paper_2609_28568_amd/csrc`): `{h.hexdigest()}`.", "",
             f"Counter scale factors from the 1 GiB device-to-device copy: FETCH_SIZE x {fs:.3f}, "
             f"WRITE_SIZE x {ws:.3f} (KiB per dispatch to bytes).", "",
             "| kernel | calls | avg us | % time | HBM read MB | HBM write MB | HBM GB/s | MFMA busy % |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for name, (calls, avg, tot) in sorted(stats.items(), key=lambda kv: -kv[1][2]):
        if tot < 0.002 * total:
            continue
        fb = sum(fetch[name]) / len(fetch[name]) * 1024.0 * fs if fetch.get(name) and fs else None
        wb = sum(write[name]) / len(write[name]) * 1024.0 * ws if write.get(name) and ws else None
        mu = sum(mfma[name]) / len(mfma[name]) if mfma.get(name) else None
        gbs = (fb + wb) / (avg * 1e-6) / 1e9 if fb is not None and wb is not None else None
        f = lambda x, d: "" if x is None else f"{x:.{d}f}"
        short = name.replace("void ", "").replace("(anonymous namespace)::", "")
        short = short[:short.index("(")] if "(" in short else short
        lines.append(f"| `{short}` | {calls} | {avg:.1f} | {100 * tot / total:.1f} | {f(fb and fb / 1e6, 1)} | "
                     f"{f(wb and wb / 1e6, 1)} | {f(gbs, 0)} | {f(mu, 1)} |")
    lines += ["", "`gemm_kernel<BM, BN, BK, NS, A_T, B_T, EPI, SEG2, GROUPED>`: block tile BM x BN, contraction "
              "step BK, NS-stage LDS ring, A and B read transposed, epilogue (0 bf16 with optional bias, 1 bias + "
              "GELU storing the pre-activation too, 2 GELU derivative, 3 fp32, 4 bf16 with bias and residual, "
              "5 fp32 accumulate, 7 and 8 the two-pass head's softmax statistics and gradient), a second "
              "contraction segment (adapters), the grouped weight-gradient launch. Calls cover the warm-up and "
              "timed steps of the profiled command (no evaluation passes); HBM bytes are per dispatch."]
    out = os.path.join(ROOT, "profiles", f"{workload}_kernel_counters.md")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gpt2_124m")
    ap.add_argument("--probe", default=None, help="kernel class timed for the roofline entry (default: the "
                    "grouped weight-gradient launch for GPT-2, the attention backward for the adapter step)")
    ap.add_argument("--no-eval", action="store_true", help="skip the forward-only evaluation passes")
    ap.add_argument("--pmc-report", nargs=4, metavar=("STATS_CSV", "FETCH_CSV", "WRITE_CSV", "MFMA_CSV"),
                    help="write profiles/<workload>_kernel_counters.md from a rocprofv3 kernel-statistics run and "
                         "three counter passes (FETCH_SIZE, WRITE_SIZE, MfmaUtil) and exit")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--classes", action="store_true", help="also report every kernel class (extra pass)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="after the timed steps, copy 1 GiB device-to-device (counter calibration)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/<probe>_<workload>_traffic.json from two rocprofv3 counter passes and exit")
    ap.add_argument("--pmc-command", default="", help="the profiling command, recorded with --pmc-summary")
    ap.add_argument("--head-ce", type=int, default=0,
                    help="LM head and cross-entropy: 0 logits stored and one cross-entropy kernel, 1 two head "
                         "GEMM passes (softmax statistics, then dlogits) with the logits never stored")
    ap.add_argument("--residual-norm", type=int, default=0,
                    help="how residual connections meet the following pre-norm: 0 in the projection's epilogue, "
                         "1 the fused add + LayerNorm kernel, 2 separate add and LayerNorm kernels")
    ap.add_argument("--no-accum", action="store_true",
                    help="skip the accumulation configuration (20 optimizer steps of 32 micro-batches)")
    ap.add_argument("--no-block", action="store_true",
                    help="skip the single-block (16 x 1024 tokens through one block) measurement")
    ap.add_argument("--swiglu", type=int, default=1,
                    help="Qwen3-shaped workload: 1 SwiGLU in the GEMM epilogues, 0 separate SwiGLU kernels")
    args = ap.parse_args()
    if args.probe is None:
        args.probe = "attn_bwd" if args.workload.startswith("qwen3") else "gemm_dw_grouped"
    if args.pmc_report:
        pmc_report(args.workload, *args.pmc_report, args.pmc_command)
        return
    if args.pmc_summary:
        d = pmc_summary(args.probe, args.workload, *args.pmc_summary, args.pmc_command)
        d["workload"] = args.workload
        with open(traffic_path(args.probe, args.workload), "w") as f:
            json.dump(d, f, indent=1)
        print(json.dumps(d, indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); this build has no multi-GPU path",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_28568_amd import binding, synth

    if args.workload in synth.QWEN3_WORKLOADS:
        qwen3_bench(args)
        return
    w = dict(synth.WORKLOADS[args.workload])
    cfg = binding.make_config(w, synth.OPTIM)
    print(f"bench: {args.workload} B={w['B']} T={w['T']} on {torch.cuda.get_device_name(0)}",
          file=sys.stderr, flush=True)
    params = synth.init_params(w)
    batches = [synth.token_batch(w, micro=i) for i in range(2)]
    m = binding.GPT2(cfg)
    m.set_params(params)
    m.set_fusion("residual_norm", args.residual_norm)
    m.set_fusion("head_ce", args.head_ce)
    dev = [(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()) for a, b in batches]
    torch.cuda.synchronize()

    accum = w.get("grad_accum", 1)

    def step(i):
        # one optimizer step: grad_accum micro-batches (forward + backward
        # accumulating into the gradients), then clip + AdamW
        for k in range(accum):
            ids, tgt = dev[(i * accum + k) % len(dev)]
            m.forward(ids, tgt)
            m.backward(accumulate=k > 0)
        m.adamw_step(i)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"bench: warmup done, loss {m.loss():.4f}", file=sys.stderr, flush=True)

    # The roofline kernel's launches are bracketed with HIP events during the
    # last timed step only: each event pair costs a few microseconds of queue
    # time, which would otherwise inflate every step's time.
    m.probe_reset()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    ev_step = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for i in range(args.steps):
        if i == args.steps - 1:
            m.probe_enable([args.probe])
        step(args.warmup + i)
        ev_step[i].record(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    # per-step times from the events recorded after each step (the last step
    # also carries the roofline kernel's probe events)
    per_step = [ev0.elapsed_time(ev_step[0])] + [ev_step[i - 1].elapsed_time(ev_step[i])
                                                 for i in range(1, args.steps)]
    step_stats = {"median": round(float(np.median(per_step)), 3), "min": round(min(per_step), 3),
                  "max": round(max(per_step), 3)}
    probe = m.probe_read(args.probe)
    m.probe_enable([])
    loss = m.loss()
    print(f"bench: timed {args.steps} steps, wall {wall:.3f} s, events {gpu_ms / 1e3:.3f} s, loss {loss:.4f}",
          file=sys.stderr, flush=True)

    # forward-only evaluation of the same batch (held-out loss path)
    eval_out = None
    if not args.no_eval:
        ev_ids, ev_tgt = dev[0]
        for _ in range(2):
            m.evaluate(ev_ids, ev_tgt)
        n_eval = 10
        t_ev = time.perf_counter()
        for _ in range(n_eval):
            m.evaluate(ev_ids, ev_tgt)
        ev_ms = (time.perf_counter() - t_ev) * 1e3 / n_eval
        eval_out = {"tokens_per_s": round(w["B"] * w["T"] / (ev_ms * 1e-3), 1), "ms_per_pass": round(ev_ms, 3),
                    "passes": n_eval, "note": "forward only, one block's activations kept, logits never stored, "
                                              "no dlogits; each pass synchronises to return its loss"}

    tokens = w["B"] * w["T"] * w.get("grad_accum", 1)
    ms_step = wall * 1e3 / args.steps
    tok_s = tokens / (wall / args.steps)
    f_tok = flops_per_token(w)
    mfu = tok_s * f_tok / (PEAK_BF16_TFLOPS * 1e12)

    extra = {}
    if args.classes:
        classes = list(binding.KCLASS)
        m.probe_reset()
        m.probe_enable(classes)
        for i in range(3):
            step(args.warmup + args.steps + i)
        torch.cuda.synchronize()
        for c in classes:
            r = m.probe_read(c)
            if r["launches"]:
                extra[c] = {"ms_per_step": round(r["ms"] / 3, 4), "launches_per_step": r["launches"] // 3,
                            "tflops": round(r["flops"] / (r["ms"] * 1e-3) / 1e12, 1) if r["flops"] else None,
                            "gbs": round(r["bytes"] / (r["ms"] * 1e-3) / 1e9, 1) if r["bytes"] else None}
        m.probe_enable([])
        print("bench: per-class " + json.dumps(extra), file=sys.stderr, flush=True)

    avg_ms = probe["ms"] / max(probe["launches"], 1)
    achieved = probe["flops"] / (probe["ms"] * 1e-3) / 1e12 if probe["ms"] else 0.0
    flops_launch = probe["flops"] / max(probe["launches"], 1)
    tb = traffic_from_profiles(args.probe, args.workload)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": tb,
                "kernel": args.probe, "launches": probe["launches"], "avg_launch_ms": round(avg_ms, 4),
                "flops_per_launch": flops_launch}

    if args.calibration_copy:
        calibration_copy()

    cpu = None
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle on a 4-sequence sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, params, *batches[0])

    block = None
    if not args.no_block and args.workload == "gpt2_124m":
        block = block_measure(not args.no_cpu_baseline)
    accum_out = None
    if not args.no_accum and args.workload == "gpt2_124m":
        m.close()
        print("bench: timing the accumulation configuration (20 optimizer steps of 32 micro-batches)",
              file=sys.stderr, flush=True)
        accum_out = accum_measure()

    out = {
        "metric": "training tokens/sec on 1 MI355X at GPT-2 124M; bf16 MFMA model-FLOPs util",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"GPT-2 124M training step (fwd+bwd+clip+AdamW), {args.workload}",
                   "n_layer": w["n_layer"], "d_model": w["d_model"], "n_head": w["n_head"],
                   "vocab": w["vocab"], "vocab_padded": w["vocab_padded"], "global_batch": w["B"],
                   "seq_len": w["T"], "grad_accum": w.get("grad_accum", 1), "tokens_per_step": tokens,
                   "token_dist": "zipf(1.1)", "parallelism": "none", "residual_norm": args.residual_norm, "head_ce": args.head_ce},
        "mfu": round(mfu, 4),
        "flops_per_token": f_tok,
        "flops_per_token_6n_12lct": flops_per_token_palm(w, m.n_params - (w["vocab_padded"] - w["vocab"]) * w["d_model"]),
        "peak_tflops": PEAK_BF16_TFLOPS,
        "gpu_event_ms_per_step": round(gpu_ms / args.steps, 3),
        "gpu_event_ms_step_stats": step_stats,
        "device": device_info(),
        "final_loss": round(loss, 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "eval": eval_out,
        "block": block,
        "accum": accum_out,
    }
    if extra:
        out["classes"] = extra
    print(json.dumps(out), flush=True)
    m.close()


if __name__ == "__main__":
    main()
