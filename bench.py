#!/usr/bin/env python3
"""Throughput of the mixed embedding-chunk + decode step on one MI355X.

Workload: one 7B-shape decoder layer in bf16 (hidden 4096, 32 query heads sharing 8 KV heads
of 128, SwiGLU 14336, vocab-32000 LM head) over a 2048-token-budget mixed batch: 1024
embedding-chunk tokens from two requests (chunk 512, last-token pooling; one request resumes
after 1536 cached tokens) plus 64 decode rows with contexts uniform in [1024, 4096] on 16-token
pages.  Weights N(0, 0.02), caches N(0, 1), token ids uniform: all seeded and synthetic.

A step is one orthrus_step call over that batch (every kernel of the path).  The same step is
repeated: the decode rows rewrite their own slot and the resuming request's token count is
restored before each step (a one-element device fill), so every repetition is a valid step.

Prints one JSON line.  `value` = (embedding tokens + decode tokens) per second of step time,
inputs resident in HBM.  `roofline` describes the kernel with the largest share of the step,
from HIP events around each launch on the step's stream.  `cpu_baseline` times the float64
CPU oracle on the same step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
METRIC = "mixed-step throughput: embed tokens/s + decode tokens/s; %MFMA and %HBM peak"
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_gate_up_7b_layer_mixed_traffic.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_25405_amd", "csrc", f) for f in ("gemm.hip", "common.hpp")]


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel: str):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter summary,
    or None when the summary is missing, covers another kernel, or the source changed since."""
    try:
        kv = {}
        with open(TRAFFIC_SUMMARY) as f:
            for line in f:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip().lstrip("- ").strip()] = v.strip()
        if kv.get("step_kernel") != kernel or kv.get("source_sha256") != kernel_source_hash():
            return None
        return float(kv["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def algorithmic_work(cfg, batch):
    """Flops (GEMMs, attention) and bytes (decode KV reads) the step must do, per launch class."""
    T, Te, D = batch.n_tokens, batch.n_emb_tokens, len(batch.rows)
    d, F, V = cfg.d_model, cfg.d_ff, cfg.vocab
    qd, qkv = cfg.q_dim, cfg.qkv_dim
    L = cfg.n_layers
    es = 2 if cfg.dtype == "bf16" else 4
    work = {
        "gemm_qkv": ("flop", 2.0 * T * d * qkv, L),
        "gemm_qkv_rope": ("flop", 2.0 * T * d * qkv, L),   # bf16: rotation and cache append fused
        "gemm_o": ("flop", 2.0 * T * qd * d, L),
        "gemm_gate_up": ("flop", 2.0 * T * d * 2 * F, L),
        "gemm_down": ("flop", 2.0 * T * F * d, L),
        "lm_head": ("flop", 2.0 * D * d * V, 1),
    }
    # attention: chunk rows (query, visible key) pairs on MFMA; decode rows read K and V of every
    # visible key once per KV head
    pairs = sum(sum(c.offset + i + 1 for i in range(c.len)) for c in batch.chunks)
    dec_keys = sum(r.ctx_len + 1 for r in batch.rows)
    work["attention"] = ("byte", 2.0 * dec_keys * cfg.n_kv_heads * cfg.head_dim * es, L)
    work["_attention_flop"] = ("flop", 4.0 * pairs * cfg.head_dim * cfg.n_q_heads, L)
    return work


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0, help="BLAS threads for the oracle (0 = all)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run three plain 1 GiB device copies (the reference kernel for scaling "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        x = torch.ones(256 * 1024 * 1024, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print("copied 1 GiB x3", flush=True)
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the mixed step runs whole on a single MI355X "
              "(independent replicas per GPU; no collective in the method). Use --gpus 1.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_25405_amd import runtime as R
    from workload import layer7b_mixed_workload

    t0 = time.time()
    wl = layer7b_mixed_workload()
    cfg, batch = wl.cfg, wl.batch
    print(f"[bench] workload built in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    dm = R.DeviceModel(cfg, wl.weights)
    kv = R.DeviceKV.from_paged(wl.kv)
    acc_sum = torch.tensor(wl.acc_sum, device="cuda")
    acc_w0 = torch.tensor(wl.acc_w, device="cuda")
    acc_w = acc_w0.clone()
    D, nc = len(batch.rows), len(batch.chunks)
    logits = torch.empty((D, cfg.vocab), device="cuda")
    out_emb = torch.empty((nc, cfg.d_model), device="cuda")
    ws = R.Workspace(dm, dm, batch.n_tokens, nc, D, 4096)
    packed = R.PackedBatch(batch)

    def one_step():
        acc_w.copy_(acc_w0)
        R.step(dm, dm, batch, kv, kv, acc_sum, acc_w, logits, out_emb, ws, packed=packed)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    assert ws.device_error() == 0, "device error during warmup"
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        one_step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    assert ws.device_error() == 0, "device error during timed steps"
    print(f"[bench] {args.steps} steps, {ms:.3f} ms/step", file=sys.stderr, flush=True)

    # per-kernel times: HIP events around each launch, on the step's stream
    R.profile_begin(dm)
    for _ in range(args.steps):
        one_step()
    prof = R.profile_end(dm)
    torch.cuda.synchronize()
    work = algorithmic_work(cfg, batch)
    kernels = {}
    for name, (n, tot) in prof.items():
        avg = tot / max(n, 1)
        ent = {"launches_per_step": n / args.steps, "avg_ms": avg}
        if name in work:
            kind, amount, per_step = work[name]
            per_launch = amount * per_step / (n / args.steps)
            if kind == "flop":
                ent["tflops"] = per_launch / (avg * 1e-3) / 1e12
                ent["frac_mfma"] = ent["tflops"] / PEAK_BF16_TFLOPS
            else:
                ent["gbs"] = per_launch / (avg * 1e-3) / 1e9
                ent["frac_hbm"] = ent["gbs"] / PEAK_HBM_GBS
        kernels[name] = ent
    dom = max(prof, key=lambda k: prof[k][1])
    dk = kernels[dom]
    kind, amount, per_step = work.get(dom, ("flop", 0.0, 1))
    per_launch = amount * per_step / max(dk["launches_per_step"], 1e-9)
    if kind == "flop":
        roof = {"kernel": dom, "bound": "mfma", "achieved": dk.get("tflops"), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": dk.get("frac_mfma"), "traffic": measured_traffic(dom),
                "algorithmic_per_launch": per_launch, "avg_launch_ms": dk["avg_ms"]}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": dk.get("gbs"), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": dk.get("frac_hbm"), "traffic": None,
                "algorithmic_per_launch": per_launch, "avg_launch_ms": dk["avg_ms"]}
    gemm_names = ["gemm_qkv", "gemm_qkv_rope", "gemm_o", "gemm_gate_up", "gemm_down", "lm_head"]
    gemm_flop = sum(work[k][1] * work[k][2] for k in gemm_names if k in prof)
    gemm_ms = sum(prof[k][1] for k in gemm_names if k in prof) / args.steps
    attn_ms = prof.get("attention", (0, 0.0))[1] / args.steps
    Te, T = batch.n_emb_tokens, batch.n_tokens
    result = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) bf16 KV, uniform token ids)",
        "config": {"workload": "7b-layer-mixed-2048: 1 layer d4096 32q/8kv x128 ffn14336 vocab32000 bf16; "
                               "2 chunks x512 (offsets 0 and 1536, last-token pooling) + 64 decode rows "
                               "ctx U[1024,4096], page 16",
                   "embed_tokens": Te, "decode_tokens": D, "layers": cfg.n_layers},
        "embed_tokens_per_s": Te / (ms * 1e-3),
        "decode_tokens_per_s": D / (ms * 1e-3),
        "gemm_frac_mfma": gemm_flop / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS if gemm_ms else None,
        "attention_frac_hbm": kernels.get("attention", {}).get("frac_hbm"),
        "roofline": roof,
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_threads)
    print(json.dumps(result), flush=True)
    return 0


def cpu_baseline(wl, threads: int, min_seconds: float = 10.0):
    """The float64 oracle on the same step (decode rows and both chunks), host cores, repeated
    until about `min_seconds` of CPU work (a bounded sample: whole steps of the same batch)."""
    import numpy as np
    from oracle import OracleKV, step_oracle
    from workload import as_float64
    n = threads or len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        lim = threadpool_limits(limits=n)
    except Exception:
        lim = None
    okv = OracleKV.from_paged(wl.kv)
    W64 = as_float64(wl.weights)   # one-time upcast, like loading, outside the timed calls
    reps, t0 = 0, time.time()
    while reps == 0 or time.time() - t0 < min_seconds:
        # the decode rows rewrite their own slots, so repeating the step is a valid step
        step_oracle((wl.cfg, W64), (wl.cfg, W64), wl.batch, okv, okv, wl.acc_sum, wl.acc_w)
        reps += 1
    dt = (time.time() - t0) / reps
    T = wl.batch.n_tokens
    return {"value": T / dt, "unit": "tokens/s", "cores": n, "kind": "oracle",
            "sample": f"{reps} full steps of the same workload ({T} tokens each), float64 NumPy, "
                      f"{dt:.2f} s per step"}


if __name__ == "__main__":
    sys.exit(main())
