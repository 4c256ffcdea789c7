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
    """SHA-256 of the dominant kernel's sources with comments and whitespace removed: a change of
    code invalidates the committed counter summary, a change of comments does not."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)   # block comments
        text = re.sub(r"//[^\n]*", " ", text)                # line comments (no '//' in strings here)
        h.update(" ".join(text.split()).encode())
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


def step_roofline(cfg, batch, t_step_ms):
    """Ideal step time if every kernel class ran at its own roofline, one after another:
    sum over classes of max(F / bf16 MFMA peak, B / HBM peak), with F the algorithmic flops and
    B the least HBM bytes the class must move (weights, activations in and out, the KV it reads
    and writes, the residual stream read and written once; split-K slabs, partials and
    metadata are implementation traffic and not counted).  Returns (ideal_ms, ideal / measured)."""
    T, Te, D = batch.n_tokens, batch.n_emb_tokens, len(batch.rows)
    d, F, V = cfg.d_model, cfg.d_ff, cfg.vocab
    qd, kvd, qkv = cfg.q_dim, cfg.kv_dim, cfg.qkv_dim
    es = 2 if cfg.dtype == "bf16" else 4
    L = cfg.n_layers
    pairs = sum(sum(c.offset + i + 1 for i in range(c.len)) for c in batch.chunks)
    dec_keys = sum(r.ctx_len + 1 for r in batch.rows)
    chunk_keys = sum(c.offset + c.len for c in batch.chunks)       # each chunk reads its keys once
    kv_per_key = 2 * kvd * es
    n_lm = D + sum(1 for c in getattr(batch, "gen_chunks", None) or [] if c.last)
    classes = {
        "gather_norm": (0.0, T * d * (es + 4 + es)),
        "gemm_qkv_rope": (2.0 * T * d * qkv * L, (d * qkv * es + T * d * es + T * qd * es + T * kv_per_key) * L),
        "attention": (4.0 * pairs * cfg.head_dim * cfg.n_q_heads * L,
                      ((dec_keys + chunk_keys) * kv_per_key + 2 * T * qd * es) * L),
        "gemm_o": (2.0 * T * qd * d * L, (qd * d * es + T * qd * es + 2 * T * d * 4) * L),
        "rmsnorm": (0.0, T * d * (4 + es) * (2 * L - 1)),
        "gemm_gate_up": (2.0 * T * d * 2 * F * L, (2 * F * d * es + T * d * es + T * F * es) * L),
        "gemm_down": (2.0 * T * F * d * L, (F * d * es + T * F * es + 2 * T * d * 4) * L),
        "final_norm_pool": (0.0, (n_lm + len(batch.chunks)) * d * (4 + es)),
        "lm_head": (2.0 * n_lm * d * V, d * V * es + n_lm * d * es + n_lm * V * 4),
    }
    ideal_s = sum(max(f / (PEAK_BF16_TFLOPS * 1e12), b / (PEAK_HBM_GBS * 1e9)) for f, b in classes.values())
    return ideal_s * 1e3, ideal_s * 1e3 / t_step_ms


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0, help="BLAS threads for the oracle (0 = all)")
    ap.add_argument("--workload", default="7b-layer-mixed",
                    choices=["7b-layer-mixed", "retrieval-sweep-32l", "long-docs-32l", "decode-heavy-32l",
                             "serving-32l"],
                    help="7b-layer-mixed (default): the headline one-layer step with roofline and CPU "
                         "baseline.  The others run the full 32-layer configurations on device-drawn "
                         "weights and caches: two models over an embedding-fraction sweep, 16 documents "
                         "of 8192 tokens chunked by 512 next to 32 decode rows, and 256 decode rows at "
                         "contexts 4096-8192 next to 8 short queries")
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
    if args.workload != "7b-layer-mixed":
        print(json.dumps(full_model_bench(args)), flush=True)
        return 0

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
    ideal_ms, frac = step_roofline(cfg, batch, ms)
    result["step_roofline"] = {"ideal_ms": ideal_ms, "frac": frac,
                               "definition": "sum over kernel classes of max(algorithmic flops / 2.5 PFLOP/s, "
                                             "least HBM bytes / 8 TB/s), divided by the measured step time"}
    # the decode rows alone (no chunk tiles in the attention launch): HBM figure of the decode
    # attention without the chunk tiles that share its CUs in the mixed step
    from workload import Batch
    dec_batch = Batch([], batch.rows, batch.token_ids[Te:])
    dec_packed = R.PackedBatch(dec_batch)
    for _ in range(3):
        R.step(dm, dm, dec_batch, kv, kv, acc_sum, acc_w, logits, out_emb, ws, packed=dec_packed)
    R.profile_begin(dm)
    for _ in range(20):
        R.step(dm, dm, dec_batch, kv, kv, acc_sum, acc_w, logits, out_emb, ws, packed=dec_packed)
    prof_dec = R.profile_end(dm)
    torch.cuda.synchronize()
    assert ws.device_error() == 0, "device error during the decode-only pass"
    n_a, tot_a = prof_dec["attention"]
    dec_bytes = algorithmic_work(cfg, dec_batch)["attention"][1]
    result["attention_decode_only"] = {"avg_ms": tot_a / n_a, "gbs": dec_bytes / (tot_a / n_a * 1e-3) / 1e9,
                                       "frac_hbm": dec_bytes / (tot_a / n_a * 1e-3) / 1e9 / PEAK_HBM_GBS}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_threads)
    print(json.dumps(result), flush=True)
    return 0


def full_model_bench(args) -> dict:
    """The 32-layer configurations: seeded weights and caches drawn on the device (their host
    images would not fit), batches from the workload module's scenario generators.  Parity at
    these sizes is covered by the one-layer tests of the same kernels; no CPU baseline here (the
    float64 oracle would take hours per step)."""
    import numpy as np
    import torch

    from paper_2609_25405_amd import runtime as R
    from workload import (decode_heavy_scenario, device_weights, fill_device_pools, llm7b_config,
                          long_document_scenario, retrieval_mix_scenario)

    L = 32

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    def device_kv(cfg, n_pages, n_seq, max_blocks, block_table, seed):
        need = 2 * cfg.n_layers * n_pages * cfg.n_kv_heads * cfg.page_size * cfg.head_dim * 2
        free = torch.cuda.mem_get_info()[0]
        if need > 0.9 * free:
            raise SystemExit(f"cache of {need / 2**30:.1f} GiB does not fit ({free / 2**30:.1f} GiB free)")
        kv = R.DeviceKV(cfg, n_pages, n_seq, max_blocks, fill=0.0)
        kv.set_block_table(block_table)
        fill_device_pools(kv.k, kv.v, seed)
        torch.cuda.synchronize()
        log(f"cache {need / 2**30:.1f} GiB drawn")
        return kv

    def model(cfg, seed, tag):
        W = device_weights(cfg, seed, tag)
        torch.cuda.synchronize()
        dm = R.DeviceModel(cfg, W)
        del W
        log(f"model (tag {tag}) drawn: {cfg.n_layers} layers")
        return dm

    def time_steps(dm_e, dm_g, kv_e, kv_g, batches, ws, n_seq_e, repeat):
        """Each batch run `repeat` times back to back (a repeated step rewrites the same cache
        slots and restarts its offset-0 chunks, so every repetition is a valid step)."""
        acc_sum = torch.zeros((n_seq_e, dm_e.cfg.d_model), device="cuda")
        acc_w = torch.zeros(n_seq_e, device="cuda")
        D_max = max(b.n_logit_rows for b in batches)
        logits = torch.empty((max(1, D_max), dm_g.cfg.vocab), device="cuda")
        out_emb = torch.empty((max(1, max(len(b.chunks) for b in batches)), dm_e.cfg.d_model), device="cuda")
        packed = [R.PackedBatch(b) for b in batches]
        times = []
        for b, pb in zip(batches, packed):
            st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            st.record()
            for _ in range(repeat):
                R.step(dm_e, dm_g, b, kv_e, kv_g, acc_sum, acc_w, logits, out_emb, ws, packed=pb)
            en.record()
            torch.cuda.synchronize()
            times.append(st.elapsed_time(en) / repeat)
        assert ws.device_error() == 0, "device error"
        return times

    def attention_gbs(dm, kv_e, kv_g, batch, ws, n_seq_e):
        acc_sum = torch.zeros((n_seq_e, dm.cfg.d_model), device="cuda")
        acc_w = torch.zeros(n_seq_e, device="cuda")
        logits = torch.empty((max(1, batch.n_logit_rows), dm.cfg.vocab), device="cuda")
        out_emb = torch.empty((max(1, len(batch.chunks)), dm.cfg.d_model), device="cuda")
        R.profile_begin(dm)
        R.step(dm, dm, batch, kv_e, kv_g, acc_sum, acc_w, logits, out_emb, ws)
        prof = R.profile_end(dm)
        n, tot = prof["attention"]
        per_launch = algorithmic_work(dm.cfg, batch)["attention"][1]
        return per_launch / (tot / n * 1e-3) / 1e9, {k: round(v[1] / v[0] * 1e3, 1) for k, v in prof.items()}

    rep = max(1, args.steps // 4)
    base = {"metric": METRIC, "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded N(0,0.02) weights and N(0,1) bf16 caches drawn on the device, "
                    "uniform token ids)"}
    if args.workload == "decode-heavy-32l":
        _, _, batch, rec = decode_heavy_scenario(n_layers=1)
        cfg = llm7b_config(n_layers=L)
        dm = model(cfg, rec.seed, 0)
        kv = device_kv(cfg, rec.n_pages, rec.n_seq, rec.max_blocks, rec.block_table, rec.seed)
        ws = R.Workspace(dm, dm, batch.n_tokens, len(batch.chunks), len(batch.rows), 8192)
        time_steps(dm, dm, kv, kv, [batch], ws, rec.n_seq, 2)
        (ms,) = time_steps(dm, dm, kv, kv, [batch], ws, rec.n_seq, rep)
        gbs, kern = attention_gbs(dm, kv, kv, batch, ws, rec.n_seq)
        Te, D = batch.n_emb_tokens, len(batch.rows)
        return dict(base, value=(Te + D) / (ms * 1e-3), steps=rep, warmup=2, ms_per_step=ms,
                    config={"workload": "decode-heavy-32l: 32 layers 7B shape bf16 vocab 32000; 256 decode "
                                        "rows ctx U[4096,8192] + 8 queries x16 tokens (mean pooling), page 16",
                            "embed_tokens": Te, "decode_tokens": D, "layers": L},
                    embed_tokens_per_s=Te / (ms * 1e-3), decode_tokens_per_s=D / (ms * 1e-3),
                    attention_gbs=gbs, attention_frac_hbm=gbs / PEAK_HBM_GBS, kernel_avg_us=kern)
    if args.workload == "retrieval-sweep-32l":
        cfg_e1, _, cfg_g1, _, paged_e, paged_g, steps = retrieval_mix_scenario(n_layers=1)
        cfg_e, cfg_g = llm7b_config(n_layers=L, has_lm_head=False), llm7b_config(n_layers=L)
        dm_e, dm_g = model(cfg_e, 1003, 1), model(cfg_g, 1003, 2)
        kv_e = device_kv(cfg_e, paged_e.n_pages, paged_e.n_seq, paged_e.max_blocks, paged_e.block_table, 1)
        kv_g = device_kv(cfg_g, paged_g.n_pages, paged_g.n_seq, paged_g.max_blocks, paged_g.block_table, 2)
        ws = R.Workspace(dm_e, dm_g, max(b.n_tokens for b in steps), max(1, max(len(b.chunks) for b in steps)),
                         max(len(b.rows) for b in steps), 4096)
        time_steps(dm_e, dm_g, kv_e, kv_g, steps, ws, paged_e.n_seq, 1)
        times = time_steps(dm_e, dm_g, kv_e, kv_g, steps, ws, paged_e.n_seq, rep)
        sweep = []
        for f, b, t in zip((0.0, 0.25, 0.5, 0.75, 1.0), steps, times):
            sweep.append({"embedding_fraction": f, "embed_tokens": b.n_emb_tokens, "decode_rows": len(b.rows),
                          "ms_per_step": t, "tokens_per_s": (b.n_emb_tokens + len(b.rows)) / (t * 1e-3)})
        tok = sum(b.n_emb_tokens + len(b.rows) for b in steps)
        ms = sum(times) / len(times)
        return dict(base, value=tok / (sum(times) * 1e-3), steps=rep * len(steps), warmup=len(steps),
                    ms_per_step=ms,
                    config={"workload": "retrieval-sweep-32l: two 32-layer 7B-shape models (embedding: mean "
                                        "pooling, no LM head; generator: vocab 32000), 2048-token budget, "
                                        "embedding fraction 0/.25/.5/.75/1, queries lognormal mean 64, up to "
                                        "256 decode rows with contexts lognormal mean 512",
                            "layers": L},
                    embed_tokens_per_s=sum(b.n_emb_tokens for b in steps) / (sum(times) * 1e-3),
                    decode_tokens_per_s=sum(len(b.rows) for b in steps) / (sum(times) * 1e-3),
                    sweep=sweep)
    if args.workload == "serving-32l":
        return serving_bench(args, model, log, L)
    # long documents
    _, _, paged, steps = long_document_scenario(n_layers=1, n_docs=16, doc_len=8192, chunk=512, per_step=3,
                                                n_dec=32, ctx0=2048)
    cfg = llm7b_config(n_layers=L)
    dm = model(cfg, 1004, 0)
    kv = device_kv(cfg, paged.n_pages, paged.n_seq, paged.max_blocks, paged.block_table, 4)
    ws = R.Workspace(dm, dm, max(b.n_tokens for b in steps), 3, 32, paged.max_blocks * 16)
    time_steps(dm, dm, kv, kv, steps[:1], ws, paged.n_seq, 2)
    times = time_steps(dm, dm, kv, kv, steps, ws, paged.n_seq, 1)
    Te = sum(b.n_emb_tokens for b in steps)
    D = sum(len(b.rows) for b in steps)
    tsum = sum(times) * 1e-3
    return dict(base, value=(Te + D) / tsum, steps=len(steps), warmup=2, ms_per_step=sum(times) / len(times),
                config={"workload": "long-docs-32l: 32 layers 7B shape bf16 vocab 32000; 16 documents x8192 "
                                    "tokens chunked by 512 (mean pooling), 3 chunks per step, + 32 decode rows "
                                    "from context 2048", "layers": L, "steps": len(steps)},
                embed_tokens_per_s=Te / tsum, decode_tokens_per_s=D / tsum,
                ms_per_step_first_last=[times[0], times[-1]])


def serving_bench(args, model, log, L: int) -> dict:
    """The serving loop on the GPU: the native intra-batch scheduler and the runner (schedule,
    step, sample, commit; one host synchronisation per iteration) serve a closed set of
    requests to completion on a 32-layer 7B-shape model.  Value: every token the model processed
    (embedding inputs, prompts, generated tokens) per second of wall time.  The run length is
    the request set's (244 iterations), so --steps and --warmup do not apply: one short
    embedding and one short generation go through a scheduler of their own first, untimed."""
    import numpy as np
    import torch

    from paper_2609_25405_amd import runtime as R
    from workload import llm7b_config

    cfg = llm7b_config(n_layers=L)
    dm = model(cfg, 1005, 0)
    rng = np.random.default_rng(1005)
    n_emb, n_gen, prompt, new = 384, 96, 512, 128
    sigma = 0.6
    emb_len = np.clip(np.round(rng.lognormal(np.log(512) - sigma * sigma / 2, sigma, n_emb)), 16, 4096).astype(int)
    budget, chunk, n_seq, page = 2048, 512, 512, cfg.page_size
    max_blocks = (max(int(emb_len.max()), prompt + new) + page - 1) // page + 1
    n_pages = 16384                                   # 2 MiB per page over 32 layers: 32 GiB
    kv = R.DeviceKV(cfg, n_pages, n_seq, max_blocks, fill=0.0)
    # untimed warm-up: one embedding and one short generation through a scheduler of their own
    w_sched = R.Scheduler(budget, chunk, [(n_seq, n_pages, max_blocks)])
    w_run = R.Runner(dm, dm, kv, kv, w_sched)
    w_sched.submit_embedding(0, 600, rng.integers(0, cfg.vocab, 600).tolist(), "mean")
    w_sched.submit_generation(1, 600, 4, rng.integers(0, cfg.vocab, 600).tolist())
    for _ in range(16):
        w_run.iterate()
        c = w_sched.counts()
        if c["queued_emb"] == 0 and c["queued_gen"] == 0 and c["running"] == 0:
            break
    w_run.close()
    w_sched.close()
    del w_run, w_sched
    sched = R.Scheduler(budget, chunk, [(n_seq, n_pages, max_blocks)])
    run = R.Runner(dm, dm, kv, kv, sched)
    rid = 0
    for i in range(max(n_emb, n_gen)):                # interleaved arrivals, all at time 0
        if i < n_gen:
            sched.submit_generation(rid, prompt, new, rng.integers(0, cfg.vocab, prompt).tolist())
            rid += 1
        if i < n_emb:
            n = int(emb_len[i])
            sched.submit_embedding(rid, n, rng.integers(0, cfg.vocab, n).tolist(), "mean")
            rid += 1
    log(f"serving: {n_emb} embedding requests ({int(emb_len.sum())} tokens), {n_gen} generations "
        f"({prompt}-token prompts, {new} new tokens)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    it, used, gen_tokens, n_embs, fills, iter_s = 0, 0, 0, 0, [], []
    while True:
        t1 = time.perf_counter()
        out = run.iterate()                           # synchronises the stream
        iter_s.append(time.perf_counter() - t1)
        it += 1
        used += out["used"]
        fills.append(out["used"] / budget)
        gen_tokens += len(out["tokens"])
        n_embs += len(out["embeddings"])
        c = sched.counts()
        if c["queued_emb"] == 0 and c["queued_gen"] == 0 and c["running"] == 0:
            break
        if it >= 2000:
            raise SystemExit("serving run did not drain in 2000 iterations")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert n_embs == n_emb, (n_embs, n_emb)
    emb_tokens, prompt_tokens = int(emb_len.sum()), n_gen * prompt
    processed = emb_tokens + prompt_tokens + n_gen * (new - 1)   # the last sampled token is never fed back
    return {"metric": METRIC, "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded N(0,0.02) weights drawn on the device, uniform token ids)",
            "value": processed / wall, "steps": it, "warmup": 1, "ms_per_step": wall / it * 1e3,
            "config": {"workload": "serving-32l: 32 layers 7B shape bf16 vocab 32000; native scheduler (budget "
                                   "2048, chunk 512) and runner serve 384 embedding requests (lognormal lengths, "
                                   "mean 512, mean pooling) and 96 generations (512-token prompts, 128 new tokens, "
                                   "greedy) to completion, one synchronisation per iteration",
                       "layers": L},
            "embed_tokens_per_s": emb_tokens / wall, "prompt_tokens_per_s": prompt_tokens / wall,
            "generated_tokens_per_s": n_gen * new / wall, "iterations": it,
            "mean_budget_fill": float(np.mean(fills)), "budget_tokens_used": used,
            "full_budget_iterations": int(sum(f >= 1.0 for f in fills)),
            "full_budget_ms_mean": float(np.mean([t for t, f in zip(iter_s, fills) if f >= 1.0] or [0])) * 1e3,
            "decode_only_iterations": int(sum(f * budget <= n_gen for f in fills)),
            "decode_only_ms_mean": float(np.mean([t for t, f in zip(iter_s, fills) if f * budget <= n_gen]
                                                 or [0])) * 1e3}


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
