#!/usr/bin/env python3
"""Throughput of the mixed embedding-chunk + decode step on one MI355X.

Default workload (the largest configuration that fits one GPU): two resident 32-layer 7B-shape
models in bf16 (hidden 4096, 32 query heads sharing 8 KV heads of 128, SwiGLU 14336): an
embedding model (mean pooling, L2-normalised output, no LM head) and a generator (vocab 32000).
One step holds half of a 2048-token budget in embedding-query chunks (lengths lognormal with
mean 64, single final chunks) and 256 decode rows of generation requests (contexts lognormal
with mean 512, 16-token pages).  Weights N(0, 0.02) and caches N(0, 1) are drawn on the device
from seeds, token ids uniform: all synthetic.

A step is one orthrus_step call over that batch (every kernel of the path, both models).  The
same step is repeated: the queries restart at offset 0 and the decode rows rewrite their own
slot, so every repetition is a valid step.

Prints one JSON line.  `value` = (embedding tokens + decode tokens) per second of step time,
inputs resident in HBM.  `kernels` gives every launch class's average time (HIP events around
each launch on the stream it runs on, in steps of their own after the timed ones: those events
shift how the two models' streams overlap) against its own roofline: algorithmic flops against
bf16 MFMA peak or algorithmic bytes against HBM peak, whichever bounds it.  `roofline` describes
the kernel with the largest share of the step, timed by event pairs around its launches inside
the timed steps (no events on any other launch there).  `cpu_baseline` times the float64 CPU oracle on a
sample of the same step (see cpu_baseline_sample), with its embedding and decode tokens/s and the
GPU/CPU ratio.  Extra keys: the same two models over an embedding-fraction sweep (`sweep`), the
dominant kernel's launches with the embedding rows alone (`dominant_alone`: no generator launches
sharing the CUs), the one-7B-layer mixed step (`layer7b`), and a plain 1 GiB device copy's rate
(`copy_ceiling`, a practical HBM ceiling, not a target).
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
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_25405_amd", "csrc", f) for f in ("gemm.hip", "common.hpp")]
DATA = "synthetic (seeded N(0,0.02) weights and N(0,1) bf16 caches drawn on the device, uniform token ids)"
GEMMS = ("gemm_qkv", "gemm_qkv_rope", "gemm_o", "gemm_gate_up", "gemm_down", "lm_head")


def kernel_source_hash() -> str:
    """SHA-256 of the GEMM kernel's sources with comments and whitespace removed: a change of
    code invalidates a committed counter summary, a change of comments does not."""
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


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` in `workload` from a committed rocprofv3 counter summary
    (profiles/*_traffic.md), or None when there is none for that pair or the GEMM sources changed
    since it was taken."""
    if not os.path.isdir(PROFILES):
        return None
    for fn in sorted(os.listdir(PROFILES)):
        if not fn.endswith("_traffic.md"):
            continue
        kv = {}
        try:
            with open(os.path.join(PROFILES, fn)) as f:
                for line in f:
                    if ":" in line and line.startswith("- "):
                        k, v = line[2:].split(":", 1)
                        kv[k.strip()] = v.strip()
        except OSError:
            continue
        if kv.get("step_kernel") == kernel and kv.get("workload") == workload:
            if kv.get("source_sha256") != kernel_source_hash():
                return None
            try:
                return float(kv["traffic_bytes_per_launch"])
            except (KeyError, ValueError):
                return None
    return None


# ------------------------------------------------------------------------------ work per launch
def group_rows(batch, two_models: bool):
    """Rows of each profile tag: '' (the embedding model's rows, or all rows with one model) and
    '@gen' (the generator's rows of a two-model step)."""
    T, Te = batch.n_tokens, batch.n_emb_tokens
    return {"": Te, "@gen": T - Te} if two_models else {"": T}


def launch_work(cfg, batch, two_models: bool):
    """Algorithmic work of every profiled launch name: {name: (flops, bytes)} per launch.

    What the method must compute or move, not what the kernels execute: GEMMs 2 M K N flops over
    their weights, input rows and output rows (residual-add projections read and write the fp32
    residual rows once); attention 4 hd nq flops per (query, visible key) pair of chunk rows and
    decode rows, over every visible key's K and V once per KV head plus q and o; norms and the
    final norm / pooler over their rows.  Split-K slabs, attention partials and the fp32 rows of
    the unfused rotation path are implementation traffic: rope_append and attn_combine carry no
    algorithmic work (their work is counted in gemm_qkv and attention)."""
    d, F, V, L = cfg.d_model, cfg.d_ff, cfg.vocab, cfg.n_layers
    qd, kvd, qkv = cfg.q_dim, cfg.kv_dim, cfg.qkv_dim
    es = 2 if cfg.dtype == "bf16" else 4
    T = batch.n_tokens
    work = {}
    for tag, M in group_rows(batch, two_models).items():
        if M == 0:
            continue
        work["gather_norm" + tag] = (0.0, M * d * (es + 4 + es))
        work["rmsnorm" + tag] = (0.0, M * d * (4 + es))
        qkv_w = (2.0 * M * d * qkv, d * qkv * es + M * d * es + M * qd * es + M * 2 * kvd * es)
        work["gemm_qkv_rope" + tag] = qkv_w
        work["gemm_qkv" + tag] = qkv_w
        work["gemm_o" + tag] = (2.0 * M * qd * d, qd * d * es + M * qd * es + 2 * M * d * 4)
        work["gemm_gate_up" + tag] = (2.0 * M * d * 2 * F, 2 * F * d * es + M * d * es + M * F * es)
        work["gemm_down" + tag] = (2.0 * M * F * d, F * d * es + M * F * es + 2 * M * d * 4)
    kv_per_key = 2 * kvd * es

    def attention(chunks, rows, n_tok):
        pairs = sum(sum(c.offset + i + 1 for i in range(c.len)) for c in chunks)
        dec_keys = sum(r.ctx_len + 1 for r in rows)
        chunk_keys = sum(c.offset + c.len for c in chunks)
        return (4.0 * (pairs + dec_keys) * cfg.head_dim * cfg.n_q_heads,
                (dec_keys + chunk_keys) * kv_per_key + 2 * n_tok * qd * es)

    gen_chunks = list(getattr(batch, "gen_chunks", None) or [])
    if two_models:
        # one attention launch per model: the embedding chunks; the prompt chunks and decode rows
        Te = batch.n_emb_tokens
        work["attention"] = attention(batch.chunks, [], Te)
        work["attention@gen"] = attention(gen_chunks, batch.rows, T - Te)
        work["rope_append@gen"] = (0.0, 0.0)
        work["attn_combine@gen"] = (0.0, 0.0)
    else:
        work["attention"] = attention(list(batch.chunks) + gen_chunks, batch.rows, T)
    work["rope_append"] = (0.0, 0.0)
    work["attn_combine"] = (0.0, 0.0)
    n_lm = batch.n_logit_rows
    final = batch.n_emb_tokens * d * 4 + n_lm * d * (4 + es) + len(batch.chunks) * d * 4 * 3
    work["final_norm_pool"] = (0.0, final)
    work["final_norm"] = (0.0, final)
    work["pool"] = (0.0, 0.0)
    if n_lm:
        work["lm_head"] = (2.0 * n_lm * d * V, d * V * es + n_lm * d * es + n_lm * V * 4)
    return work


def decode_kv_bytes(cfg, batch) -> float:
    """Keys and values the decode rows must read per layer (every visible key once per KV head)."""
    es = 2 if cfg.dtype == "bf16" else 4
    return 2.0 * sum(r.ctx_len + 1 for r in batch.rows) * cfg.kv_dim * es


def kernel_table(cfg, batch, two_models: bool, prof: dict, steps: int):
    """Per launch name: launches per step, average ms, and the launch against its roofline."""
    work = launch_work(cfg, batch, two_models)
    out = {}
    for name, (n, tot) in prof.items():
        avg = tot / max(n, 1)
        ent = {"launches_per_step": n / steps, "avg_ms": avg}
        if name in work and any(work[name]):
            f, b = work[name]
            t_f, t_b = f / (PEAK_BF16_TFLOPS * 1e12), b / (PEAK_HBM_GBS * 1e9)
            ent["bound"] = "mfma" if t_f >= t_b else "hbm"
            if ent["bound"] == "mfma":
                ent["tflops"] = f / (avg * 1e-3) / 1e12
            else:
                ent["gbs"] = b / (avg * 1e-3) / 1e9
            ent["frac"] = max(t_f, t_b) / (avg * 1e-3)
            ent["algorithmic_flop"], ent["algorithmic_bytes"] = f, b
        out[name] = ent
    return out


def dominant_kernel(cfg, batch, two_models: bool, prof: dict, steps: int) -> str:
    """The launch name with the largest share of the profiled steps' kernel time."""
    kernels = kernel_table(cfg, batch, two_models, prof, steps)
    return max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches_per_step"])


def summarize(cfg, batch, two_models: bool, ms: float, prof: dict, steps: int, workload: str,
              dom_timed=None) -> dict:
    """tokens/s, the kernel table, the MFMA fraction of the MFMA-bound GEMMs, the HBM fraction
    of the decode attention, the dominant kernel's roofline and the step roofline.  `dom_timed`
    = (name, launches, total ms) of the dominant kernel timed by events inside the timed steps;
    without it the roofline takes the dominant kernel's time from the profiled steps."""
    kernels = kernel_table(cfg, batch, two_models, prof, steps)
    Te, T, D = batch.n_emb_tokens, batch.n_tokens, len(batch.rows)
    work = launch_work(cfg, batch, two_models)
    f_m = t_m = b_h = t_h = 0.0
    for name, e in kernels.items():
        if name.split("@")[0] in GEMMS and "bound" in e:
            t = e["avg_ms"] * e["launches_per_step"]
            if e["bound"] == "mfma":
                f_m += e["algorithmic_flop"] * e["launches_per_step"]
                t_m += t
            else:
                b_h += e["algorithmic_bytes"] * e["launches_per_step"]
                t_h += t
    attn = kernels.get("attention@gen" if two_models else "attention")
    res = {
        "ms_per_step": ms,
        "value": T / (ms * 1e-3),
        "embed_tokens_per_s": Te / (ms * 1e-3),
        "decode_tokens_per_s": D / (ms * 1e-3),
        "gemm_frac_mfma": f_m / (t_m * 1e-3) / 1e12 / PEAK_BF16_TFLOPS if t_m else None,
        "gemm_hbm_bound_frac_hbm": b_h / (t_h * 1e-3) / 1e9 / PEAK_HBM_GBS if t_h else None,
        "attention_frac_hbm": (decode_kv_bytes(cfg, batch) / (attn["avg_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS
                               if attn and batch.rows else None),
        "attention_roofline_frac": attn.get("frac") if attn else None,   # the decode rows' launch
    }
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches_per_step"])
    dk = kernels[dom]
    f, b = work.get(dom, (0.0, 0.0))
    avg, timing = dk["avg_ms"], "HIP events around every launch, in separately profiled steps"
    if dom_timed is not None and dom_timed[0] == dom and dom_timed[1] > 0:
        avg = dom_timed[2] / dom_timed[1]
        timing = (f"HIP events around each of its {dom_timed[1]} launches inside the timed steps "
                  "(on its stream; no events on other launches)")
    if dk.get("bound") == "mfma":
        ach = f / (avg * 1e-3) / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": measured_traffic(dom, workload),
                "algorithmic_per_launch": f, "algorithmic_bytes_per_launch": b, "avg_launch_ms": avg,
                "timing": timing}
    else:
        ach = b / (avg * 1e-3) / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": measured_traffic(dom, workload),
                "algorithmic_per_launch": b, "avg_launch_ms": avg, "timing": timing}
    res["roofline"] = roof
    res["kernels"] = kernels
    ideal = sum(max(w[0] / (PEAK_BF16_TFLOPS * 1e12), w[1] / (PEAK_HBM_GBS * 1e9)) * kernels[k]["launches_per_step"]
                for k, w in work.items() if k in kernels)
    res["step_roofline"] = {"ideal_ms": ideal * 1e3, "frac": ideal * 1e3 / ms,
                            "definition": "sum over the step's launches of max(algorithmic flops / 2.5 PFLOP/s, "
                                          "algorithmic bytes / 8 TB/s), divided by the measured step time"}
    return res


# ------------------------------------------------------------------------------ device set-up
def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def device_model(cfg, seed, tag):
    import torch
    from paper_2609_25405_amd import runtime as R
    from workload import device_weights
    W = device_weights(cfg, seed, tag)
    torch.cuda.synchronize()
    dm = R.DeviceModel(cfg, W)
    log(f"model (tag {tag}) drawn: {cfg.n_layers} layers")
    return dm, W


def device_kv(cfg, n_pages, n_seq, max_blocks, block_table, seed):
    import torch
    from paper_2609_25405_amd import runtime as R
    from workload import fill_device_pools
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


class Stepper:
    """Repeats one batch through orthrus_step with fixed output buffers; `reset` restores what a
    repetition must find (e.g. a resuming request's token count) before each step."""

    def __init__(self, dm_e, dm_g, kv_e, kv_g, batch, ws, n_seq_e, acc_w0=None):
        import torch
        from paper_2609_25405_amd import runtime as R
        self.R = R
        self.args = (dm_e, dm_g, kv_e, kv_g)
        self.batch, self.ws = batch, ws
        d = dm_e.cfg.d_model
        self.acc_sum = torch.zeros((n_seq_e, d), device="cuda")
        self.acc_w0 = (torch.zeros(n_seq_e, device="cuda") if acc_w0 is None
                       else torch.as_tensor(acc_w0, dtype=torch.float32, device="cuda"))
        self.acc_w = self.acc_w0.clone()
        self.logits = torch.empty((max(1, batch.n_logit_rows), dm_g.cfg.vocab), device="cuda")
        self.out_emb = torch.empty((max(1, len(batch.chunks)), d), device="cuda")
        self.packed = R.PackedBatch(batch)

    def __call__(self):
        dm_e, dm_g, kv_e, kv_g = self.args
        self.acc_w.copy_(self.acc_w0)
        self.R.step(dm_e, dm_g, self.batch, kv_e, kv_g, self.acc_sum, self.acc_w, self.logits, self.out_emb,
                    self.ws, packed=self.packed)

    def time(self, steps: int, warmup: int, only: str | None = None):
        """Average ms per step over `steps` steps after `warmup` untimed ones.  With `only`, the
        launches of that name inside the timed steps also carry HIP event pairs on their stream
        (two events per such launch, none on the others), and the result is (ms per step,
        (launches, total ms of those launches))."""
        import torch
        for _ in range(warmup):
            self()
        torch.cuda.synchronize()
        assert self.ws.device_error() == 0, "device error during warmup"
        dm_e = self.args[0]
        if only:
            self.R.profile_only(dm_e, only)
            self.R.profile_begin(dm_e)
        st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        st.record()
        for _ in range(steps):
            self()
        en.record()
        torch.cuda.synchronize()
        assert self.ws.device_error() == 0, "device error during timed steps"
        ms = st.elapsed_time(en) / steps
        if not only:
            return ms
        prof = self.R.profile_end(dm_e)
        self.R.profile_only(dm_e, None)
        return ms, prof.get(only, (0, 0.0))

    def warm_dominant(self, cfg, two_models: bool, warmup: int) -> str:
        """`warmup` untimed steps (at least two): the first plain (it pays the first launches'
        one-time costs), the rest with events around every launch; returns the launch name
        with the largest share of those."""
        import torch
        self()
        torch.cuda.synchronize()
        n = max(1, warmup - 1)
        return dominant_kernel(cfg, self.batch, two_models, self.profile(n), n)

    def profile(self, steps: int) -> dict:
        """Per launch name (launches, total ms) from HIP events around each launch."""
        import torch
        dm_e = self.args[0]
        self.R.profile_begin(dm_e)
        for _ in range(steps):
            self()
        prof = self.R.profile_end(dm_e)
        torch.cuda.synchronize()
        assert self.ws.device_error() == 0, "device error during the profiled steps"
        return prof


# ------------------------------------------------------------------------------ CPU baseline
def host_info() -> dict:
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}


def blas_threads(n: int):
    """Limit BLAS threads to n; returns (limiter or None, threads in use)."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        lim = threadpool_limits(limits=n)
        used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        return lim, used
    except Exception:
        return None, n


def host_layers(W, n_layers: int):
    """float64 host copies of the global tensors and the first n_layers layers of device weights."""
    import numpy as np
    f = lambda t: None if t is None else t.float().cpu().numpy().astype(np.float64)
    return {"tok_emb": f(W["tok_emb"]), "final_norm": f(W["final_norm"]), "lm_head": f(W.get("lm_head")),
            "layers": [{k: f(v) for k, v in W["layers"][l].items()} for l in range(n_layers)]}


def cpu_baseline_sample(W_e, W_g, kv_g, batch, block_table, max_blocks: int, threads: int, n_rows: int = 64,
                        layers: int = 32, emb_lm_head: bool = False, reps: int = 3) -> dict:
    """The float64 oracle on a sample of a 32-layer step, extrapolated to the whole step.

    Sample: every embedding chunk of the step (through the embedding model W_e, each run as one
    final chunk at offset 0 over its own tokens) and the first `n_rows` decode rows (through the
    generator W_g, keys and values copied from the device cache `kv_g` by `block_table`), each at
    1 and at 2 layers of the same device-drawn weights (copied to the host).  Per-layer time =
    t(2) - t(1); the whole-depth time of each part is t(1) + (layers - 1) (t(2) - t(1)) (the LM
    head and the final norm counted once), and the decode part is scaled by D / n_rows (the
    oracle runs each request alone).  Each part is timed `reps` times at each depth and its
    fastest run kept (about 10 s of CPU work in all on the two-model step).  With one model, W_e
    is W_g.  An extrapolation, stated as one in the result."""
    import numpy as np
    import torch
    from oracle import OracleKV, step_oracle
    from workload import Batch, DecodeRow, EmbChunk, llm7b_config
    n = threads or len(os.sched_getaffinity(0))
    lim, used = blas_threads(n)
    P = 16
    Te, D = batch.n_emb_tokens, len(batch.rows)
    rows = batch.rows[:n_rows]
    q = Batch([EmbChunk(i, 0, c.len, True, c.pool) for i, c in enumerate(batch.chunks)], [],
              batch.token_ids[:Te])
    r = Batch([], [DecodeRow(i, x.ctx_len) for i, x in enumerate(rows)], batch.token_ids[Te:Te + len(rows)])
    pages = [block_table[x.seq][:-(-(x.ctx_len + 1) // P)] for x in rows]
    flat = torch.from_numpy(np.concatenate(pages).astype(np.int64)).to(kv_g.k.device)
    bt = np.full((len(rows), max_blocks), -1, np.int64)
    o = 0
    for i, p in enumerate(pages):
        bt[i, :len(p)] = np.arange(o, o + len(p))
        o += len(p)
    q_pages = sum(-(-c.len // P) for c in batch.chunks)
    q_bt = np.full((len(batch.chunks), max(-(-c.len // P) for c in batch.chunks) if batch.chunks else 1), -1,
                   np.int64)
    o = 0
    for i, c in enumerate(batch.chunks):
        k = -(-c.len // P)
        q_bt[i, :k] = np.arange(o, o + k)
        o += k
    times = {}
    for L in (1, 2):
        cfg_e = llm7b_config(n_layers=L, has_lm_head=emb_lm_head)
        cfg_g = llm7b_config(n_layers=L)
        We = host_layers(W_e, L)
        Wg = We if W_g is W_e else host_layers(W_g, L)
        k64 = kv_g.k[:L, flat].float().cpu().numpy().astype(np.float64)
        v64 = kv_g.v_by_position[:L, flat].float().cpu().numpy().astype(np.float64)
        okv_g = OracleKV(k64, v64, bt, P, bf16=True)
        shape = (L, max(q_pages, 1), cfg_e.n_kv_heads, P, cfg_e.head_dim)
        okv_e = OracleKV(np.zeros(shape), np.zeros(shape), q_bt, P, bf16=True)
        n_q = max(1, len(batch.chunks))
        tq, tr = float("inf"), float("inf")
        for _ in range(reps):
            t0 = time.perf_counter()
            if batch.chunks:
                step_oracle((cfg_e, We), (cfg_g, Wg), q, okv_e, okv_g, np.zeros((n_q, cfg_e.d_model)), np.zeros(n_q))
            t1 = time.perf_counter()
            step_oracle((cfg_e, We), (cfg_g, Wg), r, okv_e, okv_g, np.zeros((n_q, cfg_e.d_model)), np.zeros(n_q))
            t2 = time.perf_counter()
            tq, tr = min(tq, t1 - t0), min(tr, t2 - t1)
        times[L] = (tq, tr)
        del We, Wg, okv_g, okv_e, k64, v64
    (q1, r1), (q2, r2) = times[1], times[2]
    t_q = q1 + (layers - 1) * (q2 - q1)
    t_r = (r1 + (layers - 1) * (r2 - r1)) * D / len(rows)
    if lim is not None:
        lim.restore_original_limits()
    return {"value": (Te + D) / (t_q + t_r), "unit": "tokens/s", "cores": used, "kind": "oracle",
            "embed_tokens_per_s": Te / (t_q + t_r), "decode_tokens_per_s": D / (t_q + t_r),
            "seconds_per_step": t_q + t_r,
            "sample": f"float64 oracle on the same step's {len(batch.chunks)} embedding chunks ({Te} tokens) and "
                      f"{len(rows)} of its {D} decode rows, each at 1 and 2 layers of the same weights, fastest "
                      f"of {reps} runs (chunks {q1:.2f} / {q2:.2f} s, rows {r1:.2f} / {r2:.2f} s); extrapolated to {layers} "
                      f"layers as t1 + {layers - 1} (t2 - t1) and to all {D} rows: {t_q + t_r:.1f} s per step",
            "extrapolated": True, **host_info()}


def cpu_baseline_step(wl, threads: int, min_seconds: float = 10.0) -> dict:
    """The float64 oracle on a whole one-layer step, repeated to about `min_seconds`."""
    from oracle import OracleKV, step_oracle
    from workload import as_float64
    n = threads or len(os.sched_getaffinity(0))
    lim, used = blas_threads(n)
    okv = OracleKV.from_paged(wl.kv)
    W64 = as_float64(wl.weights)
    reps, t0 = 0, time.time()
    while reps == 0 or time.time() - t0 < min_seconds:
        step_oracle((wl.cfg, W64), (wl.cfg, W64), wl.batch, okv, okv, wl.acc_sum, wl.acc_w)
        reps += 1
    dt = (time.time() - t0) / reps
    if lim is not None:
        lim.restore_original_limits()
    T = wl.batch.n_tokens
    return {"value": T / dt, "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": f"{reps} full steps of the same workload ({T} tokens each), float64 NumPy, {dt:.2f} s per step",
            **host_info()}


# ------------------------------------------------------------------------------ workloads
TWO_MODELS = ("two-models-32l: two resident 32-layer 7B-shape bf16 models (embedding: mean pooling, no LM "
              "head; generator: vocab 32000), 2048-token budget at embedding fraction 0.5: {nq} query "
              "chunks (lognormal mean 64, {te} tokens) + {d} decode rows (contexts lognormal mean 512), page 16")
LAYER7B = ("7b-layer-mixed-2048: 1 layer d4096 32q/8kv x128 ffn14336 vocab32000 bf16; 2 chunks x512 (offsets 0 "
           "and 1536, last-token pooling) + 64 decode rows ctx U[1024,4096], page 16")


def two_models_bench(args, layers: int = 32) -> dict:
    """The headline: both models at embedding fraction 0.5, with the fraction sweep as extras."""
    import torch
    from paper_2609_25405_amd import runtime as R
    from workload import llm7b_config, retrieval_mix_scenario
    _, _, _, _, paged_e, paged_g, steps = retrieval_mix_scenario(n_layers=1)
    cfg_e, cfg_g = llm7b_config(n_layers=layers, has_lm_head=False), llm7b_config(n_layers=layers)
    dm_e, W_e = device_model(cfg_e, 1003, 1)
    dm_g, W_g = device_model(cfg_g, 1003, 2)
    kv_e = device_kv(cfg_e, paged_e.n_pages, paged_e.n_seq, paged_e.max_blocks, paged_e.block_table, 1)
    kv_g = device_kv(cfg_g, paged_g.n_pages, paged_g.n_seq, paged_g.max_blocks, paged_g.block_table, 2)
    ws = R.Workspace(dm_e, dm_g, max(b.n_tokens for b in steps), max(1, max(len(b.chunks) for b in steps)),
                     max(len(b.rows) for b in steps), 4096)
    batch = steps[2]
    st = Stepper(dm_e, dm_g, kv_e, kv_g, batch, ws, paged_e.n_seq)
    # the warm-up steps (after a plain first one) time every launch, naming the dominant kernel;
    # the timed steps carry events on the dominant kernel's launches only, and steps of their own
    # time every launch for the per-launch table (events around every launch shift the two
    # streams' overlap)
    dom = st.warm_dominant(cfg_g, True, args.warmup)
    ms, (n_dom, t_dom) = st.time(args.steps, 0, only=dom)
    log(f"{args.steps} steps, {ms:.3f} ms/step")
    prof = st.profile(args.steps)
    res = summarize(cfg_g, batch, True, ms, prof, args.steps, "two-models-32l", (dom, n_dom, t_dom))
    config = {"workload": TWO_MODELS.format(nq=len(batch.chunks), te=batch.n_emb_tokens, d=len(batch.rows)),
              "embed_tokens": batch.n_emb_tokens, "decode_tokens": len(batch.rows), "layers": layers,
              "models": 2}
    sweep = []
    for f, b in zip((0.0, 0.25, 0.5, 0.75, 1.0), steps):
        t = Stepper(dm_e, dm_g, kv_e, kv_g, b, ws, paged_e.n_seq).time(max(3, args.steps // 4), 2)
        sweep.append({"embedding_fraction": f, "embed_tokens": b.n_emb_tokens, "decode_rows": len(b.rows),
                      "ms_per_step": t, "tokens_per_s": b.n_tokens / (t * 1e-3)})
    res["sweep"] = sweep
    res["sweep_tokens_per_s"] = sum(b.n_tokens for b in steps) / (sum(s["ms_per_step"] for s in sweep) * 1e-3)
    try:
        res["dominant_alone"] = dominant_alone(dm_e, kv_e, batch, paged_e.n_seq, dom, max(5, args.steps // 2))
    except Exception as e:   # noqa: BLE001  (an extra: reported, not fatal to the headline)
        log(f"dominant_alone failed: {e!r}")
        res["dominant_alone"] = {"error": repr(e)}
    if not args.no_cpu_baseline:
        from workload import DeviceKVRecipe
        rec_g = DeviceKVRecipe(paged_g.n_pages, paged_g.n_seq, paged_g.max_blocks, paged_g.block_table, 2)
        res["cpu_baseline"] = cpu_baseline_sample(W_e, W_g, kv_g, batch, rec_g.block_table, rec_g.max_blocks,
                                                  args.cpu_threads)
    del st, ws, kv_e, kv_g, dm_e, dm_g, W_e, W_g
    torch.cuda.empty_cache()
    return config, res


def dominant_alone(dm_e, kv_e, batch, n_seq_e, dom: str, steps: int) -> dict:
    """The headline batch's embedding chunks alone through the embedding model (no generator
    launches beside them): HIP events around each launch of the dominant kernel in `steps`
    steps, against its roofline.  The same launches as in the headline step, without the CUs
    they share there."""
    from paper_2609_25405_amd import runtime as R
    from workload import Batch
    name = dom.split("@")[0]
    b = Batch(batch.chunks, [], batch.token_ids[:batch.n_emb_tokens])
    ws = R.Workspace(dm_e, dm_e, b.n_tokens, max(1, len(b.chunks)), 1, 4096)
    st = Stepper(dm_e, dm_e, kv_e, kv_e, b, ws, n_seq_e)
    ms, (n, tot) = st.time(steps, 2, only=name)
    flop, byts = launch_work(dm_e.cfg, b, False).get(name, (0.0, 0.0))
    avg = tot / max(1, n)
    out = {"kernel": name, "launches": n, "avg_launch_ms": avg, "step_ms": ms,
           "what": "the headline batch's embedding chunks through the embedding model alone; HIP events "
                   "around each launch of the kernel"}
    if flop > 0 and avg > 0:
        out.update(achieved=flop / (avg * 1e-3) / 1e12, unit="TFLOP/s", frac=flop / (avg * 1e-3) / 1e12 / PEAK_BF16_TFLOPS)
    del st, ws
    return out


def layer7b_bench(args, with_cpu: bool) -> dict:
    """The one-7B-layer mixed step (device-drawn weights and caches) with a decode-only pass."""
    import torch
    from paper_2609_25405_amd import runtime as R
    from workload import Batch, layer7b_mixed_workload
    wl = layer7b_mixed_workload(with_pools=False, weights={})
    cfg, batch = wl.cfg, wl.batch
    dm, W = device_model(cfg, 1002, 0)
    kv = device_kv(cfg, wl.kv.n_pages, wl.kv.n_seq, wl.kv.max_blocks, wl.kv.block_table, 1002)
    ws = R.Workspace(dm, dm, batch.n_tokens, len(batch.chunks), len(batch.rows), 4096)
    st = Stepper(dm, dm, kv, kv, batch, ws, wl.kv.n_seq, acc_w0=wl.acc_w)
    dom = st.warm_dominant(cfg, False, args.warmup)
    ms, (n_dom, t_dom) = st.time(args.steps, 0, only=dom)
    prof = st.profile(args.steps)
    res = summarize(cfg, batch, False, ms, prof, args.steps, "7b-layer-mixed", (dom, n_dom, t_dom))
    # the decode rows alone: HBM figure of the decode attention without the chunk tiles
    dec = Batch([], batch.rows, batch.token_ids[batch.n_emb_tokens:])
    sd = Stepper(dm, dm, kv, kv, dec, ws, wl.kv.n_seq)
    sd.time(3, 3)
    n_a, tot_a = sd.profile(20)["attention"]
    gbs = decode_kv_bytes(cfg, dec) / (tot_a / n_a * 1e-3) / 1e9
    res["attention_decode_only"] = {"avg_ms": tot_a / n_a, "gbs": gbs, "frac_hbm": gbs / PEAK_HBM_GBS}
    config = {"workload": LAYER7B, "embed_tokens": batch.n_emb_tokens, "decode_tokens": len(batch.rows), "layers": 1}
    if with_cpu and not args.no_cpu_baseline:
        from workload import make_weights
        wl_host = layer7b_mixed_workload()
        res["cpu_baseline"] = cpu_baseline_step(wl_host, args.cpu_threads)
    del st, sd, ws, kv, dm, W
    torch.cuda.empty_cache()
    return config, res


def copy_ceiling() -> dict:
    """A plain 1 GiB device-to-device copy (torch): read + written bytes per second, a practical
    HBM ceiling reported beside the rooflines (not a target)."""
    import torch
    x = torch.ones(256 * 1024 * 1024, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(10):
        y.copy_(x)
    en.record()
    torch.cuda.synchronize()
    ms = st.elapsed_time(en) / 10
    del x, y
    torch.cuda.empty_cache()
    return {"gbs": 2 * (1 << 30) / (ms * 1e-3) / 1e9, "ms": ms, "what": "torch copy of 1 GiB: bytes read + written / time"}


def line(args, config: dict, res: dict, steps: int, warmup: int) -> dict:
    out = {"metric": METRIC, "value": res.pop("value"), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": res.pop("ms_per_step"), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": DATA, "config": config}
    out.update(res)
    cb = out.get("cpu_baseline")
    if cb and cb.get("value"):
        cb["gpu_over_cpu"] = out["value"] / cb["value"]
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="headline only (no one-layer figures)")
    ap.add_argument("--cpu-threads", type=int, default=0, help="BLAS threads for the oracle (0 = all)")
    ap.add_argument("--workload", default="two-models-32l",
                    choices=["two-models-32l", "7b-layer-mixed", "long-docs-32l", "decode-heavy-32l", "serving-32l"],
                    help="two-models-32l (default): both 32-layer models at embedding fraction 0.5, with the "
                         "fraction sweep and the one-layer step as extra keys.  7b-layer-mixed: one 7B layer, "
                         "1024 chunk tokens + 64 decode rows.  long-docs-32l: 16 documents of 8192 tokens "
                         "chunked by 512 next to 32 decode rows.  decode-heavy-32l: 256 decode rows at contexts "
                         "4096-8192 next to 8 short queries.  serving-32l: the scheduler and runner")
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
    if args.workload == "two-models-32l":
        config, res = two_models_bench(args)
        out = line(args, config, res, args.steps, args.warmup)
        if not args.no_extras:
            # extras: a Python-level failure in one of them is reported in its key, not allowed to
            # take the measured headline line with it
            try:
                c7, r7 = layer7b_bench(args, with_cpu=False)
                out["layer7b"] = dict(config=c7, **r7)
            except Exception as e:   # noqa: BLE001
                log(f"layer7b failed: {e!r}")
                out["layer7b"] = {"error": repr(e)}
            try:
                out["copy_ceiling"] = copy_ceiling()
            except Exception as e:   # noqa: BLE001
                log(f"copy_ceiling failed: {e!r}")
                out["copy_ceiling"] = {"error": repr(e)}
    elif args.workload == "7b-layer-mixed":
        config, res = layer7b_bench(args, with_cpu=True)
        out = line(args, config, res, args.steps, args.warmup)
    else:
        out = full_model_bench(args)
    print(json.dumps(out), flush=True)
    return 0


def full_model_bench(args) -> dict:
    """The other 32-layer configurations, on weights and caches drawn on the device."""
    import torch
    from paper_2609_25405_amd import runtime as R
    from workload import decode_heavy_scenario, llm7b_config, long_document_scenario

    L = 32
    base = {"metric": METRIC, "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": DATA}
    if args.workload == "decode-heavy-32l":
        _, _, batch, rec = decode_heavy_scenario(n_layers=1)
        cfg = llm7b_config(n_layers=L)
        dm, W = device_model(cfg, rec.seed, 0)
        kv = device_kv(cfg, rec.n_pages, rec.n_seq, rec.max_blocks, rec.block_table, rec.seed)
        ws = R.Workspace(dm, dm, batch.n_tokens, len(batch.chunks), len(batch.rows), 8192)
        st = Stepper(dm, dm, kv, kv, batch, ws, rec.n_seq)
        steps = max(1, args.steps // 4)
        dom = st.warm_dominant(cfg, False, 2)
        ms, (n_dom, t_dom) = st.time(steps, 0, only=dom)
        res = summarize(cfg, batch, False, ms, st.profile(steps), steps, "decode-heavy-32l", (dom, n_dom, t_dom))
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = cpu_baseline_sample(W, W, kv, batch, rec.block_table, rec.max_blocks,
                                                      args.cpu_threads, n_rows=16, emb_lm_head=True)
            res["cpu_baseline"]["gpu_over_cpu"] = res["value"] / res["cpu_baseline"]["value"]
        config = {"workload": "decode-heavy-32l: 32 layers 7B shape bf16 vocab 32000; 256 decode rows ctx "
                              "U[4096,8192] + 8 queries x16 tokens (mean pooling), page 16",
                  "embed_tokens": batch.n_emb_tokens, "decode_tokens": len(batch.rows), "layers": L}
        return dict(base, steps=steps, warmup=2, config=config, **res)
    if args.workload == "serving-32l":
        return serving_bench(args, L)
    # long documents: every step once, in order (each chunk's keys are written by earlier steps)
    _, _, paged, steps = long_document_scenario(n_layers=1, n_docs=16, doc_len=8192, chunk=512, per_step=3,
                                                n_dec=32, ctx0=2048)
    cfg = llm7b_config(n_layers=L)
    dm, W = device_model(cfg, 1004, 0)
    kv = device_kv(cfg, paged.n_pages, paged.n_seq, paged.max_blocks, paged.block_table, 4)
    ws = R.Workspace(dm, dm, max(b.n_tokens for b in steps), 3, 32, paged.max_blocks * 16)
    acc_sum = torch.zeros((paged.n_seq, cfg.d_model), device="cuda")
    acc_w = torch.zeros(paged.n_seq, device="cuda")
    logits = torch.empty((32, cfg.vocab), device="cuda")
    out_emb = torch.empty((3, cfg.d_model), device="cuda")
    packed = [R.PackedBatch(b) for b in steps]
    times = []
    for b, pb in zip(steps, packed):
        st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        st.record()
        R.step(dm, dm, b, kv, kv, acc_sum, acc_w, logits, out_emb, ws, packed=pb)
        en.record()
        torch.cuda.synchronize()
        times.append(st.elapsed_time(en))
    assert ws.device_error() == 0, "device error"
    Te = sum(b.n_emb_tokens for b in steps)
    D = sum(len(b.rows) for b in steps)
    tsum = sum(times) * 1e-3
    out = dict(base, value=(Te + D) / tsum, steps=len(steps), warmup=0, ms_per_step=sum(times) / len(times),
               config={"workload": "long-docs-32l: 32 layers 7B shape bf16 vocab 32000; 16 documents x8192 "
                                   "tokens chunked by 512 (mean pooling), 3 chunks per step, + 32 decode rows "
                                   "from context 2048", "layers": L, "steps": len(steps)},
               embed_tokens_per_s=Te / tsum, decode_tokens_per_s=D / tsum,
               ms_per_step_first_last=[times[0], times[-1]])
    if not args.no_cpu_baseline:
        # the first step: three 512-token chunks at offset 0 and the 32 decode rows (their keys and
        # values from the cache as it was drawn; the decode rows' own slots rewritten since)
        out["cpu_baseline"] = cpu_baseline_sample(W, W, kv, steps[0], paged.block_table, paged.max_blocks,
                                                  args.cpu_threads, n_rows=8, emb_lm_head=True)
        out["cpu_baseline"]["gpu_over_cpu"] = out["value"] / out["cpu_baseline"]["value"]
    return out


def serving_bench(args, L: int) -> dict:
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
    dm, _ = device_model(cfg, 1005, 0)
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


if __name__ == "__main__":
    sys.exit(main())
