"""GPU parity of LoRA adapters on the embedding slice against the float64 oracle.

The paper's shared-backbone deployment serves embeddings through the generator plus a LoRA
adapter.  Here embedding chunks name adapters (or the base model) chunk by chunk; the library
computes the shrink x A^T in its own kernel and adds U B^T inside each projection's GEMM
(before the rotation, the SwiGLU and the residual add).  Each case checks every output against
the oracle step by step and finished embeddings against the single-pass definition through the
same adapter; the adapters are strong enough that the base model's embedding is far off.
"""
import numpy as np
import pytest
import torch

from oracle import embed_single_pass
from tests.parity import Pair, assert_vectors_close, vec_errors
from workload import (Batch, DecodeRow, EmbChunk, ModelConfig, PagedKV, as_float64, draw_tokens,
                      layer7b_mixed_workload, make_lora, make_weights, tiny_config)
from paper_2609_25405_amd import runtime as R

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _lora_run(cfg, W, seed, lens, adapters_of, chunk, max_blocks=32, decode_ctx=(50, 90)):
    """Embedding requests of `lens` tokens, chunked by `chunk` over several steps, each through
    adapter adapters_of[i] (-1 = base), beside decode rows of the base model."""
    n_req = len(lens)
    n_seq = n_req + len(decode_ctx)
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, seed)
    for s in range(n_req):
        pk.reserve(s, lens[s])
    for i, c in enumerate(decode_ctx):
        pk.fill_random(n_req + i, c, seed + 1)
        pk.reserve(n_req + i, c + 8)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=chunk * n_req + len(decode_ctx), max_chunks=n_req,
                   max_decode=len(decode_ctx), max_ctx=max_blocks * 16)
    ids = {s: draw_tokens(seed, s, lens[s], cfg.vocab) for s in range(n_req)}
    done = {}
    off = 0
    step = 0
    while off < max(lens):
        chunks, toks, ads = [], [], []
        for s in range(n_req):
            if off < lens[s]:
                ln = min(chunk, lens[s] - off)
                chunks.append(EmbChunk(s, off, ln, off + ln == lens[s], "mean"))
                toks.append(ids[s][off:off + ln])
                ads.append(adapters_of[s])
        rows = [DecodeRow(n_req + i, c + step) for i, c in enumerate(decode_ctx)]
        toks.append(draw_tokens(seed, 100 + step, len(rows), cfg.vocab))
        ref, _, out = pair.step(Batch(chunks, rows, np.concatenate(toks).astype(np.int32),
                                      chunk_adapter=ads))
        for i, c in enumerate(chunks):
            if c.last:
                done[c.seq] = out[i].cpu().numpy()
        off += chunk
        step += 1
    return pair, ids, done


@pytest.mark.parametrize("dtype,qk_std", [("f32", None), ("bf16", 0.09)])
def test_lora_tiny_two_adapters_and_base(dtype, qk_std):
    cfg = tiny_config(dtype)
    W = make_weights(cfg, 101, qk_std=qk_std)
    W["adapters"] = [make_lora(cfg, 101, 16, tag=1), make_lora(cfg, 101, 16, tag=2, scale=1.0)]
    W64 = as_float64(W)
    lens = [150, 97, 64, 33]
    ads = [0, 1, -1, 1]
    pair, ids, done = _lora_run(cfg, W, 101, lens, ads, chunk=64)
    for s, ad in enumerate(ads):
        lora = W64["adapters"][ad] if ad >= 0 else None
        want = embed_single_pass(cfg, W64, ids[s], "mean", lora=lora)
        assert_vectors_close(done[s][None], want[None], dtype, f"request {s} vs single pass")
        if ad >= 0:
            base = embed_single_pass(cfg, W64, ids[s], "mean")
            _, cos = vec_errors(base[None], want[None])
            assert cos[0] < 0.99, "the adapter barely changes the embedding"
    print(pair.report, flush=True)


def test_lora_gqa_rank64_four_adapters():
    """Group-4 heads of 128 dims, rank 64 (qkv rank 192, gate/up 128), four adapters in one
    batch (the most a batch may hold) and a multi-split decode row."""
    cfg = ModelConfig(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                      vocab=512, dtype="bf16")
    W = make_weights(cfg, 103, qk_std=0.06)
    W["adapters"] = [make_lora(cfg, 103, 64, tag=t, std_b=0.05) for t in range(4)]
    W64 = as_float64(W)
    lens = [200, 129, 77, 40, 31]
    ads = [2, 0, 3, 1, 2]
    pair, ids, done = _lora_run(cfg, W, 103, lens, ads, chunk=96, max_blocks=80, decode_ctx=(1100,))
    for s, ad in enumerate(ads):
        want = embed_single_pass(cfg, W64, ids[s], "mean", lora=W64["adapters"][ad])
        assert_vectors_close(done[s][None], want[None], "bf16", f"request {s} vs single pass")
    print(pair.report, flush=True)


def test_lora_layer7b_mixed_step():
    """The 7B-layer mixed step (split-K O and down projections) with its two 512-token chunks
    through two rank-16 adapters."""
    wl = layer7b_mixed_workload()
    W = dict(wl.weights)
    W["adapters"] = [make_lora(wl.cfg, 105, 16, tag=1), make_lora(wl.cfg, 105, 16, tag=2)]
    b = wl.batch
    batch = Batch(b.chunks, b.rows, b.token_ids, chunk_adapter=[0, 1])
    pair = Pair(wl.cfg, W, wl.kv, acc_w=wl.acc_w)
    pair.workspace(max_tokens=b.n_tokens, max_chunks=2, max_decode=len(b.rows), max_ctx=4096)
    pair.step(batch, check_kv=False)
    print(pair.report, flush=True)


def test_runner_lora_requests():
    """Adapter-named embedding requests through the scheduler and the runner (bf16)."""
    cfg = tiny_config("bf16")
    W = make_weights(cfg, 107, qk_std=0.09)
    W["adapters"] = [make_lora(cfg, 107, 16, tag=t) for t in range(3)]
    W64 = as_float64(W)
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV(cfg, 96, 6, 16)
    sched = R.Scheduler(budget=96, chunk=32, caches=[(6, 96, 16)])
    runner = R.Runner(dm, dm, kv, kv, sched)
    reqs = {}
    for rid, n, ad in ((1, 70, 0), (2, 45, 2), (3, 20, -1), (4, 64, 1), (5, 9, 0)):
        ids = draw_tokens(107, rid, n, cfg.vocab)
        reqs[rid] = (ids, ad)
        sched.submit_embedding(rid, n, ids, "mean", adapter=ad)
    sched.submit_generation(6, 30, 4, draw_tokens(107, 6, 30, cfg.vocab))
    embs = {}
    for _ in range(60):
        out = runner.iterate()
        embs.update(out["embeddings"])
        c = sched.counts()
        if out["n_items"] == 0 and c["queued_emb"] == c["queued_gen"] == c["running"] == 0:
            break
    assert runner.ws.device_error() == 0
    for rid, (ids, ad) in reqs.items():
        lora = W64["adapters"][ad] if ad >= 0 else None
        assert_vectors_close(embs[rid][None], embed_single_pass(cfg, W64, ids, "mean", lora=lora)[None],
                             "bf16", f"embedding {rid}")


@pytest.mark.parametrize("dtype,qk_std", [("f32", None), ("bf16", 0.09)])
def test_lora_two_models_concurrent_groups(dtype, qk_std):
    """Adapters on the embedding model of a two-model step: the embedding rows (adapted and
    base chunks) run on one stream with their shrink launches, the generator's decode rows over
    its own weights and cache on the other, every step checked against the oracle."""
    cfg = tiny_config(dtype)
    W_e = make_weights(cfg, 107, model_tag=1, qk_std=qk_std)
    W_e["adapters"] = [make_lora(cfg, 107, 16, tag=1), make_lora(cfg, 107, 16, tag=2, scale=1.0)]
    W_g = make_weights(cfg, 107, model_tag=2, qk_std=qk_std)
    W64 = as_float64(W_e)
    lens, ads, chunk, max_blocks = [150, 97, 64], [0, 1, -1], 64, 32
    decode_ctx = (50, 90, 300)
    pe = PagedKV(cfg, len(lens) * max_blocks + 3, len(lens), max_blocks, 107)
    for s, n in enumerate(lens):
        pe.reserve(s, n)
    pg = PagedKV(cfg, len(decode_ctx) * max_blocks + 3, len(decode_ctx), max_blocks, 108)
    for i, c in enumerate(decode_ctx):
        pg.fill_random(i, c, 109)
        pg.reserve(i, c + 8)
    pair = Pair(cfg, W_e, pe, cfg, W_g, pg)
    pair.workspace(max_tokens=chunk * len(lens) + len(decode_ctx), max_chunks=len(lens),
                   max_decode=len(decode_ctx), max_ctx=max_blocks * 16)
    ids = {s: draw_tokens(107, s, lens[s], cfg.vocab) for s in range(len(lens))}
    done = {}
    for step, off in enumerate(range(0, max(lens), chunk)):
        chunks, toks, cads = [], [], []
        for s in range(len(lens)):
            if off < lens[s]:
                ln = min(chunk, lens[s] - off)
                chunks.append(EmbChunk(s, off, ln, off + ln == lens[s], "mean"))
                toks.append(ids[s][off:off + ln])
                cads.append(ads[s])
        rows = [DecodeRow(i, c + step) for i, c in enumerate(decode_ctx)]
        toks.append(draw_tokens(107, 100 + step, len(rows), cfg.vocab))
        _, _, out = pair.step(Batch(chunks, rows, np.concatenate(toks).astype(np.int32), chunk_adapter=cads))
        for i, c in enumerate(chunks):
            if c.last:
                done[c.seq] = out[i].cpu().numpy()
    for s, ad in enumerate(ads):
        want = embed_single_pass(cfg, W64, ids[s], "mean", lora=W64["adapters"][ad] if ad >= 0 else None)
        assert_vectors_close(done[s][None], want[None], dtype, f"request {s} vs single pass")
    print(pair.report, flush=True)
