"""Oracle parity at depth: the error of the bf16 path grows with the number of layers (every
layer rounds its GEMM inputs and its cached keys/values to bf16), so the shallow cases of the
other files do not show that the full-depth models stay inside the output bounds.

* a narrow grouped-query decoder (hidden 512, 8 query heads sharing 2 KV heads of 128) at 2, 8
  and 32 layers, fp32 and bf16, through C1-style mixed steps: cache-filling chunks, chunked
  mean / last-token / CLS embeddings, generation prompt chunks and decode rows, every output and
  every cache write against the oracle;
* the 7B-shape mixed step (1024 chunk tokens + 64 decode rows) at 4 layers against the oracle;
* long documents (the 16 x 8192-token configuration, two of its documents) on a two-layer
  7B-shape model: 16 chunks of 512 per document next to 32 decode rows, the finished embeddings
  against the single-pass definition (Section 3.3: chunked equals unchunked).

Each case prints max relative error and cosine per output kind.
"""
import numpy as np
import pytest
import torch

from oracle import embed_single_pass
from tests.parity import Pair, assert_vectors_close
from paper_2609_25405_amd import runtime as R
from workload import (Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, as_float64, draw_tokens,
                      layer7b_mixed_workload, long_document_scenario, make_weights)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def narrow_gqa_config(n_layers: int, dtype: str) -> ModelConfig:
    return ModelConfig(n_layers=n_layers, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       d_ff=1024, vocab=512, dtype=dtype)


def mixed_steps(cfg, seed: int):
    """Four steps over eight requests (one shared cache):
    step 0: cache-filling chunks of generation requests 4..7 (64 / 100 / 150 / 200 tokens);
    step 1: embeddings 0 (mean) and 1 (CLS), first chunks of 128, 2 (last-token, one chunk of 60),
            prompt 3's first chunk (80), decode rows 4..7;
    step 2: embedding 0's second chunk, embedding 1's final chunk (44), prompt 3's final chunk
            (40, gets logits), decode rows 4..7;
    step 3: embedding 0's final chunk (44), decode rows 3..7 (3 decodes its first new token)."""
    prompts = [64, 100, 150, 200]
    steps = [Batch([EmbChunk(4 + i, 0, p, False, "none") for i, p in enumerate(prompts)], [],
                   draw_tokens(seed, 0, sum(prompts), cfg.vocab))]
    ctx = list(prompts)

    def rows(first=4):
        out = [DecodeRow(s, ctx[s - 4]) for s in range(4, 8)]
        return ([DecodeRow(3, 120)] if first == 3 else []) + out

    b1 = Batch([EmbChunk(0, 0, 128, False, "mean"), EmbChunk(1, 0, 128, False, "cls"),
                EmbChunk(2, 0, 60, True, "last")], rows(),
               draw_tokens(seed, 1, 128 + 128 + 60 + 80 + 4, cfg.vocab), gen_chunks=[GenChunk(3, 0, 80, False)])
    steps.append(b1)
    ctx = [c + 1 for c in ctx]
    b2 = Batch([EmbChunk(0, 128, 128, False, "mean"), EmbChunk(1, 128, 44, True, "cls")], rows(),
               draw_tokens(seed, 2, 128 + 44 + 40 + 4, cfg.vocab), gen_chunks=[GenChunk(3, 80, 40, True)])
    steps.append(b2)
    ctx = [c + 1 for c in ctx]
    b3 = Batch([EmbChunk(0, 256, 44, True, "mean")], rows(first=3), draw_tokens(seed, 3, 44 + 5, cfg.vocab))
    steps.append(b3)
    return steps


def depth_qk_std(dtype: str, n_layers: int) -> float:
    """Spread of the query/key weights: attention logits of std ~ qk_std^2 * 512.  bf16: 0.06
    (std ~1.8).  fp32: as sharp as the depth allows at the 1e-4 bound, because sharp attention
    through many layers is ill-conditioned (tests/test_conditioning.py: the float64 definition
    itself, under a 2^-24 relative change of its inputs, moves 1.1e-2 at 32 layers with 0.15 and
    grows tenfold from 2 to 32 layers with 0.09, while fp32 arithmetic rounds at every
    operation): 0.15 (std ~12, near one-hot) at two layers, 0.09 (std ~4) at eight, 0.06 at 32."""
    if dtype == "bf16":
        return 0.06
    return 0.15 if n_layers <= 2 else 0.09 if n_layers <= 8 else 0.06


@pytest.mark.parametrize("n_layers", [2, 8, 32])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_narrow_gqa_mixed_steps_at_depth(dtype, n_layers):
    cfg = narrow_gqa_config(n_layers, dtype)
    seed = 2100 + n_layers
    W = make_weights(cfg, seed, qk_std=depth_qk_std(dtype, n_layers))
    n_seq, max_blocks = 8, 32
    pk = PagedKV(cfg, n_seq * max_blocks + 5, n_seq, max_blocks, seed)
    for s, n in enumerate([300, 172, 60, 122, 67, 103, 153, 203]):
        pk.reserve(s, n)
    pair = Pair(cfg, W, pk)
    steps = mixed_steps(cfg, seed)
    pair.workspace(max_tokens=max(b.n_tokens for b in steps), max_chunks=4, max_decode=5, max_ctx=512)
    for b in steps:
        pair.step(b)
    print(f"{dtype} {n_layers} layers: {pair.report}", flush=True)


def test_layer7b_mixed_step_four_layers():
    """The 7B-shape mixed step (two 512-token chunks, one resuming after 1536 cached tokens, last-
    token pooling; 64 decode rows at contexts U[1024, 4096]) through four layers."""
    wl = layer7b_mixed_workload(n_layers=4)
    pair = Pair(wl.cfg, wl.weights, wl.kv, acc_w=wl.acc_w)
    pair.workspace(max_tokens=wl.batch.n_tokens, max_chunks=2, max_decode=64, max_ctx=4096)
    pair.step(wl.batch)
    print(f"4 layers: {pair.report}", flush=True)


def chunk_tokens(batch, j: int) -> np.ndarray:
    """Token ids of embedding chunk j of a batch (chunk tokens come first, in chunk order)."""
    start = sum(c.len for c in batch.chunks[:j])
    return batch.token_ids[start:start + batch.chunks[j].len]


def test_long_documents_sixteen_chunks_against_single_pass():
    """Two 8192-token documents on a two-layer 7B-shape model, chunked by 512 (one chunk of each
    per step, 16 steps) next to 32 decode rows that advance one token per step.  The first step
    (outputs, pooling state, cache writes) is checked against the step oracle; after the 16th
    the finished embeddings against the single-pass definition and W against 8192 exactly."""
    cfg, W, paged, steps = long_document_scenario(n_layers=2, n_docs=2, doc_len=8192, chunk=512, per_step=2,
                                                  n_dec=32, ctx0=2048)
    assert len(steps) == 16 and all(len(b.chunks) == 2 for b in steps)
    pair = Pair(cfg, W, paged)
    pair.workspace(max_tokens=max(b.n_tokens for b in steps), max_chunks=2, max_decode=32,
                   max_ctx=paged.max_blocks * cfg.page_size)
    pair.step(steps[0])
    print(f"step 0 against the step oracle: {pair.report[-1]}", flush=True)
    logits = torch.empty((32, cfg.vocab), device="cuda")
    out = torch.full((2, cfg.d_model), float("nan"), device="cuda")
    for b in steps[1:]:
        R.step(pair.dm_e, pair.dm_e, b, pair.dkv_e, pair.dkv_e, pair.acc_sum, pair.acc_w, logits, out, pair.ws)
    torch.cuda.synchronize()
    assert pair.ws.device_error() == 0
    assert all(c.last for c in steps[-1].chunks)
    assert pair.acc_w[:2].tolist() == [8192.0, 8192.0]
    W64 = as_float64(W)
    for i, c in enumerate(steps[-1].chunks):
        ids = np.concatenate([chunk_tokens(b, j) for b in steps for j, x in enumerate(b.chunks) if x.seq == c.seq])
        assert ids.size == 8192
        ref = embed_single_pass(cfg, W64, ids, "mean")
        g = out[i:i + 1].cpu().numpy()
        rel, cos = assert_vectors_close(g, ref[None], "bf16", f"document {c.seq}: 16 chunks vs single pass")
        print(f"document {c.seq}: max rel {rel:.3g}, cos {cos:.6f}", flush=True)
