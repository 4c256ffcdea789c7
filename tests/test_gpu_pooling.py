"""GPU parity of the weighted-mean and buffered pooling heads (Section 3.3) against the oracle.

Weighted mean takes one caller weight per embedding token (Eq. (1)-(2) with general weights);
the buffered head writes each chunk's final-normed hidden rows to a caller buffer, from which
any head can be applied after the final chunk.  Both are checked step by step against the
oracle (embeddings, buffered rows, token counts, cache writes) and, at the end, against the
single-pass definitions of the whole request.
"""
import numpy as np
import pytest
import torch

from oracle import embed_single_pass, forward_full
from tests.parity import Pair, assert_vectors_close
from workload import (Batch, DecodeRow, EmbChunk, PagedKV, as_float64, draw_token_weights,
                      draw_tokens, layer7b_mixed_workload, make_weights, tiny_config)
from paper_2609_25405_amd import runtime as R

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


@pytest.mark.parametrize("dtype,qk_std,two_models", [("f32", None, False), ("bf16", 0.09, False), ("bf16", 0.09, True)])
def test_weighted_and_buffered_heads_over_two_steps(dtype, qk_std, two_models):
    """Requests: 0 weighted mean (150 tokens in 100 + 50), 1 buffered (90 in 64 + 26), 2 mean
    (40, one chunk), 3 weighted mean with all-zero weights (20), plus decode rows; with two
    models the decode rows run through a generator of its own weights and cache, concurrently."""
    cfg = tiny_config(dtype)
    W = make_weights(cfg, 91, qk_std=qk_std)
    W64 = as_float64(W)
    n_seq, mb = 7, 16
    pk = PagedKV(cfg, n_seq * mb + 3, n_seq, mb, 91)
    for s in range(4):
        pk.reserve(s, 200)
    if two_models:
        pg = PagedKV(cfg, n_seq * mb + 3, n_seq, mb, 93)
        W_g = make_weights(cfg, 91, model_tag=2, qk_std=qk_std)
    else:
        pg = pk
    for s in (4, 5):
        pg.fill_random(s, 60 + 10 * s, 92)
        pg.reserve(s, 64 + 10 * s)
    pair = Pair(cfg, W, pk, cfg, W_g, pg) if two_models else Pair(cfg, W, pk)
    pair.workspace(max_tokens=256, max_chunks=4, max_decode=2, max_ctx=256)
    ids = {0: draw_tokens(91, 0, 150, cfg.vocab), 1: draw_tokens(91, 1, 90, cfg.vocab),
           2: draw_tokens(91, 2, 40, cfg.vocab), 3: draw_tokens(91, 3, 20, cfg.vocab)}
    w0 = draw_token_weights(91, 0, 150)
    stride = 96
    # step 1
    ch = [EmbChunk(0, 0, 100, False, "wmean"), EmbChunk(1, 0, 64, False, "buffer"),
          EmbChunk(2, 0, 40, True, "mean"), EmbChunk(3, 0, 20, True, "wmean")]
    tok = np.concatenate([ids[0][:100], ids[1][:64], ids[2], ids[3],
                          draw_tokens(91, 9, 2, cfg.vocab)]).astype(np.int32)
    tw = np.concatenate([w0[:100], np.full(64, -1.0, np.float32),   # ignored: not weighted chunks
                         np.full(40, np.nan, np.float32), np.zeros(20, np.float32)])
    ref1, _, out1 = pair.step(Batch(ch, [DecodeRow(4, 100), DecodeRow(5, 110)], tok,
                                    token_weights=tw, hidden_stride=stride))
    # step 2
    ch2 = [EmbChunk(1, 64, 26, True, "buffer"), EmbChunk(0, 100, 50, True, "wmean")]
    tok2 = np.concatenate([ids[1][64:], ids[0][100:]]).astype(np.int32)
    tw2 = np.concatenate([np.ones(26, np.float32), w0[100:]])
    ref2, _, out2 = pair.step(Batch(ch2, [], tok2, token_weights=tw2, hidden_stride=stride))
    # whole-request definitions
    e0 = out2[1].cpu().numpy()
    assert_vectors_close(e0[None], embed_single_pass(cfg, W64, ids[0], "wmean", w0)[None], dtype,
                         "weighted mean vs single pass")
    assert_vectors_close(out1[2].cpu().numpy()[None], embed_single_pass(cfg, W64, ids[2], "mean")[None],
                         dtype, "mean vs single pass")
    assert np.all(out1[3].cpu().numpy() == 0)
    H1 = np.concatenate([ref1["hidden"][1], ref2["hidden"][0]])
    assert_vectors_close(H1, forward_full(cfg, W64, ids[1]), dtype, "buffered rows vs single pass")
    print(pair.report, flush=True)


def test_layer7b_weighted_and_buffered_heads():
    """The 7B-layer mixed step with its two 512-token chunks switched to weighted mean (request
    0, resuming after 1536 cached tokens) and the buffered head (request 1)."""
    wl = layer7b_mixed_workload()
    b = wl.batch
    c0, c1 = b.chunks
    chunks = [EmbChunk(c0.seq, c0.offset, c0.len, c0.last, "wmean"),
              EmbChunk(c1.seq, c1.offset, c1.len, c1.last, "buffer")]
    n_emb = c0.len + c1.len
    tw = np.concatenate([draw_token_weights(1002, 5, c0.len), np.zeros(c1.len, np.float32)])
    batch = Batch(chunks, b.rows, b.token_ids, token_weights=tw, hidden_stride=2048)
    pair = Pair(wl.cfg, wl.weights, wl.kv, acc_w=wl.acc_w)
    pair.workspace(max_tokens=b.n_tokens, max_chunks=2, max_decode=len(b.rows), max_ctx=4096)
    pair.step(batch, check_kv=False)
    print(pair.report, flush=True)


def test_runner_weighted_requests():
    """Weighted-mean requests through the scheduler and the runner (bf16)."""
    cfg = tiny_config("bf16")
    W = make_weights(cfg, 93, qk_std=0.09)
    W64 = as_float64(W)
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV(cfg, 64, 4, 16)
    sched = R.Scheduler(budget=64, chunk=24, caches=[(4, 64, 16)])
    runner = R.Runner(dm, dm, kv, kv, sched)
    reqs = {}
    for rid, n in ((1, 70), (2, 33), (3, 5)):
        ids = draw_tokens(93, rid, n, cfg.vocab)
        w = draw_token_weights(93, rid, n)
        reqs[rid] = (ids, w)
        sched.submit_embedding(rid, n, ids, "wmean", weights=w)
    sched.submit_embedding(4, 40, draw_tokens(93, 4, 40, cfg.vocab), "mean")
    embs = {}
    for _ in range(50):
        out = runner.iterate()
        embs.update(out["embeddings"])
        if out["n_items"] == 0:
            break
    assert runner.ws.device_error() == 0
    for rid, (ids, w) in reqs.items():
        assert_vectors_close(embs[rid][None], embed_single_pass(cfg, W64, ids, "wmean", w)[None], "bf16",
                             f"embedding {rid}")
