"""Parity at the larger scenario shapes: 7B-shape layers (d 4096, 32 q / 8 kv heads x 128,
SwiGLU 14336, vocab 32000), bf16, at reduced depth so the float64 oracle stays in seconds.

* two models, one step per embedding fraction of a 2048-token budget (queries with lognormal
  lengths, decode rows with lognormal contexts): every output against the oracle;
* long documents chunked by 512 and interleaved with decode rows: every step against the
  oracle, and one 8192-token document chunked sixteen ways against the same document in one
  pass on the GPU (a property that holds at any size);
* decode-heavy: 256 decode rows at contexts 4096..8192 (6.4 GB of cache) plus short queries in
  one launch; the oracle recomputes a sample of rows and every query from the same cache bytes
  (each request's outputs depend only on its own cache and tokens).
"""
import numpy as np
import pytest
import torch

from oracle import OracleKV, step_oracle
from tests.parity import Pair, assert_vectors_close
from paper_2609_25405_amd import runtime as R
from workload import (Batch, DecodeRow, EmbChunk, as_float64, decode_heavy_scenario, draw_tokens,
                      fill_device_pools, llm7b_config, long_document_scenario, make_weights,
                      retrieval_mix_scenario)

pytestmark = pytest.mark.gpu


def test_two_models_embedding_fraction_sweep():
    cfg_e, W_e, cfg_g, W_g, pe, pg, steps = retrieval_mix_scenario()
    pair = Pair(cfg_e, W_e, pe, cfg_g, W_g, pg)
    pair.workspace(max_tokens=2048, max_chunks=max(len(b.chunks) for b in steps), max_decode=256,
                   max_ctx=4096)
    for b in steps:
        print(f"step: {len(b.chunks)} queries / {b.n_emb_tokens} tokens + {len(b.rows)} decode rows",
              flush=True)
        pair.step(b)
        print("  ", pair.report[-1], flush=True)


def test_long_documents_chunked_with_decode():
    cfg, W, paged, steps = long_document_scenario()
    pair = Pair(cfg, W, paged)
    pair.workspace(max_tokens=1536 + 32, max_chunks=3, max_decode=32, max_ctx=2048 + 8)
    for b in steps:
        print(f"step: chunks {[(c.seq, c.offset, c.len, c.last) for c in b.chunks]} + {len(b.rows)} rows",
              flush=True)
        pair.step(b)
        print("  ", pair.report[-1], flush=True)


def test_long_document_sixteen_chunks_equal_one_pass():
    """One 8192-token document through 16 chunks of 512 and through one chunk (GPU both ways)."""
    cfg = llm7b_config(n_layers=1)
    W = make_weights(cfg, 1006)
    n, C, P = 8192, 512, cfg.page_size
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV(cfg, 2 * n // P, 2, n // P)
    bt = np.arange(2 * n // P, dtype=np.int32)[::-1].reshape(2, n // P).copy()   # disjoint pages
    kv.set_block_table(bt)
    ids = draw_tokens(1006, 1, n, cfg.vocab)
    S = torch.zeros((2, cfg.d_model), device="cuda")
    Wc = torch.zeros(2, device="cuda")
    out = torch.full((1, cfg.d_model), float("nan"), device="cuda")
    ws = R.Workspace(dm, dm, n, 1, 0, n)
    for k in range(n // C):
        b = Batch([EmbChunk(0, k * C, C, k == n // C - 1, "mean")], [], ids[k * C:(k + 1) * C])
        R.step(dm, dm, b, kv, kv, S, Wc, None, out, ws)
    chunked = out.clone()
    R.step(dm, dm, Batch([EmbChunk(1, 0, n, True, "mean")], [], ids), kv, kv, S, Wc, None, out, ws)
    torch.cuda.synchronize()
    assert ws.device_error() == 0
    assert Wc.tolist() == [float(n), float(n)]
    rel, cos = assert_vectors_close(chunked.cpu().numpy(), out.cpu().numpy(), "bf16", "16 chunks vs one")
    print(f"max rel {rel:.3g}, cos {cos:.6f}", flush=True)


def test_decode_heavy_sampled_rows():
    cfg, W, batch, rec = decode_heavy_scenario()
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV(cfg, rec.n_pages, rec.n_seq, rec.max_blocks)
    kv.set_block_table(rec.block_table)
    fill_device_pools(kv.k, kv.v, rec.seed)
    nq, nd = len(batch.chunks), len(batch.rows)
    S = torch.zeros((rec.n_seq, cfg.d_model), device="cuda")
    Wc = torch.zeros(rec.n_seq, device="cuda")
    logits = torch.full((nd, cfg.vocab), float("nan"), device="cuda")
    out = torch.full((nq, cfg.d_model), float("nan"), device="cuda")
    ws = R.Workspace(dm, dm, batch.n_tokens, nq, nd, max(r.ctx_len for r in batch.rows) + 1)
    print(f"decode-heavy step: {nd} rows, {rec.n_pages} pages, {nq} queries", flush=True)
    R.step(dm, dm, batch, kv, kv, S, Wc, logits, out, ws)
    torch.cuda.synchronize()
    assert ws.device_error() == 0

    # the oracle on every query and a sample of rows (shortest, longest, seeded others), from the
    # same cache bytes copied into a compact cache with the same page contents
    ctx = np.array([r.ctx_len for r in batch.rows])
    rng = np.random.default_rng(7)
    sample = sorted({int(ctx.argmin()), int(ctx.argmax()), 0, nd - 1, *rng.choice(nd, 2, replace=False).tolist()})
    seqs = [c.seq for c in batch.chunks] + [batch.rows[i].seq for i in sample]
    P = cfg.page_size
    pages = [rec.block_table[s][rec.block_table[s] >= 0] for s in seqs]
    flat = torch.from_numpy(np.concatenate(pages).astype(np.int64)).cuda()
    k64 = kv.k[:, flat].float().cpu().numpy().astype(np.float64)
    v64 = kv.v_by_position[:, flat].float().cpu().numpy().astype(np.float64)
    bt = np.full((len(seqs), rec.max_blocks), -1, np.int64)
    o = 0
    for i, p in enumerate(pages):
        bt[i, :len(p)] = np.arange(o, o + len(p))
        o += len(p)
    okv = OracleKV(k64, v64, bt, P)
    q_ids = batch.token_ids[:batch.n_emb_tokens]
    r_ids = batch.token_ids[batch.n_emb_tokens:][sample]
    sub = Batch([EmbChunk(i, c.offset, c.len, c.last, c.pool) for i, c in enumerate(batch.chunks)],
                [DecodeRow(nq + k, batch.rows[i].ctx_len) for k, i in enumerate(sample)],
                np.concatenate([q_ids, r_ids]).astype(np.int32))
    W64 = as_float64(W)
    ref = step_oracle((cfg, W64), (cfg, W64), sub, okv, okv, np.zeros((len(seqs), cfg.d_model)),
                      np.zeros(len(seqs)))
    rl = assert_vectors_close(logits[sample].cpu().numpy(), ref["logits"], "bf16", "logits (sampled rows)")
    re = assert_vectors_close(out.cpu().numpy(), ref["out_emb"], "bf16", "query embeddings")
    np.testing.assert_array_equal(Wc[:nq].cpu().numpy(), ref["acc_w"][:nq])
    # cache slots written by the step: every query token and each sampled row's new token
    for i, s in enumerate(seqs):
        positions = range(batch.chunks[i].len) if i < nq else [batch.rows[sample[i - nq]].ctx_len]
        for p in positions:
            dev_page = int(rec.block_table[s][p // P])
            gk = kv.k[0, dev_page, :, p % P, :].float().cpu().numpy()
            gv = kv.v_by_position[0, dev_page, :, p % P, :].float().cpu().numpy()
            ok_page = int(bt[i, p // P])
            assert_vectors_close(gk, okv.k[0, ok_page, :, p % P, :], "bf16", f"key seq {s} pos {p}")
            assert_vectors_close(gv, okv.v[0, ok_page, :, p % P, :], "bf16", f"value seq {s} pos {p}")
    print(f"sampled rows {sample}: logits {rl}, embeddings {re}", flush=True)
