"""Parity at the larger scenario shapes: 7B-shape layers (d 4096, 32 q / 8 kv heads x 128,
SwiGLU 14336, vocab 32000), bf16, at reduced depth so the float64 oracle stays in seconds.

* two models, one step per embedding fraction of a 2048-token budget (queries with lognormal
  lengths, decode rows with lognormal contexts): every output against the oracle;
* long documents chunked by 512 and interleaved with decode rows: every step against the
  oracle, and one 8192-token document chunked sixteen ways against the same document in one
  pass on the GPU (a property that holds at any size);
* decode-heavy: 256 decode rows at contexts 4096..8192 (6.4 GB of cache) plus short queries in
  one launch; the oracle recomputes every row and every query from the same cache bytes (each
  request's outputs depend only on its own cache and tokens), and every pool byte the step does
  not own is compared bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import OracleKV, step_oracle
from tests.parity import TOL_STATE, Pair, assert_vectors_close
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


def _oracle_cache(k_pool, v_pool, rec, seqs, P):
    """float64 host image of the pages of `seqs` (same page contents, compact page ids) and the
    block table that maps each sequence's blocks onto it.  k_pool [L][page][kvh][slot][hd], v_pool
    [L][page][kvh][hd][slot]: the drawn contents, copied before the step; a bf16 cache, so the
    oracle stores what the step writes rounded to bfloat16."""
    pages = [rec.block_table[s][rec.block_table[s] >= 0] for s in seqs]
    flat = torch.from_numpy(np.concatenate(pages).astype(np.int64)).cuda()
    k64 = k_pool[:, flat].float().cpu().numpy().astype(np.float64)
    v64 = v_pool[:, flat].transpose(-1, -2).float().cpu().numpy().astype(np.float64)
    bt = np.full((len(seqs), rec.max_blocks), -1, np.int64)
    o = 0
    for i, p in enumerate(pages):
        bt[i, :len(p)] = np.arange(o, o + len(p))
        o += len(p)
    return OracleKV(k64, v64, bt, P, bf16=True)


def test_decode_heavy_every_row():
    """256 decode rows at contexts U[4096, 8192] (6.4 GB of keys and values) next to 8 queries of
    16 tokens, one launch.  Every decode row's logits and cache write, every query's embedding and
    pooling count against the oracle; the oracle runs in groups of 32 requests from the same cache
    bytes (each request's outputs depend only on its own cache and tokens), so host memory stays
    bounded; it reads the pools as drawn (a copy taken before the step).  Every byte of both
    pools outside the step's slots is compared bit for bit with that copy."""
    cfg, W, batch, rec = decode_heavy_scenario()
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV(cfg, rec.n_pages, rec.n_seq, rec.max_blocks)
    kv.set_block_table(rec.block_table)
    fill_device_pools(kv.k, kv.v, rec.seed)
    before_k, before_v = kv.k.clone(), kv.v.clone()
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

    # every slot the step does not own keeps its bytes (both pools, compared on the device)
    P = cfg.page_size
    owned = torch.zeros((rec.n_pages, P), dtype=torch.bool, device="cuda")
    slots = [(int(rec.block_table[c.seq][p // P]), p % P) for c in batch.chunks for p in range(c.len)]
    slots += [(int(rec.block_table[r.seq][r.ctx_len // P]), r.ctx_len % P) for r in batch.rows]
    assert len(set(slots)) == len(slots) == batch.n_tokens
    idx = torch.tensor(slots, device="cuda")
    owned[idx[:, 0], idx[:, 1]] = True
    # keys [L][page][kvh][slot][hd], values [L][page][kvh][hd][slot]
    assert bool((kv.k.view(torch.int16) == before_k.view(torch.int16)).all(dim=-1).permute(1, 3, 0, 2)[~owned].all())
    assert bool((kv.v.view(torch.int16) == before_v.view(torch.int16)).all(dim=-2).permute(1, 3, 0, 2)[~owned].all())

    W64 = as_float64(W)
    q_ids = batch.token_ids[:batch.n_emb_tokens]
    r_ids = batch.token_ids[batch.n_emb_tokens:]
    worst = {"logits": (0.0, 1.0), "emb": (0.0, 1.0)}

    def check_slots(okv, slots, what):
        """slots: (request index in okv, request's seq in the device cache, position)"""
        for i, s, p in slots:
            dev_page = int(rec.block_table[s][p // P])
            gk = kv.k[0, dev_page, :, p % P, :].float().cpu().numpy()
            gv = kv.v_by_position[0, dev_page, :, p % P, :].float().cpu().numpy()
            ok_page = int(okv.block_table[i, p // P])
            assert_vectors_close(gk, okv.k[0, ok_page, :, p % P, :], "bf16", f"key of {what} {s} pos {p}", TOL_STATE)
            assert_vectors_close(gv, okv.v[0, ok_page, :, p % P, :], "bf16", f"value of {what} {s} pos {p}",
                                 TOL_STATE)

    # the queries
    seqs = [c.seq for c in batch.chunks]
    okv = _oracle_cache(before_k, before_v, rec, seqs, P)
    sub = Batch([EmbChunk(i, c.offset, c.len, c.last, c.pool) for i, c in enumerate(batch.chunks)], [], q_ids)
    ref = step_oracle((cfg, W64), (cfg, W64), sub, okv, okv, np.zeros((nq, cfg.d_model)), np.zeros(nq))
    worst["emb"] = assert_vectors_close(out.cpu().numpy(), ref["out_emb"], "bf16", "query embeddings")
    np.testing.assert_array_equal(Wc[:nq].cpu().numpy(), ref["acc_w"])
    check_slots(okv, [(i, c.seq, p) for i, c in enumerate(batch.chunks) for p in range(c.len)], "query")
    # the decode rows, 32 requests at a time
    g_logits = logits.cpu().numpy()
    for g0 in range(0, nd, 32):
        grp = list(range(g0, min(nd, g0 + 32)))
        seqs = [batch.rows[i].seq for i in grp]
        okv = _oracle_cache(before_k, before_v, rec, seqs, P)
        sub = Batch([], [DecodeRow(k, batch.rows[i].ctx_len) for k, i in enumerate(grp)], r_ids[grp])
        ref = step_oracle((cfg, W64), (cfg, W64), sub, okv, okv, np.zeros((0, cfg.d_model)), np.zeros(0))
        rl = assert_vectors_close(g_logits[grp], ref["logits"], "bf16", f"logits of rows {grp[0]}..{grp[-1]}")
        worst["logits"] = (max(worst["logits"][0], rl[0]), min(worst["logits"][1], rl[1]))
        check_slots(okv, [(k, batch.rows[i].seq, batch.rows[i].ctx_len) for k, i in enumerate(grp)], "decode row")
        print(f"rows {grp[0]}..{grp[-1]}: logits {rl}", flush=True)
    print(f"every row: logits {worst['logits']}, embeddings {worst['emb']}", flush=True)
