"""GPU parity of orthrus_step against the float64 oracle (needs an MI355X and the built library).

Every case runs the same seeded inputs through the oracle and through the C ABI, step by step,
and compares logits, finished embeddings, the pooling state and the cache writes.
"""
import sys

import numpy as np
import pytest
import torch

from workload import (Batch, DecodeRow, EmbChunk, ModelConfig, PagedKV, draw_tokens, make_weights,
                      tiny_config, tiny_mixed_scenario, layer7b_mixed_workload)
from tests.parity import Pair, assert_vectors_close
from paper_2609_25405_amd import runtime as R

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _tiny_pair(dtype, qk_std=None, seed=1001):
    cfg, W, n_seq, steps = tiny_mixed_scenario(seed=seed, dtype=dtype, qk_std=qk_std)
    max_tok = 512
    pk = PagedKV(cfg, n_pages=n_seq * (max_tok // 16) + 7, n_seq=n_seq, max_blocks=max_tok // 16, seed=seed)
    for s in range(n_seq):
        pk.reserve(s, 320)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=max(b.n_tokens for b in steps), max_chunks=4, max_decode=4, max_ctx=max_tok)
    return pair, steps


# qk_std sets the attention logit spread: std(q.k / sqrt(hd)) ~ qk_std^2 * d_model, i.e. ~10
# at 0.2 (near one-hot softmax: exact fp32 only, bf16 rounding of q and k alone moves such
# weights by several percent) and ~2 at 0.09 (sharp enough that a wrong key or position shows).
@pytest.mark.parametrize("dtype,qk_std", [("f32", None), ("f32", 0.2), ("bf16", None), ("bf16", 0.09)])
def test_tiny_mixed_scenario(dtype, qk_std):
    """Two-layer decoder: KV-only prompt chunks, then three mixed steps (300-token embeddings
    chunked 128/128/44 with mean pooling, four decode rows)."""
    pair, steps = _tiny_pair(dtype, qk_std)
    for b in steps:
        pair.step(b)
    print(pair.report, flush=True)


def _gqa_config(dtype="bf16", n_layers=2):
    return ModelConfig(n_layers=n_layers, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       d_ff=1024, vocab=512, dtype=dtype)


def test_long_prefix_prefill_key_splits():
    """Chunks over long cached prefixes (bf16): the planner cuts their query tiles along the keys
    into pieces whose partials the combine merges in piece order.  Two resuming chunks with
    ragged query tails (6000 and 2500 cached tokens), a chunk with no prefix and a decode row;
    embeddings, pooling state, logits and every cache write match the oracle."""
    cfg = _gqa_config("bf16")
    W = make_weights(cfg, 11, qk_std=0.06)
    n_seq, max_blocks = 4, 400
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, 11)
    pk.fill_random(0, 6000, 11)
    pk.reserve(0, 6070)
    pk.fill_random(1, 2500, 12)
    pk.reserve(1, 2540)
    pk.reserve(2, 50)
    pk.fill_random(3, 3000, 13)
    pk.reserve(3, 3001)
    acc_w = np.zeros(n_seq)
    acc_w[0], acc_w[1] = 6000, 2500
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=256, max_chunks=3, max_decode=1, max_ctx=4096)
    chunks = [EmbChunk(0, 6000, 70, True, "mean"), EmbChunk(1, 2500, 40, False, "mean"),
              EmbChunk(2, 0, 50, True, "last")]
    b = Batch(chunks, [DecodeRow(3, 3000)], draw_tokens(11, 1, 70 + 40 + 50 + 1, cfg.vocab))
    npre, _, items = R.plan(pair.dm_e, pair.dm_e, b, pair.dkv_e, pair.dkv_e)
    pieces = items[:npre][items[:npre, 7] >= 0]
    # chunk 0's tiles in 3 pieces (6032..6070 keys, 2048-key target), chunk 1's in 2
    assert len(pieces) == 2 * (3 * 3 + 2 * 2), pieces
    # some pieces start on an odd 64-key block (the kernel's LDS buffers alternate from a
    # piece's own first block, not from block 0)
    assert any((int(p[5]) // 64) % 2 == 1 for p in pieces), pieces[:, 5]
    pair.step(b)
    print(pair.report, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gqa_long_context_splits(dtype):
    """Grouped-query shape (group 4, head_dim 128) with multi-split decode rows, chunk offsets
    past earlier cached tokens, ragged chunk tails and every pooling head."""
    cfg = _gqa_config(dtype)
    W = make_weights(cfg, 7, qk_std=0.06 if dtype == "bf16" else 0.15)
    n_seq, max_blocks = 8, 64
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, 7)
    ctx = [0, 17, 255, 256, 700]
    for i, c in enumerate(ctx):
        pk.fill_random(3 + i, c, 7)
        pk.reserve(3 + i, c + 1)
    pk.fill_random(1, 300, 8)          # request 1 resumes at offset 300
    for s, n in ((0, 200), (1, 433), (2, 97)):
        pk.reserve(s, n)
    acc_w = np.zeros(n_seq)
    acc_w[1] = 300
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=512, max_chunks=3, max_decode=5, max_ctx=1024)
    chunks = [EmbChunk(0, 0, 200, True, "mean"), EmbChunk(1, 300, 133, True, "last"),
              EmbChunk(2, 0, 97, True, "cls")]
    rows = [DecodeRow(3 + i, c) for i, c in enumerate(ctx)]
    ids = draw_tokens(7, 1, 200 + 133 + 97 + len(rows), cfg.vocab)
    pair.step(Batch(chunks, rows, ids))
    # no mean-pooled chunk: the single-row heads take their own final norm (and any pending
    # split-K slabs) inside the pooler; requests 0 and 2 restart at offset 0
    chunks2 = [EmbChunk(0, 0, 64, False, "cls"), EmbChunk(2, 0, 80, True, "last")]
    pair.step(Batch(chunks2, [], draw_tokens(7, 2, 144, cfg.vocab)))
    print(pair.report, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_split_and_single_decode_rows_together(dtype):
    """Decode rows with one key split (written by the attention launch itself) next to rows
    with two and three splits (merged by the launch over the split rows only), beside a chunk."""
    cfg = _gqa_config(dtype)
    W = make_weights(cfg, 8, qk_std=0.06 if dtype == "bf16" else 0.15)
    n_seq, max_blocks = 5, 136
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, 8)
    ctx = [50, 1100, 300, 2100]
    for i, c in enumerate(ctx):
        pk.fill_random(1 + i, c, 8)
        pk.reserve(1 + i, c + 1)
    pk.reserve(0, 96)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=128, max_chunks=1, max_decode=4, max_ctx=2176)
    rows = [DecodeRow(1 + i, c) for i, c in enumerate(ctx)]
    b = Batch([EmbChunk(0, 0, 96, True, "mean")], rows, draw_tokens(8, 1, 100, cfg.vocab))
    npre, _, items = R.plan(pair.dm_e, pair.dm_e, b, pair.dkv_e, pair.dkv_e)
    dec = items[npre:]
    splits = [int(dec[dec[:, 1] == j, 4].max()) for j in range(len(rows))]
    assert splits == ([1, 2, 1, 3] if dtype == "bf16" else [1, 5, 2, 9]), splits
    pair.step(b)
    print(pair.report, flush=True)


def test_two_models_two_pools():
    """Separate embedding and generation models (same shape) with separate caches."""
    cfg = tiny_config("bf16")
    We = make_weights(cfg, 21, model_tag=1)
    Wg = make_weights(cfg, 21, model_tag=2)
    pe = PagedKV(cfg, 80, 4, 20, 1)
    pg = PagedKV(cfg, 80, 4, 20, 2)
    for s in range(4):
        pe.reserve(s, 300)
        pg.fill_random(s, 40 + 30 * s, 3)
        pg.reserve(s, 41 + 30 * s)
    pair = Pair(cfg, We, pe, cfg, Wg, pg)
    pair.workspace(max_tokens=300, max_chunks=2, max_decode=4, max_ctx=320)
    ids = draw_tokens(3, 3, 150 + 4, cfg.vocab)
    # seq 0 appears in both sections: legal, the two pools are separate namespaces
    b = Batch([EmbChunk(0, 0, 100, True, "mean"), EmbChunk(1, 0, 50, False, "mean")],
              [DecodeRow(s, 40 + 30 * s) for s in range(4)], ids)
    pair.step(b)


def test_chunked_equals_single_pass_on_gpu():
    """Section 3.3 equivalence on the device: 300 tokens in chunks of 128 vs one chunk."""
    cfg = tiny_config("bf16")
    W = make_weights(cfg, 5, qk_std=0.09)
    ids = draw_tokens(5, 9, 300, cfg.vocab)
    outs = {}
    for C in (128, 300, 37):
        pk = PagedKV(cfg, 40, 1, 20, 4)
        pk.reserve(0, 300)
        dm = R.DeviceModel(cfg, W)
        kv = R.DeviceKV.from_paged(pk)
        ws = R.Workspace(dm, dm, 300, 1, 0, 320)
        S = torch.zeros((1, cfg.d_model), device="cuda")
        Wc = torch.zeros(1, device="cuda")
        out = torch.zeros((1, cfg.d_model), device="cuda")
        for off in range(0, 300, C):
            ln = min(C, 300 - off)
            R.step(dm, dm, Batch([EmbChunk(0, off, ln, off + ln == 300, "mean")], [], ids[off:off + ln]),
                   kv, kv, S, Wc, None, out, ws)
        torch.cuda.synchronize()
        assert ws.device_error() == 0
        assert Wc.item() == 300
        outs[C] = out[0].cpu().numpy()
    for C in (128, 37):
        assert_vectors_close(outs[C][None], outs[300][None], "bf16", f"chunk {C} vs single pass")


def test_layer7b_mixed_step():
    """One 7B-shape layer (bf16, vocab 32000): 1024 chunk tokens (two requests, chunk 512,
    last-token pooling, one of them resuming after 1536 cached tokens) + 64 decode rows with
    contexts in [1024, 4096] over N(0,1) bf16 caches.  Full comparison of every output."""
    wl = layer7b_mixed_workload()
    pair = Pair(wl.cfg, wl.weights, wl.kv, acc_w=wl.acc_w)
    pair.workspace(max_tokens=wl.batch.n_tokens, max_chunks=2, max_decode=64, max_ctx=4096)
    pair.step(wl.batch)
    print(pair.report, flush=True)


def test_layer7b_decode_rows_alone():
    """The 7B-layer step's 64 decode rows without its chunks: a 64-row batch, whose QKV
    projection splits K into fp32 partials that the rotation/append kernel sums (and whose
    other projections stream their weights once).  Logits and every cache write compared."""
    wl = layer7b_mixed_workload()
    pair = Pair(wl.cfg, wl.weights, wl.kv, acc_w=wl.acc_w)
    pair.workspace(max_tokens=wl.batch.n_tokens, max_chunks=2, max_decode=64, max_ctx=4096)
    Te = wl.batch.n_emb_tokens
    pair.step(Batch([], wl.batch.rows, wl.batch.token_ids[Te:]))
    print(pair.report, flush=True)


@pytest.mark.parametrize("n_dec", [96, 128, 192])
def test_layer7b_decode_batches_up_to_192_rows(n_dec):
    """Decode-only 7B-layer batches of 65..192 rows.  Up to 128 rows the QKV projection splits
    K in two into fp32 partials the rotation/append kernel sums, gate/up and the LM head stream
    their weights through one 128-row tile, O and down split K four ways on 128x64 tiles; at 192
    rows QKV takes the fused rotation epilogue and O and down 4-deep 128x128 tiles.  Contexts
    U[256, 1024]; logits and every cache write compared."""
    cfg = ModelConfig(n_layers=1, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128, d_ff=14336,
                      vocab=32000, dtype="bf16")
    seed = 1006
    W = make_weights(cfg, seed)
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(n_dec,)))
    ctx = rng.integers(256, 1024, size=n_dec, endpoint=True)
    P = cfg.page_size
    max_blocks = 1024 // P + 1
    pk = PagedKV(cfg, sum(-(-(int(c) + 1) // P) for c in ctx) + 8, n_dec, max_blocks, seed)
    rows = [DecodeRow(seq=i, ctx_len=int(c)) for i, c in enumerate(ctx)]
    for r in rows:
        pk.fill_random(r.seq, r.ctx_len, seed)
        pk.reserve(r.seq, r.ctx_len + 1)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=n_dec, max_chunks=1, max_decode=n_dec, max_ctx=max_blocks * P)
    pair.step(Batch([], rows, draw_tokens(seed, 1, n_dec, cfg.vocab)))
    print(pair.report, flush=True)


@pytest.mark.parametrize("n_dec", [33, 47, 64, 128, 200])
def test_blocked_lm_head_gives_the_same_logits(n_dec):
    """The LM head read from its 64 x 64 blocked copy (the default for bf16 models) and from the
    row-major weights give bit-identical logits (same tiles, same arithmetic); a vocabulary that
    is not a multiple of 64 exercises the zero-padded last row block, and 33 or 47 rows a partly
    filled row tile of the 64 x 128 tiles that serve 33..64 rows."""
    cfg = ModelConfig(n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                      vocab=4000 + 37, dtype="bf16")
    W = make_weights(cfg, 71)
    P = cfg.page_size
    pk = PagedKV(cfg, n_dec * 4 + 3, n_dec, 4, 71)
    rows = [DecodeRow(i, 17 + i % 40) for i in range(n_dec)]
    for r in rows:
        pk.fill_random(r.seq, r.ctx_len, 71)
        pk.reserve(r.seq, r.ctx_len + 1)
    batch = Batch([], rows, draw_tokens(71, 1, n_dec, cfg.vocab))
    out = {}
    for blocked in (True, False):
        dm = R.DeviceModel(cfg, W, block_lm_head=blocked)
        assert (dm.lm_head_blocked is not None) == blocked
        kv = R.DeviceKV.from_paged(pk)
        ws = R.Workspace(dm, dm, n_dec, 1, n_dec, 4 * P)
        lg = torch.zeros((n_dec, cfg.vocab), device="cuda")
        S = torch.zeros((n_dec, cfg.d_model), device="cuda")
        Wc = torch.zeros(n_dec, device="cuda")
        R.step(dm, dm, batch, kv, kv, S, Wc, lg, None, ws)
        torch.cuda.synchronize()
        assert ws.device_error() == 0
        out[blocked] = lg.cpu()
    assert torch.isfinite(out[True]).all()
    assert torch.equal(out[True], out[False])


def test_device_errors_are_flagged_not_faulted():
    """A chunk whose pooling state does not match its offset, and a block-table entry past the
    pool, raise device error bits; the step still completes and nothing outside is written."""
    cfg = tiny_config("f32")
    W = make_weights(cfg, 3)
    pk = PagedKV(cfg, 20, 3, 8, 1)
    for s in range(3):
        pk.reserve(s, 64)
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV.from_paged(pk)
    ws = R.Workspace(dm, dm, 64, 2, 2, 128)
    S = torch.zeros((3, cfg.d_model), device="cuda")
    Wc = torch.zeros(3, device="cuda")
    out = torch.zeros((2, cfg.d_model), device="cuda")
    lg = torch.zeros((2, cfg.vocab), device="cuda")
    ids = draw_tokens(1, 1, 16, cfg.vocab)
    R.step(dm, dm, Batch([EmbChunk(0, 16, 16, True, "mean")], [], ids), kv, kv, S, Wc, None, out, ws)
    assert ws.device_error() == 2
    assert Wc[0].item() == 0.0                      # the rejected chunk left its state alone
    assert ws.device_error() == 0                   # reading cleared the word
    bt = pk.block_table.copy()
    bt[1, 0] = pk.n_pages                           # one past the pool
    kv.set_block_table(bt)
    R.step(dm, dm, Batch([], [DecodeRow(1, 3)], ids[:1]), kv, kv, S, Wc, lg, None, ws)
    assert ws.device_error() == 1


def test_step_is_bitwise_deterministic():
    """Two runs of the same 7B-layer step on the same inputs give identical bits (split-K slabs,
    decode partials and pooling all reduce in a fixed order; no float atomics)."""
    wl = layer7b_mixed_workload()
    cfg, b = wl.cfg, wl.batch
    dm = R.DeviceModel(cfg, wl.weights)
    kv = R.DeviceKV.from_paged(wl.kv)
    ws = R.Workspace(dm, dm, b.n_tokens, len(b.chunks), len(b.rows), 4096)
    outs = []
    for _ in range(2):
        S = torch.tensor(wl.acc_sum, device="cuda")
        Wc = torch.tensor(wl.acc_w, device="cuda")
        logits = torch.empty((len(b.rows), cfg.vocab), device="cuda")
        emb = torch.full((len(b.chunks), cfg.d_model), float("nan"), device="cuda")
        R.step(dm, dm, b, kv, kv, S, Wc, logits, emb, ws)
        torch.cuda.synchronize()
        assert ws.device_error() == 0
        outs.append((logits.cpu(), emb.cpu(), S.cpu(), Wc.cpu(), kv.k.view(torch.int16).clone(),
                     kv.v.view(torch.int16).clone()))
    for a, c in zip(*outs):
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           c.view(torch.int32) if c.dtype == torch.float32 else c)
