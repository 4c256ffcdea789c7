"""GPU parity of generation prefill chunks and the greedy sampler against the float64 oracle.

A generation request's prompt runs through the step as chunks (the third item type of the
Section 3.2 batch unit) beside embedding chunks and decode rows; the prompt's final chunk yields
logits for its last row, and generation continues with decode rows.  Both sides are fed the
token the oracle's greedy sampler picks, so the two runs never diverge.  The device sampler is
checked bit for bit against the oracle's argmax of the same fp32 logits (the decision taken in
the same precision on both sides), and against the oracle's own choice wherever the oracle's
top-two margin exceeds the logits tolerance.
"""
import numpy as np
import pytest
import torch

from oracle import greedy_token
from workload import (Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, draw_tokens,
                      make_weights, tiny_config)
from tests.parity import Pair, TOL
from paper_2609_25405_amd import runtime as R

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _sample(logits: torch.Tensor, n: int) -> np.ndarray:
    out = torch.full((max(1, n),), -1, dtype=torch.int32, device="cuda")
    R.sample_greedy(logits[:n].contiguous(), out[:n])
    torch.cuda.synchronize()
    return out[:n].cpu().numpy().astype(np.int64)


def _check_sampler(logits: torch.Tensor, ref_logits: np.ndarray, dtype: str) -> np.ndarray:
    """Device argmax == oracle argmax of the device's logits; == oracle's token where the
    oracle's top-two margin is wider than the tolerance allows the device to move."""
    n = ref_logits.shape[0]
    got = _sample(logits, n)
    g = logits[:n].cpu().numpy()
    np.testing.assert_array_equal(got, greedy_token(g))
    want = greedy_token(ref_logits)
    top2 = np.sort(ref_logits, axis=1)[:, -2:]
    scale = np.max(np.abs(ref_logits), axis=1)
    clear = (top2[:, 1] - top2[:, 0]) > 2 * TOL[dtype]["rel"] * scale
    np.testing.assert_array_equal(got[clear], want[clear])
    return want


def _generation_run(pair: Pair, cfg, seed: int, emb_seq: int, prompts, dec_seq: int, dec_ctx: int):
    """Three steps: prompt chunks (one prompt finishing in step 1, one in step 2) beside an
    embedding request in two chunks and a running decode row, then decode of every request.
    ``prompts`` = {seq: (first chunk len, second chunk len or 0)}."""
    (s_a, (a1, a2)), (s_b, (b1, b2)) = sorted(prompts.items())
    assert a2 > 0 and b2 == 0
    V = cfg.vocab
    # step 1: emb [0, 100) mean; prompt A [0, a1); prompt B [0, b1) final; decode row
    ch1 = [EmbChunk(emb_seq, 0, 100, False, "mean")]
    gen1 = [GenChunk(s_a, 0, a1, False), GenChunk(s_b, 0, b1, True)]
    rows1 = [DecodeRow(dec_seq, dec_ctx)]
    ids1 = draw_tokens(seed, 1, 100 + a1 + b1 + 1, V)
    ref1, lg1, _ = pair.step(Batch(ch1, rows1, ids1, gen1))
    t1 = _check_sampler(lg1, ref1["logits"], pair.dtype)      # rows: prompt B, decode row
    # step 2: emb [100, 160) final; prompt A [a1, a1 + a2) final; decode B and the decode row
    ch2 = [EmbChunk(emb_seq, 100, 60, True, "mean")]
    gen2 = [GenChunk(s_a, a1, a2, True)]
    rows2 = [DecodeRow(s_b, b1), DecodeRow(dec_seq, dec_ctx + 1)]
    ids2 = np.concatenate([draw_tokens(seed, 2, 60 + a2, V), t1]).astype(np.int32)
    ref2, lg2, _ = pair.step(Batch(ch2, rows2, ids2, gen2))
    t2 = _check_sampler(lg2, ref2["logits"], pair.dtype)      # rows: prompt A, decode B, decode row
    # step 3: decode only, every generation request
    rows3 = [DecodeRow(s_a, a1 + a2), DecodeRow(s_b, b1 + 1), DecodeRow(dec_seq, dec_ctx + 2)]
    ref3, lg3, _ = pair.step(Batch([], rows3, t2.astype(np.int32)))
    _check_sampler(lg3, ref3["logits"], pair.dtype)


@pytest.mark.parametrize("dtype,qk_std", [("f32", None), ("bf16", 0.09)])
def test_prompt_chunks_then_greedy_decode(dtype, qk_std):
    """Tiny decoder, one model and one cache: prompts of 37 + 53 and 20 tokens."""
    cfg = tiny_config(dtype)
    W = make_weights(cfg, 31, qk_std=qk_std)
    n_seq, max_blocks = 6, 16
    pk = PagedKV(cfg, n_seq * max_blocks + 5, n_seq, max_blocks, 31)
    pk.fill_random(3, 50, 32)
    for s in range(n_seq):
        pk.reserve(s, 200)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=256, max_chunks=3, max_decode=3, max_ctx=256)
    _generation_run(pair, cfg, 31, emb_seq=0, prompts={1: (37, 53), 2: (20, 0)}, dec_seq=3, dec_ctx=50)
    print(pair.report, flush=True)


def test_prompt_chunks_two_models_two_caches():
    """Separate embedding model and generator with separate caches: the prompt chunks must read
    and append the generator's cache, and sequence numbers of the two caches are independent."""
    cfg = tiny_config("bf16")
    We = make_weights(cfg, 41, model_tag=1, qk_std=0.09)
    Wg = make_weights(cfg, 41, model_tag=2, qk_std=0.09)
    pe = PagedKV(cfg, 60, 4, 16, 1)
    pg = PagedKV(cfg, 70, 4, 16, 2)
    pg.fill_random(3, 77, 5)
    for s in range(4):
        pe.reserve(s, 200)
        pg.reserve(s, 200)
    pair = Pair(cfg, We, pe, cfg, Wg, pg)
    pair.workspace(max_tokens=256, max_chunks=3, max_decode=3, max_ctx=256)
    # embedding seq 1 and prompt seq 1 live in different caches
    _generation_run(pair, cfg, 41, emb_seq=1, prompts={1: (45, 19), 2: (64, 0)}, dec_seq=3, dec_ctx=77)
    print(pair.report, flush=True)


def test_prompt_chunks_gqa_long_offsets():
    """Group-4 heads of 128 dims: prompt chunks of several 32-token tiles, the second starting
    at offset 300 behind cached keys, with a multi-split decode row."""
    cfg = ModelConfig(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                      vocab=512, dtype="bf16")
    W = make_weights(cfg, 51, qk_std=0.06)
    n_seq, max_blocks = 6, 96
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, 51)
    pk.fill_random(4, 1100, 52)       # 1101 keys: two splits of 256-key chunks on the bf16 path
    for s in range(n_seq):
        pk.reserve(s, 800)
    pk.reserve(4, 1104)
    pair = Pair(cfg, W, pk)
    pair.workspace(max_tokens=600, max_chunks=3, max_decode=3, max_ctx=1200)
    _generation_run(pair, cfg, 51, emb_seq=0, prompts={1: (300, 77), 2: (129, 0)}, dec_seq=4, dec_ctx=1100)
    print(pair.report, flush=True)


@pytest.mark.parametrize("vocab", [1, 7, 1000, 32000])
@pytest.mark.parametrize("aligned", [True, False])
def test_sampler_matches_oracle_argmax(vocab, aligned):
    """Ties (lowest index), NaN (first NaN wins), -inf rows and ragged vocab sizes, with the
    16-byte path (aligned rows) and the scalar path (rows off a 16-byte boundary)."""
    rng = np.random.default_rng(vocab)
    rows = 67
    x = rng.standard_normal((rows, vocab)).astype(np.float32)
    x = np.round(x * 4) / 4          # many exact ties
    if vocab > 3:
        x[1, :] = 0.5                # all equal: index 0
        x[2, vocab - 1] = 100.0      # maximum at the last column
        x[2, vocab // 2] = 100.0     # tie at an earlier column
        x[3, vocab // 3] = np.nan
        x[3, vocab - 2] = np.nan     # first NaN wins
        x[4, :] = -np.inf
        x[5, :] = -np.inf
        x[5, vocab - 1] = -1e30
    buf = torch.zeros(rows * vocab + 4, dtype=torch.float32, device="cuda")
    off = 0 if aligned else 1
    lg = buf[off:off + rows * vocab].view(rows, vocab)
    lg.copy_(torch.from_numpy(x))
    got = _sample(lg, rows)
    np.testing.assert_array_equal(got, greedy_token(x.astype(np.float64)))
    # empty launch is a no-op
    R.sample_greedy(lg[:0], torch.zeros(0, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()


def test_prompt_chunk_writes_the_cache_of_a_kv_only_chunk():
    """With one model and one cache, a non-final prompt chunk is the same computation as a
    KV-only embedding chunk over the same tokens at the same batch rows: the caches the two
    steps leave must agree bit for bit (the prompt chunk adds no pooling and no logits)."""
    cfg = tiny_config("bf16")
    W = make_weights(cfg, 61, qk_std=0.09)
    ids = draw_tokens(61, 1, 100 + 37 + 20 + 1, cfg.vocab)
    caches = []
    for kind in ("prompt", "kv_only"):
        pk = PagedKV(cfg, 6 * 16 + 5, 6, 16, 61)
        pk.fill_random(3, 50, 62)
        for s in range(6):
            pk.reserve(s, 200)
        pair = Pair(cfg, W, pk)
        pair.workspace(max_tokens=256, max_chunks=3, max_decode=1, max_ctx=256)
        head = [EmbChunk(0, 0, 100, False, "mean")]
        if kind == "prompt":
            b = Batch(head, [DecodeRow(3, 50)], ids, [GenChunk(1, 0, 37, False), GenChunk(2, 0, 20, False)])
        else:
            b = Batch(head + [EmbChunk(1, 0, 37, False, "none"), EmbChunk(2, 0, 20, False, "none")],
                      [DecodeRow(3, 50)], ids)
        pair.step(b)
        caches.append((pair.dkv_e.k.view(torch.int16).clone(), pair.dkv_e.v.view(torch.int16).clone()))
    assert torch.equal(caches[0][0], caches[1][0]) and torch.equal(caches[0][1], caches[1][1])
