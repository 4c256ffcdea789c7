"""Pins of the CPU oracle against things other than itself (no GPU).

* an independent scalar-loop forward (tests/bruteforce.py) at tiny shapes;
* a third-party implementation of the same model family (transformers' Llama);
* closed forms and invariants of rotary embedding, softmax attention and pooling;
* the equivalences the paper states for the method (Section 3.3 and the pooling
  equivalence table in the appendix): chunked embedding with incremental pooling
  equals single-pass embedding, decode through the cache equals recomputation
  from the prefix, and a mixed batch equals each request run alone.
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import OracleKV, StepError, step_oracle
from workload import (Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, draw_tokens,
                      draw_token_weights, make_weights, tiny_config)
from tests import bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def micro_config(**kw):
    base = dict(n_layers=2, d_model=16, n_q_heads=4, n_kv_heads=2, head_dim=4, d_ff=24,
                vocab=32, dtype="f32")
    base.update(kw)
    return ModelConfig(**base)


def sharp_weights(cfg, seed):
    # larger spread so attention is far from uniform and position errors show
    return make_weights(cfg, seed, std=0.3, qk_std=0.6)


# ---------------------------------------------------------------------------
# forward pass vs independent implementations
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("nkv", [1, 2, 4])
def test_forward_matches_scalar_loops(nkv):
    cfg = micro_config(n_kv_heads=nkv)
    W = sharp_weights(cfg, 5 + nkv)
    ids = draw_tokens(3, nkv, 7, cfg.vocab)
    H = oracle.forward_full(cfg, W, ids)
    Hb = np.array(bruteforce.forward(cfg, W, ids.tolist()))
    np.testing.assert_allclose(H, Hb, rtol=1e-11, atol=1e-12)
    lg = oracle.lm_logits(W, H[-1])
    np.testing.assert_allclose(lg, np.array(bruteforce.logits(W, Hb[-1].tolist())), rtol=1e-11,
                               atol=1e-12)


def _hf_llama(cfg, W):
    torch = pytest.importorskip("torch")
    tf = pytest.importorskip("transformers")
    c = tf.LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model,
                       intermediate_size=cfg.d_ff, num_hidden_layers=cfg.n_layers,
                       num_attention_heads=cfg.n_q_heads, num_key_value_heads=cfg.n_kv_heads,
                       head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_base,
                       tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                       max_position_embeddings=4096)
    c._attn_implementation = "eager"
    m = tf.LlamaForCausalLM(c).to(torch.float64).eval()
    t = lambda a: torch.tensor(np.asarray(a, np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(W["tok_emb"]))
        m.model.norm.weight.copy_(t(W["final_norm"]))
        m.lm_head.weight.copy_(t(W["lm_head"]))
        for l, lw in enumerate(W["layers"]):
            L = m.model.layers[l]
            qd, kd = cfg.q_dim, cfg.kv_dim
            L.self_attn.q_proj.weight.copy_(t(lw["w_qkv"][:qd]))
            L.self_attn.k_proj.weight.copy_(t(lw["w_qkv"][qd:qd + kd]))
            L.self_attn.v_proj.weight.copy_(t(lw["w_qkv"][qd + kd:]))
            L.self_attn.o_proj.weight.copy_(t(lw["w_o"]))
            L.mlp.gate_proj.weight.copy_(t(lw["w_gate"]))
            L.mlp.up_proj.weight.copy_(t(lw["w_up"]))
            L.mlp.down_proj.weight.copy_(t(lw["w_down"]))
            L.input_layernorm.weight.copy_(t(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(t(lw["mlp_norm"]))
    return m


@pytest.mark.parametrize("shape", ["micro_gqa", "tiny"])
def test_forward_matches_transformers_llama(shape):
    torch = pytest.importorskip("torch")
    if shape == "micro_gqa":
        cfg = micro_config(n_kv_heads=2, head_dim=8, d_model=32, d_ff=40)
        n = 40
    else:
        cfg = tiny_config()
        n = 70
    W = sharp_weights(cfg, 11)
    ids = draw_tokens(4, 0, n, cfg.vocab)
    m = _hf_llama(cfg, W)
    with torch.no_grad():
        out = m(torch.tensor(ids[None].astype(np.int64)), output_hidden_states=True)
    H = oracle.forward_full(cfg, W, ids)
    logits = oracle.lm_logits(W, H)
    # transformers evaluates the rotary angles in float32 (about 1e-7 rad per unit of
    # position), which sharp attention amplifies to ~2e-5 of the output scale; a wrong
    # convention (pairing, sign, head grouping, norm placement) is off by O(1)
    ref = out.logits[0].numpy()
    assert np.max(np.abs(logits - ref)) <= 1e-4 * np.max(np.abs(ref))
    Href = out.hidden_states[-1][0].numpy()
    assert np.max(np.abs(H - Href)) <= 1e-4 * np.max(np.abs(Href))


# ---------------------------------------------------------------------------
# closed forms and invariants
# ---------------------------------------------------------------------------
def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((1, 3, 64))
    np.testing.assert_array_equal(oracle.rope_rotate(x, np.array([0]), 10000.0), x)
    for p in (1, 17, 1000, 8191):
        y = oracle.rope_rotate(x, np.array([p]), 10000.0)
        np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1),
                                   rtol=1e-13)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    dots = []
    for m_, n_ in ((5, 2), (105, 102), (4003, 4000)):
        qm = oracle.rope_rotate(q, np.array([m_]), 10000.0)
        kn = oracle.rope_rotate(k, np.array([n_]), 10000.0)
        dots.append(float(np.sum(qm * kn)))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-9)
    # the first pair rotates by exactly `pos` radians, the last by pos * base^(-(hd-2)/hd)
    e = np.zeros((1, 1, 64))
    e[0, 0, 0] = 1.0
    y = oracle.rope_rotate(e, np.array([3]), 10000.0)
    assert abs(y[0, 0, 0] - math.cos(3.0)) < 1e-15 and abs(y[0, 0, 32] - math.sin(3.0)) < 1e-15


def test_attention_closed_forms():
    rng = np.random.default_rng(1)
    n, nq, nkv, hd = 9, 4, 2, 8
    q = rng.standard_normal((n, nq, hd))
    k = rng.standard_normal((n, nkv, hd))
    v = rng.standard_normal((n, nkv, hd))
    pos = np.arange(n)
    o = oracle.causal_gqa_attention(q, k, v, pos, pos).reshape(n, nq, hd)
    # the first query sees one key: output is that key's value
    for h in range(nq):
        np.testing.assert_allclose(o[0, h], v[0, h // 2], rtol=1e-14)
    # zero queries give uniform weights: the mean of the visible values
    o0 = oracle.causal_gqa_attention(np.zeros_like(q), k, v, pos, pos).reshape(n, nq, hd)
    for i in range(n):
        np.testing.assert_allclose(o0[i, 3], v[:i + 1, 1].mean(axis=0), rtol=1e-13)
    # value component = key position: uniform weights give position / 2
    v2 = np.zeros_like(v)
    v2[:, :, 0] = pos[:, None]
    o2 = oracle.causal_gqa_attention(np.zeros_like(q), k, v2, pos, pos).reshape(n, nq, hd)
    np.testing.assert_allclose(o2[:, 0, 0], pos / 2.0, rtol=1e-14)


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(2)
    n, nq, nkv, hd = 13, 8, 2, 16
    q = rng.standard_normal((n, nq, hd))
    k = rng.standard_normal((n, nkv, hd))
    v = rng.standard_normal((n, nkv, hd))
    pos = np.arange(n)
    o = oracle.causal_gqa_attention(q, k, v, pos, pos).reshape(n, nq, hd)
    tq = torch.tensor(q).permute(1, 0, 2)[None]
    tk = torch.tensor(k).permute(1, 0, 2)[None]
    tv = torch.tensor(v).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    np.testing.assert_allclose(o, ref[0].permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_rmsnorm_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 32))
    g = rng.standard_normal(32)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (32,), torch.tensor(g), eps=1e-5)
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref.numpy(), rtol=1e-13)


def test_zero_layer_model_pools_normed_embeddings():
    cfg = micro_config(n_layers=0)
    W = make_weights(cfg, 4)
    ids = draw_tokens(9, 1, 11, cfg.vocab)
    E = W["tok_emb"][ids].astype(np.float64)
    normed = E / np.sqrt((E * E).mean(axis=1, keepdims=True) + cfg.rms_eps)
    mean = normed.mean(axis=0)
    out = oracle.embed_single_pass(cfg, W, ids, "mean")
    np.testing.assert_allclose(out, mean / np.linalg.norm(mean), rtol=1e-13)
    assert abs(np.linalg.norm(out) - 1.0) < 1e-14
    same = oracle.pool_single_pass(np.tile(normed[:1], (6, 1)), "mean")
    np.testing.assert_allclose(same, normed[0], rtol=1e-15)
    np.testing.assert_array_equal(oracle.l2_normalize(np.zeros(4)), np.zeros(4))


# ---------------------------------------------------------------------------
# the paper's equivalences, through the step contract
# ---------------------------------------------------------------------------
def _fresh_kv(cfg, n_seq, max_tokens, seed, n_pages=None):
    P = cfg.page_size
    mb = -(-max_tokens // P)
    if n_pages is None:
        n_pages = n_seq * mb + 5
    pk = PagedKV(cfg, n_pages, n_seq, mb, seed)
    return pk


def run_chunked_embedding(cfg, W, ids, C, head, seq=0, seed=0, weights=None):
    pk = _fresh_kv(cfg, 1 + seq, len(ids), seed)
    pk.reserve(seq, len(ids))
    kv = OracleKV.from_paged(pk)
    S = np.zeros((1 + seq, cfg.d_model))
    Wc = np.zeros(1 + seq)
    out = None
    rows = []
    for off in range(0, len(ids), C):
        ln = min(C, len(ids) - off)
        b = Batch(chunks=[EmbChunk(seq, off, ln, last=off + ln == len(ids), pool=head)],
                  rows=[], token_ids=ids[off:off + ln],
                  token_weights=None if weights is None else weights[off:off + ln],
                  hidden_stride=len(ids))
        r = step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        S, Wc = r["acc_sum"], r["acc_w"]
        assert Wc[seq] == off + ln
        out = r["out_emb"][0]
        if head == "buffer":
            rows.append(r["hidden"][0])
    if head == "buffer":
        return np.concatenate(rows), kv, S, Wc
    return out, kv, S, Wc


@pytest.mark.parametrize("head", ["mean", "last", "cls"])
@pytest.mark.parametrize("C", [1, 7, 16, 23])
def test_chunked_equals_single_pass(head, C):
    cfg = micro_config()
    W = sharp_weights(cfg, 21)
    ids = draw_tokens(5, 2, 23, cfg.vocab)
    ref = oracle.embed_single_pass(cfg, W, ids, head)
    got, _, _, _ = run_chunked_embedding(cfg, W, ids, C, head)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_pooling_equivalence_table_protocol():
    """Appendix, pooling-equivalence table: mean, CLS and weighted-mean heads at C = 256/512/1024
    (weighted mean with seeded uniform weights: the paper does not say which weights it used).

    The paper's worst observed agreement (fixture) bounds what the oracle must meet
    on a random-weight model; in float64 the two paths agree to rounding.
    """
    bounds = {}
    with open(os.path.join(GOLDEN, "pooling_equivalence.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            head, C, min_cos, rel_l2_p99 = line.split()
            bounds[(head, int(C))] = (float(min_cos), float(rel_l2_p99))
    assert len(bounds) == 9
    cfg = micro_config(n_layers=1, d_model=32, head_dim=8, d_ff=32, vocab=64)
    W = sharp_weights(cfg, 31)
    ids = draw_tokens(6, 3, 1100, cfg.vocab)
    w = draw_token_weights(6, 3, len(ids))
    for (head, C), (min_cos, p99) in bounds.items():
        head = "wmean" if head == "weighted_mean" else head
        tw = w if head == "wmean" else None
        ref = oracle.embed_single_pass(cfg, W, ids, head, tw)
        got, _, _, _ = run_chunked_embedding(cfg, W, ids, C, head, weights=tw)
        cos = float(got @ ref / (np.linalg.norm(got) * np.linalg.norm(ref)))
        rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        assert cos >= min_cos and rel <= p99
        assert rel < 1e-12


def test_decode_through_cache_equals_recompute():
    cfg = micro_config()
    W = sharp_weights(cfg, 41)
    prompt = draw_tokens(7, 0, 21, cfg.vocab)
    nxt = draw_tokens(7, 1, 4, cfg.vocab)
    pk = _fresh_kv(cfg, 3, 40, 1)
    pk.reserve(2, 40)
    kv = OracleKV.from_paged(pk)
    S = np.zeros((3, cfg.d_model))
    Wc = np.zeros(3)
    # prompt written by a cache-only chunk, then one decode token per step
    b = Batch(chunks=[EmbChunk(2, 0, len(prompt), False, "none")], rows=[], token_ids=prompt)
    step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
    seqs = list(prompt)
    for i, t in enumerate(nxt):
        b = Batch(chunks=[], rows=[DecodeRow(2, len(seqs))], token_ids=np.array([t], np.int32))
        r = step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        seqs.append(int(t))
        ref = oracle.decode_full_recompute(cfg, W, np.array(seqs))
        np.testing.assert_allclose(r["logits"][0], ref, rtol=1e-11, atol=1e-13)


def test_mixed_batch_equals_each_request_alone_and_permutes():
    cfg = micro_config()
    W = sharp_weights(cfg, 51)
    n_seq = 5
    toks = {s: draw_tokens(8, s, 30, cfg.vocab) for s in range(n_seq)}

    def setup():
        pk = _fresh_kv(cfg, n_seq, 64, 2)
        for s in range(n_seq):
            pk.reserve(s, 40)
        kv = OracleKV.from_paged(pk)
        S = np.zeros((n_seq, cfg.d_model))
        Wc = np.zeros(n_seq)
        # sequences 2..4 get a prompt through cache-only chunks; 0 and 1 start an embedding
        for s in (2, 3, 4):
            n = 10 + 3 * s
            b = Batch([EmbChunk(s, 0, n, False, "none")], [], toks[s][:n])
            step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        return kv, S, Wc

    chunks = [EmbChunk(0, 0, 9, False, "mean"), EmbChunk(1, 0, 14, True, "last")]
    rows = [DecodeRow(2, 16), DecodeRow(3, 19), DecodeRow(4, 22)]
    ids_c = [toks[0][:9], toks[1][:14]]
    ids_r = [toks[2][16:17], toks[3][19:20], toks[4][22:23]]
    kv, S, Wc = setup()
    mixed = step_oracle((cfg, W), (cfg, W), Batch(chunks, rows, np.concatenate(ids_c + ids_r)),
                        kv, kv, S, Wc)
    # alone
    kv1, S1, W1 = setup()
    for i, c in enumerate(chunks):
        r = step_oracle((cfg, W), (cfg, W), Batch([c], [], ids_c[i]), kv1, kv1, S1, W1)
        S1, W1 = r["acc_sum"], r["acc_w"]
        if c.last:
            np.testing.assert_allclose(mixed["out_emb"][i], r["out_emb"][0], rtol=1e-13)
        np.testing.assert_allclose(mixed["acc_sum"][c.seq], S1[c.seq], rtol=1e-13)
    for j, row in enumerate(rows):
        r = step_oracle((cfg, W), (cfg, W), Batch([], [row], ids_r[j]), kv1, kv1, S1, W1)
        np.testing.assert_allclose(mixed["logits"][j], r["logits"][0], rtol=1e-12)
    np.testing.assert_array_equal(np.isnan(kv.k), np.isnan(kv1.k))
    # permuted order permutes outputs
    kv2, S2, W2 = setup()
    perm = Batch(chunks[::-1], rows[::-1], np.concatenate(ids_c[::-1] + ids_r[::-1]))
    r2 = step_oracle((cfg, W), (cfg, W), perm, kv2, kv2, S2, W2)
    np.testing.assert_allclose(r2["logits"][::-1], mixed["logits"], rtol=1e-12)
    np.testing.assert_allclose(r2["out_emb"][0], mixed["out_emb"][1], rtol=1e-12)


def test_page_coverage_closed_form():
    """Zero query weights make attention uniform; value channel 0 = key position.

    Then the attention output's channel 0 is exactly pos / 2 for every row, so a
    dropped, duplicated or misplaced key (wrong page, wrong slot) changes it.
    """
    cfg = micro_config(n_layers=1, n_kv_heads=2)
    W = make_weights(cfg, 61)
    lw = W["layers"][0]
    lw["w_qkv"][:cfg.q_dim] = 0.0
    pk = _fresh_kv(cfg, 2, 80, 3, n_pages=20)
    pk.reserve(1, 70)
    # fill positions 0..68 with value channel 0 = position
    for p in range(69):
        page = pk.block_table[1, p // 16]
        pk.k[0, page, :, p % 16, :] = 0.5
        pk.v[0, page, :, p % 16, :] = 0.0
        pk.v[0, page, :, p % 16, 0] = p
    kv = OracleKV.from_paged(pk)
    # capture the attention output by reading it back from the oracle's internals:
    # with Wo = identity-like selection we instead check the cached value directly
    from oracle.model import causal_gqa_attention
    K, V = kv.read(0, 1, 69)
    q = np.zeros((1, cfg.n_q_heads, cfg.head_dim))
    o = causal_gqa_attention(q, K, V, np.array([68]), np.arange(69)).reshape(cfg.n_q_heads, -1)
    assert o[0, 0] == 34.0
    assert np.all(np.isnan(kv.k[0, pk.block_table[1, 4], :, 5:, :]))


def test_contract_errors():
    cfg = micro_config()
    W = make_weights(cfg, 71)
    pk = _fresh_kv(cfg, 3, 32, 4)
    pk.reserve(0, 32)
    kv = OracleKV.from_paged(pk)
    S = np.zeros((3, cfg.d_model))
    Wc = np.zeros(3)
    ids = np.arange(8, dtype=np.int32)

    def kind(b, S=S, Wc=Wc):
        with pytest.raises(StepError) as e:
            step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        return e.value.kind

    assert kind(Batch([EmbChunk(0, 0, 4, False), EmbChunk(0, 4, 4, False)], [], ids)) == "dupseq"
    assert kind(Batch([EmbChunk(0, 0, 7, False)], [DecodeRow(0, 3)], ids)) == "dupseq"
    assert kind(Batch([EmbChunk(3, 0, 8, False)], [], ids)) == "desc"
    assert kind(Batch([EmbChunk(0, 0, 8, True, "none")], [], ids)) == "desc"
    assert kind(Batch([EmbChunk(0, 0, 9, False)], [], ids)) == "desc"
    assert kind(Batch([EmbChunk(0, 30, 8, False)], [], ids)) == "capacity"
    assert kind(Batch([EmbChunk(0, 8, 8, False)], [], ids)) == "device"   # W = 0, offset 8
    assert kind(Batch([EmbChunk(1, 0, 8, False)], [], ids)) == "device"   # no pages
    assert kind(Batch([], [DecodeRow(1, -1)], ids[:1])) == "desc"
    bad = ids.copy()
    bad[0] = cfg.vocab
    assert kind(Batch([EmbChunk(0, 0, 8, False)], [], bad)) == "desc"


# ---------------------------------------------------------------------------
# generation prefill chunks (the batch unit's third item type) and greedy sampling
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("C", [1, 7, 16, 21])
@pytest.mark.parametrize("nkv", [4, 2])
def test_prompt_chunks_then_greedy_decode_equal_recompute(C, nkv):
    """A prompt fed as generation prefill chunks of C tokens gives, on its final chunk, the
    next-token logits of the whole prompt recomputed without a cache; greedy decoding through
    the cache then matches full recompute of prompt + generated tokens at every step."""
    cfg = micro_config(n_kv_heads=nkv)
    W = sharp_weights(cfg, 61)
    prompt = draw_tokens(9, 0, 21, cfg.vocab)
    pk = _fresh_kv(cfg, 2, 40, 3)
    pk.reserve(1, 40)
    kv = OracleKV.from_paged(pk)
    S, Wc = np.zeros((2, cfg.d_model)), np.zeros(2)
    for off in range(0, len(prompt), C):
        ln = min(C, len(prompt) - off)
        last = off + ln == len(prompt)
        b = Batch(token_ids=prompt[off:off + ln], gen_chunks=[GenChunk(1, off, ln, last)])
        r = step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        assert r["logits"].shape == ((1, cfg.vocab) if last else (0, 0))
        np.testing.assert_array_equal(r["acc_w"], Wc)   # prompts touch no pooling state
    seqs = list(prompt)
    np.testing.assert_allclose(r["logits"][0], oracle.decode_full_recompute(cfg, W, np.array(seqs)),
                               rtol=1e-11, atol=1e-13)
    tok = int(oracle.greedy_token(r["logits"])[0])
    for _ in range(3):
        b = Batch(rows=[DecodeRow(1, len(seqs))], token_ids=np.array([tok], np.int32))
        r = step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        seqs.append(tok)
        np.testing.assert_allclose(r["logits"][0], oracle.decode_full_recompute(cfg, W, np.array(seqs)),
                                   rtol=1e-11, atol=1e-13)
        tok = int(oracle.greedy_token(r["logits"])[0])


def test_three_item_types_equal_each_request_alone():
    """Embedding chunks, prompt chunks and decode rows in one batch give the outputs each
    request gives alone; logits rows are the final prompt chunks' last rows (in order), then
    the decode rows."""
    cfg = micro_config()
    W = sharp_weights(cfg, 71)
    toks = {s: draw_tokens(10, s, 30, cfg.vocab) for s in range(6)}

    def setup():
        pk = _fresh_kv(cfg, 6, 64, 4)
        for s in range(6):
            pk.reserve(s, 40)
        kv = OracleKV.from_paged(pk)
        for s in (4, 5):     # generation requests with a cached prompt, now decoding
            b = Batch([EmbChunk(s, 0, 12, False, "none")], [], toks[s][:12])
            step_oracle((cfg, W), (cfg, W), b, kv, kv, np.zeros((6, cfg.d_model)), np.zeros(6))
        return kv, np.zeros((6, cfg.d_model)), np.zeros(6)

    chunks = [EmbChunk(0, 0, 8, True, "mean")]
    gens = [GenChunk(2, 0, 9, True), GenChunk(3, 0, 6, False)]
    rows = [DecodeRow(4, 12), DecodeRow(5, 12)]
    ids = [toks[0][:8], toks[2][:9], toks[3][:6], toks[4][12:13], toks[5][12:13]]
    kv, S, Wc = setup()
    mixed = step_oracle((cfg, W), (cfg, W), Batch(chunks, rows, np.concatenate(ids), gens),
                        kv, kv, S, Wc)
    assert mixed["logits"].shape == (3, cfg.vocab)
    kv1, S1, W1 = setup()
    alone = [step_oracle((cfg, W), (cfg, W), Batch(chunks, [], ids[0]), kv1, kv1, S1, W1),
             step_oracle((cfg, W), (cfg, W), Batch(token_ids=ids[1], gen_chunks=[gens[0]]), kv1, kv1, S1, W1),
             step_oracle((cfg, W), (cfg, W), Batch(token_ids=ids[2], gen_chunks=[gens[1]]), kv1, kv1, S1, W1),
             step_oracle((cfg, W), (cfg, W), Batch([], [rows[0]], ids[3]), kv1, kv1, S1, W1),
             step_oracle((cfg, W), (cfg, W), Batch([], [rows[1]], ids[4]), kv1, kv1, S1, W1)]
    np.testing.assert_allclose(mixed["out_emb"][0], alone[0]["out_emb"][0], rtol=1e-13)
    assert alone[2]["logits"].shape[0] == 0
    for j, k in enumerate((1, 3, 4)):
        np.testing.assert_allclose(mixed["logits"][j], alone[k]["logits"][0], rtol=1e-12)
    np.testing.assert_array_equal(kv.k, kv1.k)


def test_prompt_chunk_contract_errors():
    cfg = micro_config()
    W = sharp_weights(cfg, 81)
    pk = _fresh_kv(cfg, 4, 32, 5)
    for s in range(4):
        pk.reserve(s, 32)
    kv = OracleKV.from_paged(pk)
    z = (np.zeros((4, cfg.d_model)), np.zeros(4))
    ids = draw_tokens(11, 0, 40, cfg.vocab)
    bad = [
        (Batch([], [DecodeRow(1, 3)], ids[:5], [GenChunk(1, 0, 4, False)]), "dupseq"),   # prompt + decode, one seq
        (Batch([EmbChunk(2, 0, 4, False)], [], ids[:8], [GenChunk(2, 0, 4, False)]), "dupseq"),  # shared cache
        (Batch(token_ids=ids[:4], gen_chunks=[GenChunk(1, 30, 4, True)]), "capacity"),
        (Batch(token_ids=ids[:4], gen_chunks=[GenChunk(4, 0, 4, True)]), "desc"),      # seq out of range
        (Batch(token_ids=ids[:0], gen_chunks=[GenChunk(1, 0, 0, True)]), "desc"),      # empty chunk
        (Batch(token_ids=ids[:3], gen_chunks=[GenChunk(1, 0, 4, True)]), "desc"),      # token count
    ]
    for b, kind in bad:
        with pytest.raises(StepError) as e:
            step_oracle((cfg, W), (cfg, W), b, kv, kv, *z)
        assert e.value.kind == kind, (b, e.value.kind)
    nohead = cfg.replace(has_lm_head=False)
    Wn = make_weights(nohead, 81)
    with pytest.raises(StepError) as e:
        step_oracle((nohead, Wn), (nohead, Wn), Batch(token_ids=ids[:4], gen_chunks=[GenChunk(1, 0, 4, True)]),
                    kv, kv, *z)
    assert e.value.kind == "desc"


def test_greedy_token_takes_the_lowest_index_on_ties():
    logits = np.array([[0.5, 2.0, 2.0, -1.0], [3.0, 3.0, 3.0, 3.0], [-np.inf, -5.0, -7.0, -5.0]])
    np.testing.assert_array_equal(oracle.greedy_token(logits), [1, 0, 1])


# ---------------------------------------------------------------------------
# weighted-mean and buffered heads (Section 3.3, Eq. (1)-(2) with general weights)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("C", [1, 7, 16, 23])
def test_weighted_mean_chunked_equals_definition(C):
    """Chunked weighted mean equals sum_j w_j H_j / sum_j w_j of the single-pass hidden
    states, L2-normalised, with the weight sum written out here, not taken from the oracle."""
    cfg = micro_config()
    W = sharp_weights(cfg, 41)
    ids = draw_tokens(7, 1, 23, cfg.vocab)
    w = draw_token_weights(7, 1, 23).astype(np.float64)
    H = oracle.forward_full(cfg, W, ids)
    v = (w[:, None] * H).sum(axis=0) / w.sum()
    want = v / np.linalg.norm(v)
    got, _, S, Wc = run_chunked_embedding(cfg, W, ids, C, "wmean", weights=w)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)
    assert Wc[0] == 23                      # the state keeps counting tokens


def test_weighted_mean_special_cases():
    """Unit weights give the mean head; a one-hot weight on the last (first) token gives the
    last-token (CLS) head; scaling every weight changes nothing; all-zero weights give the
    zero vector."""
    cfg = micro_config()
    W = sharp_weights(cfg, 43)
    ids = draw_tokens(8, 1, 19, cfg.vocab)
    mean = oracle.embed_single_pass(cfg, W, ids, "mean")
    last = oracle.embed_single_pass(cfg, W, ids, "last")
    cls = oracle.embed_single_pass(cfg, W, ids, "cls")
    ones = np.ones(19)
    onehot_last = np.zeros(19)
    onehot_last[-1] = 1.0
    onehot_first = np.zeros(19)
    onehot_first[0] = 2.5
    w = draw_token_weights(8, 2, 19).astype(np.float64)
    for C in (5, 19):
        np.testing.assert_allclose(run_chunked_embedding(cfg, W, ids, C, "wmean", weights=ones)[0], mean,
                                   rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(run_chunked_embedding(cfg, W, ids, C, "wmean", weights=onehot_last)[0],
                                   last, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(run_chunked_embedding(cfg, W, ids, C, "wmean", weights=onehot_first)[0],
                                   cls, rtol=1e-12, atol=1e-13)
        a = run_chunked_embedding(cfg, W, ids, C, "wmean", weights=w)[0]
        b = run_chunked_embedding(cfg, W, ids, C, "wmean", weights=3.0 * w)[0]
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)
        z = run_chunked_embedding(cfg, W, ids, C, "wmean", weights=np.zeros(19))[0]
        np.testing.assert_array_equal(z, np.zeros(cfg.d_model))


@pytest.mark.parametrize("C", [1, 6, 19])
def test_buffered_head_equals_single_pass_rows(C):
    """The buffered head hands back every final-normed hidden row; concatenated over the chunks
    they are the single-pass hidden states, so any head applied to them (here an
    element-wise max, which no streaming head of the paper computes) matches."""
    cfg = micro_config()
    W = sharp_weights(cfg, 47)
    ids = draw_tokens(9, 1, 19, cfg.vocab)
    H = oracle.forward_full(cfg, W, ids)
    rows, _, _, Wc = run_chunked_embedding(cfg, W, ids, C, "buffer")
    np.testing.assert_allclose(rows, H, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(rows.max(axis=0), H.max(axis=0), rtol=1e-12, atol=1e-13)
    assert Wc[0] == 19


def test_weighted_and_buffered_contract_errors():
    cfg = micro_config()
    W = sharp_weights(cfg, 49)
    pk = _fresh_kv(cfg, 2, 64, 1)
    pk.reserve(0, 64)
    kv = OracleKV.from_paged(pk)
    S, Wc = np.zeros((2, cfg.d_model)), np.zeros(2)
    ids = draw_tokens(9, 2, 8, cfg.vocab)
    w = np.ones(8, np.float32)
    bad = [
        (Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids), "desc"),                     # no weights
        (Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids, token_weights=w[:7]), "desc"),
        (Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids,
               token_weights=np.where(np.arange(8) == 3, -1.0, 1.0)), "desc"),
        (Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids,
               token_weights=np.where(np.arange(8) == 5, np.nan, 1.0)), "desc"),
        (Batch([EmbChunk(0, 0, 8, True, "buffer")], [], ids, hidden_stride=7), "capacity"),
        (Batch([EmbChunk(0, 0, 8, True, "median")], [], ids), "desc"),
    ]
    for b, kind in bad:
        with pytest.raises(StepError) as e:
            step_oracle((cfg, W), (cfg, W), b, kv, kv, S, Wc)
        assert e.value.kind == kind, (b, e.value.kind)
    # a negative weight on a token of a chunk that does not use weights is not looked at
    ok = Batch([EmbChunk(0, 0, 4, False, "mean"), EmbChunk(1, 0, 4, True, "wmean")], [], ids,
               token_weights=np.array([-1, -1, -1, -1, 1, 1, 1, 1], np.float32))
    pk.reserve(1, 4)
    kv = OracleKV.from_paged(pk)
    step_oracle((cfg, W), (cfg, W), ok, kv, kv, S, Wc)


# ---------------------------------------------------------------------------
# LoRA on the embedding slice (the shared-backbone deployment: generator + adapter)
# ---------------------------------------------------------------------------
def _merged(W, lora):
    """Base weights with every adapted projection replaced by W + scale * B A (built here from
    the adapter's matrices, independently of the oracle's low-rank path)."""
    s = lora["scale"]
    out = {k: v for k, v in W.items() if k != "layers"}
    out["layers"] = []
    for lw, ll in zip(W["layers"], lora["layers"]):
        m = dict(lw)
        if "qkv" in ll:
            A, B = ll["qkv"]
            m["w_qkv"] = np.asarray(lw["w_qkv"], np.float64) + s * (np.asarray(B, np.float64) @ A)
        if "o" in ll:
            A, B = ll["o"]
            m["w_o"] = np.asarray(lw["w_o"], np.float64) + s * (np.asarray(B, np.float64) @ A)
        if "gate_up" in ll:
            A, Bg, Bu = ll["gate_up"]
            m["w_gate"] = np.asarray(lw["w_gate"], np.float64) + s * (np.asarray(Bg, np.float64) @ A)
            m["w_up"] = np.asarray(lw["w_up"], np.float64) + s * (np.asarray(Bu, np.float64) @ A)
        if "down" in ll:
            A, B = ll["down"]
            m["w_down"] = np.asarray(lw["w_down"], np.float64) + s * (np.asarray(B, np.float64) @ A)
        out["layers"].append(m)
    return out


@pytest.mark.parametrize("sites", [("qkv", "o", "gate_up", "down"), ("qkv",), ("o", "down"), ("gate_up",)])
def test_lora_equals_merged_weights(sites):
    from workload import make_lora
    cfg = micro_config()
    W = sharp_weights(cfg, 51)
    lora = make_lora(cfg, 51, rank=4, sites=sites)
    ids = draw_tokens(10, 1, 17, cfg.vocab)
    got = oracle.forward_full(cfg, W, ids, lora)
    want = oracle.forward_full(cfg, _merged(W, lora), ids)
    np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-12)
    # the update is not negligible: the adapted model differs from the base one
    base = oracle.forward_full(cfg, W, ids)
    assert np.abs(got - base).max() > 0.05 * np.abs(base).max()


def test_lora_with_zero_b_is_the_base_model():
    from workload import make_lora
    cfg = micro_config()
    W = sharp_weights(cfg, 53)
    lora = make_lora(cfg, 53, rank=4, std_b=0.0)
    ids = draw_tokens(10, 2, 13, cfg.vocab)
    np.testing.assert_array_equal(oracle.forward_full(cfg, W, ids, lora), oracle.forward_full(cfg, W, ids))


def test_lora_chunks_in_a_mixed_batch_equal_each_request_alone():
    """Two adapters and the base model on three embedding requests, chunked over two steps,
    beside decode rows of the generator (never adapted): every finished embedding equals the
    single-pass embedding through its own adapter, built from merged weights, and the decode
    logits equal the base model's full recompute."""
    from workload import make_lora
    cfg = micro_config()
    W = sharp_weights(cfg, 55)
    ad = [make_lora(cfg, 55, rank=4, tag=1), make_lora(cfg, 55, rank=4, tag=2, scale=0.5)]
    We = dict(W, adapters=ad)
    n_seq = 5
    pk = _fresh_kv(cfg, n_seq, 64, 3)
    lens = {0: 20, 1: 15, 2: 9}
    ids = {s: draw_tokens(11, s, n, cfg.vocab) for s, n in lens.items()}
    for s in lens:
        pk.reserve(s, 64)
    pk.fill_random(3, 10, 4)
    pk.reserve(3, 11)
    kv = OracleKV.from_paged(pk)
    S, Wc = np.zeros((n_seq, cfg.d_model)), np.zeros(n_seq)
    dec_tok = draw_tokens(11, 9, 1, cfg.vocab)
    b1 = Batch([EmbChunk(0, 0, 12, False, "mean"), EmbChunk(1, 0, 15, True, "last"),
                EmbChunk(2, 0, 4, False, "mean")], [DecodeRow(3, 10)],
               np.concatenate([ids[0][:12], ids[1], ids[2][:4], dec_tok]), chunk_adapter=[0, 1, -1])
    r1 = step_oracle((cfg, We), (cfg, We), b1, kv, kv, S, Wc)
    b2 = Batch([EmbChunk(2, 4, 5, True, "mean"), EmbChunk(0, 12, 8, True, "mean")], [],
               np.concatenate([ids[2][4:], ids[0][12:]]), chunk_adapter=[-1, 0])
    r2 = step_oracle((cfg, We), (cfg, We), b2, kv, kv, r1["acc_sum"], r1["acc_w"])
    for out, s, head, lora in ((r1["out_emb"][1], 1, "last", ad[1]), (r2["out_emb"][0], 2, "mean", None),
                               (r2["out_emb"][1], 0, "mean", ad[0])):
        Wm = _merged(W, lora) if lora else W
        np.testing.assert_allclose(out, oracle.embed_single_pass(cfg, Wm, ids[s], head), rtol=1e-11, atol=1e-12)
    # the decode row attends to random cached keys: compare with the base model through the cache
    kv_base = OracleKV.from_paged(pk)
    r_base = step_oracle((cfg, W), (cfg, W), Batch([], [DecodeRow(3, 10)], dec_tok), kv_base, kv_base,
                         np.zeros((n_seq, cfg.d_model)), np.zeros(n_seq))
    np.testing.assert_allclose(r1["logits"], r_base["logits"], rtol=1e-12, atol=1e-13)


def test_lora_contract_errors():
    from workload import make_lora
    cfg = micro_config()
    W = sharp_weights(cfg, 57)
    We = dict(W, adapters=[make_lora(cfg, 57, rank=4, tag=t) for t in range(6)])
    pk = _fresh_kv(cfg, 6, 16, 1)
    for s in range(6):
        pk.reserve(s, 16)
    kv = OracleKV.from_paged(pk)
    S, Wc = np.zeros((6, cfg.d_model)), np.zeros(6)
    ids = draw_tokens(12, 1, 12, cfg.vocab)
    bad = [
        (Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[6]), "desc"),
        (Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[-2]), "desc"),
        (Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[0, 1]), "desc"),
        (Batch([EmbChunk(s, 0, 2, True) for s in range(5)], [], ids[:10], chunk_adapter=[0, 1, 2, 3, 4]),
         "capacity"),
    ]
    for b, kind in bad:
        with pytest.raises(StepError) as e:
            step_oracle((cfg, We), (cfg, We), b, kv, kv, S, Wc)
        assert e.value.kind == kind
    with pytest.raises(StepError) as e:   # a model without adapters
        step_oracle((cfg, W), (cfg, W), Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[0]),
                    kv, kv, S, Wc)
    assert e.value.kind == "desc"


def test_bf16_rounding_of_cached_keys_and_values():
    """round_to_bf16 against round-to-nearest-even at bfloat16's 8 significant bits, worked out
    by hand: exact values, both sides of a tie, ties to the even significand, the carry into the
    exponent, signed zeros; then against torch's float32 -> bfloat16 conversion on float32 inputs
    (one rounding there, so the two must agree)."""
    from oracle.step import round_to_bf16
    u = 2.0 ** -7                      # one unit in the last place of bfloat16 at [1, 2)
    cases = [(1.0, 1.0), (1 + u / 2, 1.0), (1 + 3 * u / 2, 1 + 2 * u), (1 + u / 2 + 2.0 ** -30, 1 + u),
             (1 + u / 2 - 2.0 ** -30, 1.0), (-(1 + 3 * u / 2), -(1 + 2 * u)), (2 - u / 2, 2.0),
             (math.pi, 3.140625), (2.0 ** 100 * (1 + u / 2), 2.0 ** 100), (0.0, 0.0), (1.5, 1.5)]
    got = round_to_bf16(np.array([c[0] for c in cases]))
    np.testing.assert_array_equal(got, np.array([c[1] for c in cases]))
    assert math.copysign(1.0, float(round_to_bf16(np.array([-0.0]))[0])) == -1.0
    import torch
    x = np.random.default_rng(3).standard_normal(4096).astype(np.float32) * np.float32(5.0)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_to_bf16(x.astype(np.float64)), ref)


def test_bf16_cache_stores_rounded_keys_and_values():
    """A bf16 cache keeps what a step writes rounded to bfloat16 and gives it back as stored; an
    fp32 cache keeps the float64 values."""
    from oracle.step import round_to_bf16
    for dtype in ("f32", "bf16"):
        cfg = ModelConfig(n_layers=1, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, d_ff=256,
                          vocab=64, dtype=dtype)
        W = make_weights(cfg, 5)
        pk = _fresh_kv(cfg, 1, 32, 1)
        pk.reserve(0, 20)
        kv = OracleKV.from_paged(pk)
        assert kv.bf16 == (dtype == "bf16")
        ids = draw_tokens(5, 0, 20, cfg.vocab)
        step_oracle((cfg, W), (cfg, W), Batch([EmbChunk(0, 0, 20, False, "none")], [], ids), kv, kv,
                    np.zeros((1, cfg.d_model)), np.zeros(1))
        K, V = kv.read(0, 0, 20)
        assert np.isfinite(K).all() and np.isfinite(V).all()
        if dtype == "bf16":
            np.testing.assert_array_equal(K, round_to_bf16(K))
            np.testing.assert_array_equal(V, round_to_bf16(V))
        else:
            assert not np.array_equal(K, round_to_bf16(K))
