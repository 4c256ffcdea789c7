"""Seeded synthetic inputs for the mixed embedding-chunk + decode step.

This module only draws numbers and lays them out: model shapes, weight tensors,
token ids, paged-KV page assignment and synthetic cache contents.  It performs
no part of the forward step (no normalisation, projection, attention, pooling
or sampling), so the CPU oracle and the GPU path can both consume the very same
inputs without sharing any of the method's arithmetic.

Workload shapes follow the paper's evaluation setting: a 7B-class decoder
(Mistral / Qwen2 / LLaMA-3.1 family, 32 query heads sharing 8 KV heads of
width 128, SwiGLU MLP of width 14336), a 2048-token step budget with embedding
chunks of 512 tokens (appendix, chunk-size / token-budget sweeps), vLLM-style
16-token KV pages, and a tiny two-layer decoder of the same family for fast
exact checks.  The paper's models and datasets are not used: every weight is
drawn N(0, 0.02) from a seed, every token id uniformly over the vocabulary.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

POOL_MEAN = "mean"
POOL_LAST = "last"
POOL_CLS = "cls"
POOL_NONE = "none"
POOL_WMEAN = "wmean"
POOL_BUFFER = "buffer"
POOL_KINDS = (POOL_MEAN, POOL_LAST, POOL_CLS, POOL_NONE, POOL_WMEAN, POOL_BUFFER)


# ---------------------------------------------------------------------------
# model shapes
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    page_size: int = 16
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    dtype: str = "f32"          # "f32" or "bf16": weights, KV cache and GEMM inputs
    has_lm_head: bool = True

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_dim(self) -> int:
        return self.q_dim + 2 * self.kv_dim

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


def tiny_config(dtype: str = "f32") -> ModelConfig:
    """Two-layer decoder: hidden 256, 4 MHA heads of 64, SwiGLU 1024, vocab 1024."""
    return ModelConfig(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
                       d_ff=1024, vocab=1024, dtype=dtype)


def llm7b_config(n_layers: int = 32, dtype: str = "bf16", has_lm_head: bool = True) -> ModelConfig:
    """7B-class decoder shape: hidden 4096, 32 q heads / 8 kv heads x 128, SwiGLU 14336."""
    return ModelConfig(n_layers=n_layers, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       d_ff=14336, vocab=32000, dtype=dtype, has_lm_head=has_lm_head)


# ---------------------------------------------------------------------------
# bf16 rounding (input preparation only)
# ---------------------------------------------------------------------------
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    # finite inputs only: the rounding increment cannot carry out of 32 bits
    r = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(x.shape)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-exact."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def bf16_from_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# weights
# ---------------------------------------------------------------------------
_GLOBAL_LAYER = 1_000_000  # spawn-key slot for tensors that belong to no layer

_TENSOR_IDS = {"tok_emb": 0, "lm_head": 1, "w_q": 2, "w_k": 3, "w_v": 4, "w_o": 5,
               "w_gate": 6, "w_up": 7, "w_down": 8}


def _normal(seed: int, model_tag: int, layer: int, tensor: str, shape, std: float,
            bf16: bool) -> np.ndarray:
    ss = np.random.SeedSequence(seed, spawn_key=(model_tag, layer, _TENSOR_IDS[tensor]))
    rng = np.random.default_rng(ss)
    w = rng.standard_normal(size=shape, dtype=np.float32)
    w *= np.float32(std)
    return round_bf16(w) if bf16 else w


def make_weights(cfg: ModelConfig, seed: int, model_tag: int = 0, std: float = 0.02,
                 qk_std: Optional[float] = None) -> Dict:
    """Seeded weights, every matrix and the embedding table N(0, std), unit norm gains.

    Matrices are stored [out_features, in_features] (row = output feature).  The
    fused QKV matrix stacks the query heads, then the key heads, then the value
    heads, each head a contiguous block of head_dim rows.  The LM head is untied
    from the embedding table.  ``qk_std`` (if given) overrides the spread of the
    query and key projections to make attention sharper than N(0, 0.02) gives.
    Each tensor has its own spawn key, so any one layer can be regenerated alone.
    """
    bf16 = cfg.dtype == "bf16"
    d, F = cfg.d_model, cfg.d_ff
    qs = std if qk_std is None else qk_std
    out = {
        "tok_emb": _normal(seed, model_tag, _GLOBAL_LAYER, "tok_emb", (cfg.vocab, d), std, bf16),
        "final_norm": np.ones(d, np.float32),
        "lm_head": (_normal(seed, model_tag, _GLOBAL_LAYER, "lm_head", (cfg.vocab, d), std, bf16)
                    if cfg.has_lm_head else None),
        "layers": [],
    }
    for l in range(cfg.n_layers):
        wq = _normal(seed, model_tag, l, "w_q", (cfg.q_dim, d), qs, bf16)
        wk = _normal(seed, model_tag, l, "w_k", (cfg.kv_dim, d), qs, bf16)
        wv = _normal(seed, model_tag, l, "w_v", (cfg.kv_dim, d), std, bf16)
        out["layers"].append({
            "attn_norm": np.ones(d, np.float32),
            "w_qkv": np.concatenate([wq, wk, wv], axis=0),
            "w_o": _normal(seed, model_tag, l, "w_o", (d, cfg.q_dim), std, bf16),
            "mlp_norm": np.ones(d, np.float32),
            "w_gate": _normal(seed, model_tag, l, "w_gate", (F, d), std, bf16),
            "w_up": _normal(seed, model_tag, l, "w_up", (F, d), std, bf16),
            "w_down": _normal(seed, model_tag, l, "w_down", (d, F), std, bf16),
        })
    return out


LORA_SITES = ("qkv", "o", "gate_up", "down")


def make_lora(cfg: ModelConfig, seed: int, rank: int, scale: float = 2.0, tag: int = 0,
              std_a: float = 0.02, std_b: float = 0.1, sites=LORA_SITES) -> Dict:
    """A seeded LoRA adapter of rank `rank` on the q, k, v, o, gate, up and down projections of
    every layer (the target set of the paper's e5-mistral embedding adapter), packed per fused
    projection of this model family:
      qkv: A [3r][d] = [A_q; A_k; A_v], B [(nq+2nkv)hd][3r] block-diagonal (query rows use
           columns 0..r-1, key rows r..2r-1, value rows 2r..3r-1);
      o: A [r][nq hd], B [d][r];
      gate_up: A [2r][d] = [A_gate; A_up], B_gate [F][2r] = [B_gate | 0], B_up [F][2r] = [0 | B_up];
      down: A [r][F], B [d][r].
    A ~ N(0, std_a), B ~ N(0, std_b) (bf16-rounded for bf16 models): with the default spreads
    the update scale * B A is as large as the base weights, so it is plainly visible."""
    bf16 = cfg.dtype == "bf16"
    d, F, r = cfg.d_model, cfg.d_ff, rank

    def draw(layer, k, shape, std):
        ss = np.random.SeedSequence(seed, spawn_key=(200 + tag, layer, k))
        w = np.random.default_rng(ss).standard_normal(size=shape, dtype=np.float32) * np.float32(std)
        return round_bf16(w) if bf16 else w

    layers = []
    for l in range(cfg.n_layers):
        ll = {}
        if "qkv" in sites:
            A = draw(l, 0, (3 * r, d), std_a)
            B = np.zeros((cfg.qkv_dim, 3 * r), np.float32)
            B[:cfg.q_dim, :r] = draw(l, 1, (cfg.q_dim, r), std_b)
            B[cfg.q_dim:cfg.q_dim + cfg.kv_dim, r:2 * r] = draw(l, 2, (cfg.kv_dim, r), std_b)
            B[cfg.q_dim + cfg.kv_dim:, 2 * r:] = draw(l, 3, (cfg.kv_dim, r), std_b)
            ll["qkv"] = (A, B)
        if "o" in sites:
            ll["o"] = (draw(l, 4, (r, cfg.q_dim), std_a), draw(l, 5, (d, r), std_b))
        if "gate_up" in sites:
            A = draw(l, 6, (2 * r, d), std_a)
            Bg = np.zeros((F, 2 * r), np.float32)
            Bu = np.zeros((F, 2 * r), np.float32)
            Bg[:, :r] = draw(l, 7, (F, r), std_b)
            Bu[:, r:] = draw(l, 8, (F, r), std_b)
            ll["gate_up"] = (A, Bg, Bu)
        if "down" in sites:
            ll["down"] = (draw(l, 9, (r, F), std_a), draw(l, 10, (d, r), std_b))
        layers.append(ll)
    return {"rank": r, "scale": float(scale), "layers": layers}


def as_float64(weights: Dict) -> Dict:
    """The same weights as float64 arrays (a one-time upcast for float64 consumers)."""
    f = lambda a: None if a is None else np.asarray(a, dtype=np.float64)
    out = {"tok_emb": f(weights["tok_emb"]), "final_norm": f(weights["final_norm"]),
           "lm_head": f(weights.get("lm_head")),
           "layers": [{k: f(v) for k, v in lw.items()} for lw in weights["layers"]]}
    if weights.get("adapters"):
        out["adapters"] = [{"rank": ad["rank"], "scale": ad["scale"],
                            "layers": [{k: tuple(f(x) for x in v) for k, v in ll.items()}
                                       for ll in ad["layers"]]} for ad in weights["adapters"]]
    return out


# ---------------------------------------------------------------------------
# batch descriptors
# ---------------------------------------------------------------------------
@dataclass
class EmbChunk:
    seq: int
    offset: int
    len: int
    last: bool
    pool: str = POOL_MEAN


@dataclass
class DecodeRow:
    seq: int
    ctx_len: int


@dataclass
class GenChunk:
    """A segment of a generation request's prompt; the final one (last) yields logits."""
    seq: int
    offset: int
    len: int
    last: bool


@dataclass
class Batch:
    """One step, type-sorted: embedding chunks, generation prefill chunks, decode rows.

    ``token_ids`` holds every embedding chunk's tokens in chunk order, then every prompt
    chunk's tokens, then one input token per decode row.  ``token_weights`` (weighted-mean
    chunks) holds one weight per embedding-chunk token, in the same order.  ``hidden_stride``
    is the number of rows per request of the buffer that buffered-head chunks fill.
    ``chunk_adapter`` names, per embedding chunk, the embedding model's LoRA adapter (-1: none).
    """
    chunks: List[EmbChunk] = field(default_factory=list)
    rows: List[DecodeRow] = field(default_factory=list)
    token_ids: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    gen_chunks: List[GenChunk] = field(default_factory=list)
    token_weights: Optional[np.ndarray] = None
    hidden_stride: int = 0
    chunk_adapter: Optional[List[int]] = None

    @property
    def n_emb_tokens(self) -> int:
        return int(sum(c.len for c in self.chunks))

    @property
    def n_gen_tokens(self) -> int:
        return int(sum(c.len for c in self.gen_chunks))

    @property
    def n_logit_rows(self) -> int:
        return int(sum(1 for c in self.gen_chunks if c.last)) + len(self.rows)

    @property
    def n_tokens(self) -> int:
        return self.n_emb_tokens + self.n_gen_tokens + len(self.rows)


# ---------------------------------------------------------------------------
# paged KV bookkeeping and contents
# ---------------------------------------------------------------------------
class PagedKV:
    """Host image of a paged KV cache: pools [L][n_pages][n_kv][page][hd] and a block table.

    Physical pages are handed out in a seeded random order so logically adjacent
    pages are never physically adjacent.  Every slot starts as NaN; only slots a
    caller fills (synthetic context or a step's own writes) hold numbers, so a
    read of a slot that was never written shows up as NaN downstream.
    """

    def __init__(self, cfg: ModelConfig, n_pages: int, n_seq: int, max_blocks: int, seed: int,
                 alloc_pools: bool = True):
        self.cfg = cfg
        self.n_pages, self.n_seq, self.max_blocks = n_pages, n_seq, max_blocks
        self.block_table = np.full((n_seq, max_blocks), -1, np.int32)
        self.n_blocks = np.zeros(n_seq, np.int64)
        rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(77,)))
        self._free = list(rng.permutation(n_pages).astype(np.int64))
        shape = (cfg.n_layers, n_pages, cfg.n_kv_heads, cfg.page_size, cfg.head_dim)
        if alloc_pools:
            self.k = np.full(shape, np.nan, np.float32)
            self.v = np.full(shape, np.nan, np.float32)
        else:
            self.k = self.v = None

    def reserve(self, seq: int, n_tokens: int) -> None:
        """Make sure ``seq`` owns pages for positions [0, n_tokens)."""
        need = -(-n_tokens // self.cfg.page_size)
        if need > self.max_blocks:
            raise ValueError(f"seq {seq}: {n_tokens} tokens exceed {self.max_blocks} blocks")
        while self.n_blocks[seq] < need:
            if not self._free:
                raise ValueError("page pool exhausted")
            self.block_table[seq, self.n_blocks[seq]] = self._free.pop()
            self.n_blocks[seq] += 1

    def release(self, seq: int) -> None:
        for b in range(int(self.n_blocks[seq])):
            self._free.append(int(self.block_table[seq, b]))
        self.block_table[seq, :] = -1
        self.n_blocks[seq] = 0

    def fill_random(self, seq: int, n_tokens: int, seed: int, std: float = 1.0) -> None:
        """Write N(0, std) keys and values (bf16-rounded for bf16 caches) at positions [0, n_tokens)."""
        cfg = self.cfg
        self.reserve(seq, n_tokens)
        rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(78, seq)))
        P = cfg.page_size
        for which in ("k", "v"):
            pool = getattr(self, which)
            vals = rng.standard_normal((cfg.n_layers, n_tokens, cfg.n_kv_heads, cfg.head_dim),
                                       dtype=np.float32)
            vals *= np.float32(std)
            if cfg.dtype == "bf16":
                vals = round_bf16(vals)
            for b in range(-(-n_tokens // P)):
                page = self.block_table[seq, b]
                lo, hi = b * P, min(n_tokens, (b + 1) * P)
                pool[:, page, :, 0:hi - lo, :] = vals[:, lo:hi].transpose(0, 2, 1, 3)


# ---------------------------------------------------------------------------
# the two fixed workloads used for exact checks and for measurement
# ---------------------------------------------------------------------------
def draw_tokens(seed: int, tag: int, n: int, vocab: int) -> np.ndarray:
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(90, tag)))
    return rng.integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def draw_token_weights(seed: int, tag: int, n: int) -> np.ndarray:
    """Per-token pooling weights for weighted-mean requests: uniform on [0, 1), fp32."""
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(91, tag)))
    return rng.random(n).astype(np.float32)


@dataclass
class StepWorkload:
    """Everything one mixed step consumes: shapes, weights, the batch, KV and accumulators."""
    cfg: ModelConfig
    weights: Dict
    batch: Batch
    kv: PagedKV
    acc_sum: np.ndarray
    acc_w: np.ndarray
    name: str = ""


def layer7b_mixed_workload(seed: int = 1002, with_pools: bool = True,
                           weights: Optional[Dict] = None, n_layers: int = 1) -> StepWorkload:
    """7B-shape layers (one by default; bf16, vocab 32000 LM head), 2048-token budget mixed step.

    Two embedding requests contribute 1024 chunk tokens (chunk 512, last-token
    pooling): request 0 is at offset 0 (first chunk, not last), request 1 at
    offset 1536 (its final chunk, after 1536 tokens already cached).  64 decode
    rows have contexts drawn uniformly from [1024, 4096].  Cached keys/values
    are N(0, 1) in bf16 in every layer.
    """
    cfg = llm7b_config(n_layers=n_layers)
    if weights is None:
        weights = make_weights(cfg, seed)
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(91,)))
    n_dec = 64
    ctx = rng.integers(1024, 4096, size=n_dec, endpoint=True)
    chunks = [EmbChunk(seq=0, offset=0, len=512, last=False, pool=POOL_LAST),
              EmbChunk(seq=1, offset=1536, len=512, last=True, pool=POOL_LAST)]
    rows = [DecodeRow(seq=2 + i, ctx_len=int(c)) for i, c in enumerate(ctx)]
    n_seq = 2 + n_dec
    P = cfg.page_size
    need = (2048 // P) * 2 + sum(-(-(int(c) + 1) // P) for c in ctx)
    n_pages = need + 64
    max_blocks = 4096 // P + 1
    kv = PagedKV(cfg, n_pages, n_seq, max_blocks, seed, alloc_pools=with_pools)
    if with_pools:
        kv.fill_random(1, 1536, seed)
        for r in rows:
            kv.fill_random(r.seq, r.ctx_len, seed)
    else:
        kv.reserve(1, 1536)
        for r in rows:
            kv.reserve(r.seq, r.ctx_len)
    for c in chunks:
        kv.reserve(c.seq, c.offset + c.len)
    for r in rows:
        kv.reserve(r.seq, r.ctx_len + 1)
    toks = draw_tokens(seed, 0, sum(c.len for c in chunks) + n_dec, cfg.vocab)
    batch = Batch(chunks=chunks, rows=rows, token_ids=toks)
    acc_sum = np.zeros((n_seq, cfg.d_model), np.float32)
    acc_w = np.zeros(n_seq, np.float32)
    acc_w[1] = 1536.0
    return StepWorkload(cfg, weights, batch, kv, acc_sum, acc_w, name="7b-layer-mixed-2048")


def tiny_mixed_scenario(seed: int = 1001, dtype: str = "f32", qk_std: Optional[float] = None):
    """The two-layer decoder driven through a short run of mixed steps from empty caches.

    Two embedding requests of 300 tokens are chunked by 128 (128, 128, 44) with
    mean pooling; four generation requests first have prompts of 64/100/150/200
    tokens written to the cache by KV-only chunks, then decode one token per step
    alongside the embedding chunks.  Returns (cfg, weights, n_seq, steps) where
    steps is a list of Batch; decode input tokens are seeded, not sampled.
    """
    cfg = tiny_config(dtype)
    weights = make_weights(cfg, seed, qk_std=qk_std)
    emb_len, C = 300, 128
    prompts = [64, 100, 150, 200]
    n_seq = 2 + len(prompts)
    toks_emb = [draw_tokens(seed, 1 + i, emb_len, cfg.vocab) for i in range(2)]
    toks_prompt = [draw_tokens(seed, 10 + i, p, cfg.vocab) for i, p in enumerate(prompts)]
    steps: List[Batch] = []
    # step 0: prompts written by KV-only chunks
    chunks = [EmbChunk(seq=2 + i, offset=0, len=p, last=False, pool=POOL_NONE)
              for i, p in enumerate(prompts)]
    steps.append(Batch(chunks=chunks, rows=[], token_ids=np.concatenate(toks_prompt)))
    # steps 1..3: embedding chunks + one decode token per generation request
    ctx = list(prompts)
    dec_tok = draw_tokens(seed, 50, 3 * len(prompts), cfg.vocab).reshape(3, len(prompts))
    for k in range(3):
        off = k * C
        ln = min(C, emb_len - off)
        chunks = [EmbChunk(seq=i, offset=off, len=ln, last=(off + ln == emb_len), pool=POOL_MEAN)
                  for i in range(2)]
        rows = [DecodeRow(seq=2 + i, ctx_len=ctx[i]) for i in range(len(prompts))]
        ids = np.concatenate([t[off:off + ln] for t in toks_emb] + [dec_tok[k]]).astype(np.int32)
        steps.append(Batch(chunks=chunks, rows=rows, token_ids=ids))
        ctx = [c + 1 for c in ctx]
    return cfg, weights, n_seq, steps


# ---------------------------------------------------------------------------
# larger-shape scenarios at reduced depth (7B-shape layers)
# ---------------------------------------------------------------------------
def _lognormal_lengths(rng, mean: float, n: int, sigma: float = 0.6, lo: int = 1, hi: int = 1 << 30):
    """Integer lengths from a lognormal with the given mean (sigma in log space, mu = ln(mean) -
    sigma^2 / 2), rounded and clipped to [lo, hi]."""
    mu = np.log(mean) - 0.5 * sigma * sigma
    return np.clip(np.rint(rng.lognormal(mu, sigma, size=n)), lo, hi).astype(np.int64)


def retrieval_mix_scenario(seed: int = 1003, n_layers: int = 1, budget: int = 2048,
                           fractions=(0.0, 0.25, 0.5, 0.75, 1.0), max_decode: int = 256):
    """Two 7B-shape models (embedding: mean pooling, no LM head; generator: vocab 32000) and
    one step per embedding fraction f of the token budget.

    Each step brings fresh query requests (single final chunks, lengths lognormal with mean
    64, the last one cut to fill f * budget exactly) and decode rows of the generation
    requests: D = min(budget - T_e, max_decode) of them, the same requests step after step
    (context + 1 per step they decode in), first contexts lognormal with mean 512.  Cached
    generator keys/values are N(0, 1) in bf16.  Returns (cfg_e, W_e, cfg_g, W_g, paged_e,
    paged_g, steps).
    """
    cfg_e = llm7b_config(n_layers=n_layers, has_lm_head=False)
    cfg_g = llm7b_config(n_layers=n_layers)
    W_e = make_weights(cfg_e, seed, model_tag=1)
    W_g = make_weights(cfg_g, seed, model_tag=2)
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(92,)))
    P = cfg_g.page_size
    n_gen = max_decode
    ctx0 = _lognormal_lengths(rng, 512, n_gen, lo=16, hi=4096 - len(fractions) - 1)   # documents
    # queries of every step, and the decode participation
    plan = []
    q_total = 0
    for f in fractions:
        te = int(round(f * budget))
        lens = []
        while sum(lens) < te:
            lens.append(int(_lognormal_lengths(rng, 64, 1, lo=1, hi=budget)[0]))        # queries
        if lens:
            lens[-1] -= sum(lens) - te
            lens = [x for x in lens if x > 0]
        plan.append((lens, min(budget - te, max_decode)))
        q_total += len(lens)
    n_seq_e = max(1, q_total)
    pages_e = sum(-(-x // P) for lens, _ in plan for x in lens) + 8
    max_blocks_e = budget // P + 1
    paged_e = PagedKV(cfg_e, pages_e, n_seq_e, max_blocks_e, seed)
    steps_total = len(fractions)
    pages_g = int(sum(-(-(int(c) + steps_total + 1) // P) for c in ctx0)) + 8
    max_blocks_g = 4096 // P + 1
    paged_g = PagedKV(cfg_g, pages_g, n_gen, max_blocks_g, seed + 1)
    for s, c in enumerate(ctx0):
        paged_g.fill_random(s, int(c), seed)
        paged_g.reserve(s, int(c) + steps_total + 1)
    ctx = ctx0.copy()
    steps: List[Batch] = []
    q_seq = 0
    for k, (lens, D) in enumerate(plan):
        chunks = []
        for x in lens:
            paged_e.reserve(q_seq, x)
            chunks.append(EmbChunk(seq=q_seq, offset=0, len=x, last=True, pool=POOL_MEAN))
            q_seq += 1
        rows = [DecodeRow(seq=s, ctx_len=int(ctx[s])) for s in range(D)]
        ids = draw_tokens(seed, 100 + k, sum(lens) + D, cfg_e.vocab)
        steps.append(Batch(chunks=chunks, rows=rows, token_ids=ids))
        ctx[:D] += 1
    return cfg_e, W_e, cfg_g, W_g, paged_e, paged_g, steps


def long_document_scenario(seed: int = 1004, n_layers: int = 1, n_docs: int = 3, doc_len: int = 2048,
                           chunk: int = 512, per_step: int = 3, n_dec: int = 32, ctx0: int = 2048):
    """Long-document embedding on one 7B-shape model (mean pooling, vocab 32000 LM head).

    ``n_docs`` documents of ``doc_len`` tokens are chunked by ``chunk`` and fed
    ``per_step`` chunks per step (at most one per document: a request appears once per
    batch), round-robin over the documents, next to ``n_dec``
    decode rows starting at context ``ctx0`` (+1 per step).  Document keys/values are
    written by the steps themselves; the decode requests' first ``ctx0`` positions are
    N(0, 1) bf16.  Returns (cfg, W, paged, steps).
    """
    if per_step > n_docs:
        raise ValueError("more chunks per step than documents")
    cfg = llm7b_config(n_layers=n_layers)
    W = make_weights(cfg, seed)
    P = cfg.page_size
    n_chunks = -(-doc_len // chunk)
    order = [(d, c) for c in range(n_chunks) for d in range(n_docs)]   # round-robin
    n_steps = -(-len(order) // per_step)
    n_seq = n_docs + n_dec
    pages = n_docs * (-(-doc_len // P)) + n_dec * (-(-(ctx0 + n_steps + 1) // P)) + 8
    max_blocks = max(doc_len, ctx0 + n_steps + 1) // P + 1
    paged = PagedKV(cfg, pages, n_seq, max_blocks, seed)
    for d in range(n_docs):
        paged.reserve(d, doc_len)
    for j in range(n_dec):
        paged.fill_random(n_docs + j, ctx0, seed)
        paged.reserve(n_docs + j, ctx0 + n_steps + 1)
    doc_tok = [draw_tokens(seed, 200 + d, doc_len, cfg.vocab) for d in range(n_docs)]
    dec_tok = draw_tokens(seed, 300, n_steps * n_dec, cfg.vocab).reshape(n_steps, n_dec)
    steps: List[Batch] = []
    for k in range(n_steps):
        part = order[k * per_step:(k + 1) * per_step]
        chunks, ids = [], []
        for d, c in part:
            off = c * chunk
            ln = min(chunk, doc_len - off)
            chunks.append(EmbChunk(seq=d, offset=off, len=ln, last=off + ln == doc_len, pool=POOL_MEAN))
            ids.append(doc_tok[d][off:off + ln])
        rows = [DecodeRow(seq=n_docs + j, ctx_len=ctx0 + k) for j in range(n_dec)]
        ids.append(dec_tok[k])
        steps.append(Batch(chunks=chunks, rows=rows, token_ids=np.concatenate(ids).astype(np.int32)))
    return cfg, W, paged, steps


@dataclass
class DeviceKVRecipe:
    """Block table of a cache whose contents are drawn on the device (too large for a host image)."""
    n_pages: int
    n_seq: int
    max_blocks: int
    block_table: np.ndarray
    seed: int


def decode_heavy_scenario(seed: int = 1005, n_layers: int = 1, n_dec: int = 256, ctx_lo: int = 4096,
                          ctx_hi: int = 8192, n_queries: int = 8, q_len: int = 16):
    """Decode-heavy step on one 7B-shape generator (vocab 32000): ``n_dec`` decode rows with
    contexts uniform in [ctx_lo, ctx_hi] plus ``n_queries`` short final chunks (mean
    pooling).  Keys/values are N(0, 1) bf16 drawn on the device (``fill_device_pools``);
    physical pages are a seeded permutation.  Returns (cfg, W, batch, recipe).
    """
    cfg = llm7b_config(n_layers=n_layers)
    W = make_weights(cfg, seed)
    P = cfg.page_size
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(93,)))
    ctx = rng.integers(ctx_lo, ctx_hi, size=n_dec, endpoint=True)
    n_seq = n_queries + n_dec
    need = [-(-q_len // P)] * n_queries + [-(-(int(c) + 1) // P) for c in ctx]
    n_pages = int(sum(need))
    max_blocks = max(need)
    perm = rng.permutation(n_pages).astype(np.int32)
    bt = np.full((n_seq, max_blocks), -1, np.int32)
    o = 0
    for s, n in enumerate(need):
        bt[s, :n] = perm[o:o + n]
        o += n
    chunks = [EmbChunk(seq=i, offset=0, len=q_len, last=True, pool=POOL_MEAN) for i in range(n_queries)]
    rows = [DecodeRow(seq=n_queries + j, ctx_len=int(c)) for j, c in enumerate(ctx)]
    ids = draw_tokens(seed, 400, n_queries * q_len + n_dec, cfg.vocab)
    return cfg, W, Batch(chunks=chunks, rows=rows, token_ids=ids), DeviceKVRecipe(n_pages, n_seq, max_blocks, bt, seed)


def device_weights(cfg: ModelConfig, seed: int, model_tag: int = 0, std: float = 0.02, device="cuda") -> Dict:
    """Seeded N(0, std) weights drawn on the device in the model dtype (torch tensors), same
    layout as make_weights, for shapes whose host image would be too large (32-layer 7B models).
    Each tensor has its own generator seed, derived from (seed, model_tag, layer, tensor)."""
    import torch
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    d, F = cfg.d_model, cfg.d_ff

    def draw(layer, name, shape):
        key = np.random.SeedSequence(seed, spawn_key=(model_tag, layer, _TENSOR_IDS[name])).generate_state(1)[0]
        g = torch.Generator(device=device)
        g.manual_seed(int(key))
        out = torch.empty(shape, dtype=dt, device=device)
        flat = out.view(-1)
        step = 1 << 26
        for i in range(0, flat.numel(), step):
            part = flat[i:i + step]
            part.copy_((torch.randn(part.numel(), generator=g, device=device) * std).to(dt))
        return out

    ones = lambda: torch.ones(d, dtype=torch.float32, device=device)
    W = {"tok_emb": draw(_GLOBAL_LAYER, "tok_emb", (cfg.vocab, d)), "final_norm": ones(),
         "lm_head": draw(_GLOBAL_LAYER, "lm_head", (cfg.vocab, d)) if cfg.has_lm_head else None,
         "layers": []}
    for l in range(cfg.n_layers):
        W["layers"].append({
            "attn_norm": ones(),
            "w_qkv": torch.cat([draw(l, "w_q", (cfg.q_dim, d)), draw(l, "w_k", (cfg.kv_dim, d)),
                                draw(l, "w_v", (cfg.kv_dim, d))]),
            "w_o": draw(l, "w_o", (d, cfg.q_dim)),
            "mlp_norm": ones(),
            "w_gate": draw(l, "w_gate", (F, d)),
            "w_up": draw(l, "w_up", (F, d)),
            "w_down": draw(l, "w_down", (d, F)),
        })
    return W


def fill_device_pools(k, v, seed: int) -> None:
    """Fill device key/value pools with N(0, 1) values of their dtype from a seeded device
    generator (torch tensors; values, not a method step)."""
    import torch
    g = torch.Generator(device=k.device)
    g.manual_seed(seed)
    for t in (k, v):
        flat = t.view(-1)
        step = 1 << 26
        for i in range(0, flat.numel(), step):
            part = flat[i:i + step]
            part.copy_(torch.randn(part.numel(), generator=g, device=k.device, dtype=torch.float32).to(t.dtype))
