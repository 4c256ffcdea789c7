"""The mixed step under its contract: paged KV, incremental pooling, decode logits (float64).

One call is the body of the paper's heterogeneous-batching loop (Algorithm 1)
without the scheduler and the sampler: a forward over a type-sorted batch of
embedding chunks, generation prefill chunks and decode tokens (Section 3.2),
then the incremental pooler on the embedding slice (Section 3.3, Eq. (1)-(2) and
the positional heads) and the LM head on the last row of every prompt's final
chunk and on every decode token (the rows the sampler reads).

Requests never attend to each other, so the oracle runs them one at a time, in
batch order, each through every layer: for a chunk the rows are the positions
offset .. offset+len-1 of its request; for a decode row it is the single
position ctx_len.  At every layer the rows' rotated keys and their values are
written into the request's cache slots first, then every row attends to all
keys of its request at positions <= its own, read back through the block table.

Readings taken where the paper is silent (also listed in the design notes):
* an embedding request's chunks attend causally to the keys of its earlier
  chunks, which stay in the paged cache (needed for the equivalence the paper
  claims between chunked and single-pass embedding);
* ``ctx_len`` of a decode row counts the tokens already cached; its input token
  sits at position ctx_len, is written to that slot and attends to ctx_len + 1
  keys including its own;
* slot of position p of request s = block_table[s][p // page] * page + p % page;
* a bf16 cache stores the keys and values a step writes rounded to bfloat16 (its element
  type), and later rows and steps read them back as stored;
* a chunk at offset 0 resets its request's state (S = 0, W = 0); a later chunk
  requires W == offset exactly, which catches a lost or repeated chunk;
* mean: S += sum of the chunk's rows, W += len; emitted S / W.  Last-token: the
  final chunk stores its last row.  CLS: the offset-0 chunk stores its first
  row.  Every pooled chunk adds len to W so the offset check holds for all heads;
* a finished embedding (chunk flagged last) is v / max(||v||_2, 1e-12);
* pooling kind "none" writes keys/values only (a cache-filling prefill chunk);
* weighted mean (Eq. (1)-(2) with caller weights w_{k,j} >= 0, one per embedding-chunk token):
  S += sum_j w_j H_j.  The state's W keeps counting tokens (the offset check above), because
  the emitted embedding normalize(S / sum w) equals normalize(S) for any positive weight sum,
  so the weight sum is never needed; with every weight 0 the embedding is the zero vector;
* buffered head (an arbitrary head applied after the final chunk, buffering the hidden states
  A = [A; H]): the chunk's final-normed hidden rows are returned for buffer rows
  seq * hidden_stride + offset .. + len - 1; W counts tokens as for every pooled chunk, and no
  embedding is emitted (the caller applies its head to the buffer);
* LoRA (the shared-backbone deployment the paper evaluates: the embedding model is the
  generator plus a low-rank adapter): chunk i of the embedding slice may name adapter
  ``chunk_adapter[i]`` of the embedding model (-1: the base model); every adapted projection
  then computes x W^T + scale (x A^T) B^T.  At most four distinct adapters per batch;
* a generation prefill chunk (seq, offset, len, last) runs through the generator
  and its cache like a decode row of ``len`` tokens at positions offset ..
  offset+len-1; only the final chunk of a prompt (last) emits logits, for its
  last row.  Logits rows are those rows in chunk order, then the decode rows;
  prompt chunks and decode rows share the generator's sequence namespace.
"""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np

from .model import (F64, rmsnorm, rope_rotate, causal_gqa_attention, mlp, _split_qkv,
                    l2_normalize, lm_logits, project, _lora_layers)

# most distinct adapters the embedding chunks of one batch may use
MAX_STEP_ADAPTERS = 4


class StepError(Exception):
    """A batch the step contract rejects; ``kind`` is desc, dupseq, capacity or device."""

    def __init__(self, kind: str, msg: str):
        super().__init__(f"{kind}: {msg}")
        self.kind = kind


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Each value rounded to the nearest bfloat16 (8 significant bits, ties to the even
    significand), returned as float64: the low 45 of float64's 52 fraction bits are dropped
    with round-to-nearest-even on the bit pattern.  For finite values inside bfloat16's normal
    range (the keys and values stored here)."""
    b = np.ascontiguousarray(x, dtype=F64).view(np.uint64)
    keep = (b >> np.uint64(45)) & np.uint64(1)
    b = (b + np.uint64((1 << 44) - 1) + keep) & ~np.uint64((1 << 45) - 1)
    return b.view(F64)


class OracleKV:
    """float64 image of one paged cache: k, v[L][n_pages][nkv][page][hd] plus the block table.

    ``bf16``: the cache's element type is bfloat16, so keys and values written by a step are
    stored rounded to bfloat16 (and read back as stored), as a bf16 cache holds them."""

    def __init__(self, k: np.ndarray, v: np.ndarray, block_table: np.ndarray, page_size: int,
                 bf16: bool = False):
        self.k = np.array(k, dtype=F64, copy=True)
        self.v = np.array(v, dtype=F64, copy=True)
        self.block_table = np.array(block_table, dtype=np.int64, copy=True)
        self.page = int(page_size)
        self.bf16 = bool(bf16)
        self.n_pages = self.k.shape[1]
        self.n_seq, self.max_blocks = self.block_table.shape

    @classmethod
    def from_paged(cls, paged) -> "OracleKV":
        return cls(paged.k, paged.v, paged.block_table, paged.cfg.page_size, bf16=paged.cfg.dtype == "bf16")

    def slots(self, seq: int, positions: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
        positions = np.asarray(positions, np.int64)
        pages = self.block_table[seq, positions // self.page]
        bad = (pages < 0) | (pages >= self.n_pages)
        if bad.any():
            raise StepError("device", f"seq {seq}: page id out of range in block table")
        return pages, positions % self.page

    def write(self, layer: int, seq: int, positions, k_rows, v_rows) -> None:
        pages, offs = self.slots(seq, positions)
        if self.bf16:
            k_rows, v_rows = round_to_bf16(k_rows), round_to_bf16(v_rows)
        self.k[layer, pages, :, offs, :] = k_rows
        self.v[layer, pages, :, offs, :] = v_rows

    def read(self, layer: int, seq: int, n_keys: int) -> Tuple[np.ndarray, np.ndarray]:
        pages, offs = self.slots(seq, np.arange(n_keys))
        return self.k[layer, pages, :, offs, :], self.v[layer, pages, :, offs, :]


def _forward_cached(cfg, weights, kv: OracleKV, seq: int, ids: np.ndarray,
                    positions: np.ndarray, lora=None) -> np.ndarray:
    """Final-normed hidden rows of one request's new tokens, attending through the cache (and
    through the adapter `lora`, if given, at every adapted projection)."""
    x = np.asarray(weights["tok_emb"], F64)[np.asarray(ids, np.int64)]
    n_keys = int(positions[-1]) + 1
    key_pos = np.arange(n_keys)
    lls, sc = _lora_layers(weights, lora)
    for l, layer in enumerate(weights["layers"]):
        a = rmsnorm(x, layer["attn_norm"], cfg.rms_eps)
        q, k, v = _split_qkv(cfg, project(a, layer["w_qkv"], lls[l], "qkv", sc))
        q = rope_rotate(q, positions, cfg.rope_base)
        k = rope_rotate(k, positions, cfg.rope_base)
        kv.write(l, seq, positions, k, v)
        K, V = kv.read(l, seq, n_keys)
        o = causal_gqa_attention(q, K, V, positions, key_pos)
        x = x + project(o.reshape(len(ids), -1), layer["w_o"], lls[l], "o", sc)
        b = rmsnorm(x, layer["mlp_norm"], cfg.rms_eps)
        x = x + mlp(layer, b, lls[l], sc)
    return rmsnorm(x, weights["final_norm"], cfg.rms_eps)


def validate(emb, gen, batch, emb_kv: OracleKV, gen_kv: OracleKV) -> None:
    """Host-side contract checks: raise StepError(desc | dupseq | capacity)."""
    emb_cfg, gen_cfg = emb[0], gen[0]
    gen_chunks = list(getattr(batch, "gen_chunks", []) or [])
    n_emb = sum(int(c.len) for c in batch.chunks)
    n_gen = sum(int(c.len) for c in gen_chunks)
    T = n_emb + n_gen + len(batch.rows)
    ids = np.asarray(batch.token_ids)
    if ids.shape != (T,):
        raise StepError("desc", f"token_ids has {ids.size} entries, batch needs {T}")
    seen = set()
    shared = emb_kv is gen_kv
    for c in batch.chunks:
        if not (0 <= c.seq < emb_kv.n_seq) or c.offset < 0 or c.len < 1:
            raise StepError("desc", f"bad chunk {c}")
        if (c.pool not in ("mean", "last", "cls", "none", "wmean", "buffer")
                or (c.pool == "none" and c.last)):
            raise StepError("desc", f"bad pooling for chunk {c}")
        if c.offset + c.len > emb_kv.max_blocks * emb_kv.page:
            raise StepError("capacity", f"chunk {c} exceeds the block table")
        if c.pool == "buffer" and c.offset + c.len > getattr(batch, "hidden_stride", 0):
            raise StepError("capacity", f"chunk {c} exceeds the hidden-state buffer")
        if ("e", c.seq) in seen:
            raise StepError("dupseq", f"seq {c.seq} twice")
        seen.add(("e", c.seq))
    for c in gen_chunks:
        if not (0 <= c.seq < gen_kv.n_seq) or c.offset < 0 or c.len < 1:
            raise StepError("desc", f"bad prompt chunk {c}")
        if c.offset + c.len > gen_kv.max_blocks * gen_kv.page:
            raise StepError("capacity", f"prompt chunk {c} exceeds the block table")
        key = ("e" if shared else "g", c.seq)
        if key in seen:
            raise StepError("dupseq", f"seq {c.seq} twice")
        seen.add(key)
    for r in batch.rows:
        if not (0 <= r.seq < gen_kv.n_seq) or r.ctx_len < 0:
            raise StepError("desc", f"bad decode row {r}")
        if r.ctx_len + 1 > gen_kv.max_blocks * gen_kv.page:
            raise StepError("capacity", f"decode row {r} exceeds the block table")
        key = ("e" if shared else "g", r.seq)
        if key in seen:
            raise StepError("dupseq", f"seq {r.seq} twice")
        seen.add(key)
    if (batch.rows or any(c.last for c in gen_chunks)) and gen[1].get("lm_head") is None:
        raise StepError("desc", "logits need a model with an LM head")
    if n_emb and ((ids[:n_emb] < 0).any() or (ids[:n_emb] >= emb_cfg.vocab).any()):
        raise StepError("desc", "chunk token id out of range")
    ca = getattr(batch, "chunk_adapter", None)
    if ca is not None:
        n_ad = len(emb[1].get("adapters") or [])
        if len(ca) != len(batch.chunks) or any(not (-1 <= int(a) < n_ad) for a in ca):
            raise StepError("desc", "chunk adapter index out of range")
        if len({int(a) for a in ca if a >= 0}) > MAX_STEP_ADAPTERS:
            raise StepError("capacity", f"more than {MAX_STEP_ADAPTERS} adapters in one batch")
    if any(c.pool == "wmean" for c in batch.chunks):
        w = getattr(batch, "token_weights", None)
        if w is None or np.asarray(w).shape != (n_emb,):
            raise StepError("desc", "weighted-mean chunks need one weight per embedding token")
        t = 0
        for c in batch.chunks:
            cw = np.asarray(w[t:t + c.len], F64)
            t += c.len
            if c.pool == "wmean" and not (np.isfinite(cw).all() and (cw >= 0).all()):
                raise StepError("desc", f"weights of chunk {c} must be finite and >= 0")
    if T > n_emb and ((ids[n_emb:] < 0).any() or (ids[n_emb:] >= gen_cfg.vocab).any()):
        raise StepError("desc", "generation token id out of range")


def step_oracle(emb: Tuple, gen: Tuple, batch, emb_kv: OracleKV, gen_kv: OracleKV,
                acc_sum: np.ndarray, acc_w: np.ndarray) -> Dict[str, np.ndarray]:
    """Run one mixed step.  ``emb`` and ``gen`` are (cfg, weights); they may be the same model.

    ``emb_kv`` / ``gen_kv`` are updated in place (the step appends keys and values).
    Returns float64 ``logits``[n_last_prompt_chunks + n_decode, vocab], ``out_emb``[n_chunks, d]
    (NaN rows for chunks not flagged last and for buffered-head chunks), ``hidden`` (chunk index
    -> its final-normed hidden rows, buffered-head chunks only) and the updated
    ``acc_sum``[n_seq, d], ``acc_w``[n_seq].
    """
    validate(emb, gen, batch, emb_kv, gen_kv)
    emb_cfg, emb_w = emb
    gen_cfg, gen_w = gen
    S = np.array(acc_sum, dtype=F64, copy=True)
    W = np.array(acc_w, dtype=F64, copy=True)
    d = emb_cfg.d_model
    out_emb = np.full((len(batch.chunks), d), np.nan, F64)
    ids = np.asarray(batch.token_ids, np.int64)
    tw = getattr(batch, "token_weights", None)
    ca = getattr(batch, "chunk_adapter", None)
    adapters = emb_w.get("adapters") or []
    hidden = {}
    t = 0
    for i, c in enumerate(batch.chunks):
        if c.pool != "none" and c.offset > 0 and W[c.seq] != c.offset:
            raise StepError("device", f"seq {c.seq}: accumulator holds {W[c.seq]} tokens, "
                                      f"chunk starts at {c.offset}")
        pos = np.arange(c.offset, c.offset + c.len)
        lora = adapters[int(ca[i])] if ca is not None and int(ca[i]) >= 0 else None
        H = _forward_cached(emb_cfg, emb_w, emb_kv, c.seq, ids[t:t + c.len], pos, lora)
        w = None if tw is None else np.asarray(tw[t:t + c.len], F64)
        t += c.len
        if c.pool == "none":
            continue
        if c.offset == 0:
            S[c.seq] = 0.0
            W[c.seq] = 0.0
        if c.pool == "buffer":
            hidden[i] = H
            W[c.seq] += c.len
            continue
        if c.pool == "mean":
            S[c.seq] += H.sum(axis=0)
        elif c.pool == "wmean":
            S[c.seq] += (w[:, None] * H).sum(axis=0)
        elif c.pool == "last" and c.last:
            S[c.seq] = H[-1]
        elif c.pool == "cls" and c.offset == 0:
            S[c.seq] = H[0]
        W[c.seq] += c.len
        if c.last:
            v = S[c.seq] / W[c.seq] if c.pool == "mean" else S[c.seq]
            out_emb[i] = l2_normalize(v)
    gen_chunks = list(getattr(batch, "gen_chunks", []) or [])
    n_logits = sum(1 for c in gen_chunks if c.last) + len(batch.rows)
    logits = np.zeros((n_logits, gen_cfg.vocab if n_logits else 0), F64)
    j = 0
    for c in gen_chunks:
        pos = np.arange(c.offset, c.offset + c.len)
        H = _forward_cached(gen_cfg, gen_w, gen_kv, c.seq, ids[t:t + c.len], pos)
        t += c.len
        if c.last:
            logits[j] = lm_logits(gen_w, H[-1])
            j += 1
    for r in batch.rows:
        H = _forward_cached(gen_cfg, gen_w, gen_kv, r.seq, ids[t:t + 1], np.array([r.ctx_len]))
        t += 1
        logits[j] = lm_logits(gen_w, H[0])
        j += 1
    return {"logits": logits, "out_emb": out_emb, "hidden": hidden, "acc_sum": S, "acc_w": W}
