"""Single-request definition of the forward pass, pooling and decode logits (float64).

Section 3.1 states that the forward applies the same attention and feed-forward
layers to every request type, differing only in input length; Section 2.2 says
an embedding request is a prefill-shaped pass followed by pooling of the final
hidden states (mean or last-token), and a decode step reads the cached keys and
values of all earlier tokens.  The evaluated models (Mistral-7B, Qwen2-7B,
LLaMA-3.1-8B and their embedding derivatives) are pre-norm decoders with
RMSNorm, rotary position embedding, grouped-query attention and a SwiGLU MLP;
that is the block written out here:

    x   = E[ids]
    per layer:
        a = rms(x) * g_attn
        q, k, v = a Wq^T, a Wk^T, a Wv^T          (one fused [qkv, d] matrix)
        q, k <- RoPE at absolute positions 0..n-1
        o_h = softmax(q_h k_g^T / sqrt(hd), causal) v_g,  g = h // (nq / nkv)
        x = x + o Wo^T
        b = rms(x) * g_mlp
        x = x + (silu(b Wg^T) * (b Wu^T)) Wd^T
    H = rms(x) * g_final

Readings taken where the paper is silent: RMSNorm eps sits inside the square
root; RoPE rotates the half-split pairs (i, i + hd/2) by angle pos * base^(-2i/hd);
query head h reads KV head h // (nq / nkv) (contiguous groups); no sliding
window; the pooled tensor is the output of the final RMSNorm (the tensor the LM
head reads); finished embeddings are divided by max(||v||_2, 1e-12).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, F64)


def rope_rotate(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotary embedding of x[n, heads, hd] at integer positions[n] (half-split pairs)."""
    x = np.asarray(x, F64)
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = np.power(F64(base), -(2.0 * np.arange(half, dtype=F64)) / hd)
    ang = np.asarray(positions, F64)[:, None] * inv_freq[None, :]          # [n, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
                         k_pos: np.ndarray) -> np.ndarray:
    """Scaled dot-product attention, query i sees keys with position <= q_pos[i].

    q[nq_rows, nq, hd]; k, v[n_keys, nkv, hd].  Query head h reads KV head
    h // (nq / nkv).  Scale 1/sqrt(hd); softmax per query row over visible keys.
    Returns o[nq_rows, nq * hd].
    """
    q = np.asarray(q, F64)
    k = np.asarray(k, F64)
    v = np.asarray(v, F64)
    n, nq, hd = q.shape
    nkv = k.shape[1]
    group = nq // nkv
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]     # [n, n_keys]
    out = np.empty((n, nq, hd), F64)
    scale = 1.0 / np.sqrt(F64(hd))
    for h in range(nq):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s = np.where(visible, s, -np.inf)
        out[:, h, :] = softmax_rows(s) @ v[:, g, :]
    return out.reshape(n, nq * hd)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _split_qkv(cfg, qkv: np.ndarray):
    n = qkv.shape[0]
    q = qkv[:, :cfg.q_dim].reshape(n, cfg.n_q_heads, cfg.head_dim)
    k = qkv[:, cfg.q_dim:cfg.q_dim + cfg.kv_dim].reshape(n, cfg.n_kv_heads, cfg.head_dim)
    v = qkv[:, cfg.q_dim + cfg.kv_dim:].reshape(n, cfg.n_kv_heads, cfg.head_dim)
    return q, k, v


def lora_delta(x: np.ndarray, A, B, scale: float) -> np.ndarray:
    """Low-rank update of a projection's output: scale * (x A^T) B^T, with A [r][in], B [out][r]
    (the adapted projection computes x W^T + scale * x A^T B^T, i.e. x (W + scale B A)^T)."""
    return scale * ((np.asarray(x, F64) @ np.asarray(A, F64).T) @ np.asarray(B, F64).T)


def project(x: np.ndarray, W, layer_lora, site: str, scale: float, which: int = 1) -> np.ndarray:
    """x W^T, plus the adapter's low-rank update when the adapter covers `site` (layer_lora[site]
    = (A, B) or, for gate_up, (A, B_gate, B_up): `which` picks B_gate (1) or B_up (2))."""
    y = np.asarray(x, F64) @ np.asarray(W, F64).T
    ab = None if layer_lora is None else layer_lora.get(site)
    if ab is not None:
        y = y + lora_delta(x, ab[0], ab[which], scale)
    return y


def mlp(layer, b: np.ndarray, layer_lora=None, scale: float = 0.0) -> np.ndarray:
    gate = project(b, layer["w_gate"], layer_lora, "gate_up", scale, 1)
    up = project(b, layer["w_up"], layer_lora, "gate_up", scale, 2)
    return project(silu(gate) * up, layer["w_down"], layer_lora, "down", scale)


def _lora_layers(weights, lora):
    if lora is None:
        return [None] * len(weights["layers"]), 0.0
    return lora["layers"], float(lora["scale"])


def forward_full(cfg, weights, ids, lora=None) -> np.ndarray:
    """Final-normed hidden states H[n, d] of one request of tokens ids, positions 0..n-1, through
    the base model or, with `lora`, the base model plus that adapter's low-rank updates."""
    ids = np.asarray(ids, np.int64)
    n = ids.shape[0]
    pos = np.arange(n)
    x = np.asarray(weights["tok_emb"], F64)[ids]
    lls, sc = _lora_layers(weights, lora)
    for layer, ll in zip(weights["layers"], lls):
        a = rmsnorm(x, layer["attn_norm"], cfg.rms_eps)
        q, k, v = _split_qkv(cfg, project(a, layer["w_qkv"], ll, "qkv", sc))
        q = rope_rotate(q, pos, cfg.rope_base)
        k = rope_rotate(k, pos, cfg.rope_base)
        o = causal_gqa_attention(q, k, v, pos, pos)
        x = x + project(o.reshape(n, -1), layer["w_o"], ll, "o", sc)
        b = rmsnorm(x, layer["mlp_norm"], cfg.rms_eps)
        x = x + mlp(layer, b, ll, sc)
    return rmsnorm(x, weights["final_norm"], cfg.rms_eps)


def l2_normalize(v: np.ndarray) -> np.ndarray:
    v = np.asarray(v, F64)
    return v / max(float(np.linalg.norm(v)), 1e-12)


def pool_single_pass(H: np.ndarray, head: str, weights=None) -> np.ndarray:
    """Section 3.3 heads over all n rows at once: mean (w = 1), weighted mean
    (sum_j w_j H_j / sum_j w_j, Eq. (1)-(2) in one step; the zero vector when every weight is
    0), CLS (row 0), last (row n-1)."""
    H = np.asarray(H, F64)
    if head == "mean":
        return H.sum(axis=0) / H.shape[0]
    if head == "wmean":
        w = np.asarray(weights, F64)
        tot = w.sum()
        return (w[:, None] * H).sum(axis=0) / tot if tot > 0 else np.zeros(H.shape[1])
    if head == "cls":
        return H[0].copy()
    if head == "last":
        return H[-1].copy()
    raise ValueError(f"unknown pooling head {head!r}")


def embed_single_pass(cfg, weights, ids, head: str, token_weights=None, lora=None) -> np.ndarray:
    """Unchunked embedding: forward (optionally through a LoRA adapter), pool, L2-normalise."""
    return l2_normalize(pool_single_pass(forward_full(cfg, weights, ids, lora), head, token_weights))


def lm_logits(weights, h: np.ndarray) -> np.ndarray:
    """Untied LM head over final-normed rows h[..., d]."""
    return np.asarray(h, F64) @ np.asarray(weights["lm_head"], F64).T


def decode_full_recompute(cfg, weights, ids) -> np.ndarray:
    """Next-token logits after tokens ids, recomputed from the whole prefix without a cache."""
    H = forward_full(cfg, weights, ids)
    return lm_logits(weights, H[-1])


def greedy_token(logits: np.ndarray) -> np.ndarray:
    """Greedy sampling (the sampler of Algorithm 1 at temperature 0): the index of each row's
    largest logit, the lowest index among equal maxima (the paper fixes no tie-break)."""
    logits = np.asarray(logits, F64)
    return np.argmax(logits, axis=-1).astype(np.int64)
