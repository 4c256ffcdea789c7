"""Conditioning of the float64 definition at depth (CPU): why the deep fp32 parity cases use
moderately sharp attention.

With query/key weights of spread 0.15 on a hidden size of 512 the attention logits have a
standard deviation of about 12: the softmax is nearly one-hot and a near-tie between two keys
flips with the smallest change of the scores.  Through many layers such flips compound: the
oracle's own output moves far more than fp32 rounding under a relative change of 2^-24 of its
inputs (the rounding level of fp32).  A parity bound of 1e-4 cannot hold there for any fp32
implementation.  With spread 0.09 (logit std ~4) the same change stays small but still grows
tenfold from 2 to 32 layers; with 0.06 (logit std ~1.8, the spread of the bf16 cases) it shrinks
with depth.  The fp32 parity cases therefore use 0.15 at 2 layers, 0.09 at 8 and 0.06 at 32.
"""
import numpy as np

from oracle import forward_full
from workload import ModelConfig, as_float64, draw_tokens, make_weights


def sensitivity(qk_std: float, n_layers: int) -> float:
    cfg = ModelConfig(n_layers=n_layers, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                      vocab=512, dtype="f32")
    W = as_float64(make_weights(cfg, 2100 + n_layers, qk_std=qk_std))
    ids = draw_tokens(2100 + n_layers, 0, 200, cfg.vocab)
    H = forward_full(cfg, W, ids)
    rng = np.random.default_rng(0)
    W2 = dict(W)
    W2["tok_emb"] = W["tok_emb"] * (1 + rng.uniform(-2.0 ** -24, 2.0 ** -24, W["tok_emb"].shape))
    H2 = forward_full(cfg, W2, ids)
    return float((np.abs(H - H2).max(axis=1) / np.abs(H).max(axis=1)).max())


def test_near_one_hot_attention_is_ill_conditioned_at_depth():
    assert sensitivity(0.15, 2) < 1e-5
    assert sensitivity(0.15, 32) > 1e-3          # measured 1.1e-2


def test_moderately_sharp_attention_stays_at_rounding_level():
    assert sensitivity(0.09, 32) < 2e-5          # measured 4.7e-6 (4.7e-7 at 2 layers)
    assert sensitivity(0.06, 32) < 1e-6          # measured 7.0e-8 (1.8e-7 at 2 layers)
