"""Every (head_dim, group) shape the library accepts, fp32 and bf16, against the oracle.

orthrus_model_create accepts head_dim 64 or 128 with 1, 2 or 4 query heads per KV head; each pair
has its own instantiation of the attention kernels, the rotation epilogue and the rotation /
append row kernel.  One two-step scenario runs on all six pairs: a chunk resuming after 1500
cached tokens (mean), a one-chunk CLS request, a last-token request over two chunks, a one-chunk
prompt that gets logits, and decode rows at contexts 0, 17, 1100 and 2100 (several key splits);
then the second chunk, the prompt's first decode token and the decode rows again; then the
decode rows alone (a launch without prefill tiles: the decode-only attention kernel on the bf16
path).  Logits, embeddings, pooling state and every cache write are compared.
"""
import numpy as np
import pytest
import torch

from tests.parity import Pair
from workload import Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, draw_tokens, make_weights

pytestmark = pytest.mark.gpu

SHAPES = [(64, 1), (64, 2), (64, 4), (128, 1), (128, 2), (128, 4)]


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


@pytest.mark.parametrize("head_dim,group", SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_every_head_shape_mixed_steps(dtype, head_dim, group):
    nq = 8
    cfg = ModelConfig(n_layers=2, d_model=512, n_q_heads=nq, n_kv_heads=nq // group, head_dim=head_dim,
                      d_ff=1024, vocab=512, dtype=dtype)
    seed = 2200 + head_dim + group
    W = make_weights(cfg, seed, qk_std=0.06 if dtype == "bf16" else 0.15)
    n_seq, max_blocks = 8, 140
    pk = PagedKV(cfg, n_seq * max_blocks, n_seq, max_blocks, seed)
    dec_ctx = {4: 0, 5: 17, 6: 1100, 7: 2100}
    pk.fill_random(0, 1500, seed)
    for s, c in dec_ctx.items():
        pk.fill_random(s, c, seed + 1)
    for s, n in {0: 1600, 1: 77, 2: 80, 3: 42, 4: 3, 5: 20, 6: 1103, 7: 2103}.items():
        pk.reserve(s, n)
    acc_w = np.zeros(n_seq)
    acc_w[0] = 1500
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=300, max_chunks=4, max_decode=5, max_ctx=max_blocks * 16)
    rows = [DecodeRow(s, c) for s, c in dec_ctx.items()]
    b1 = Batch([EmbChunk(0, 1500, 100, True, "mean"), EmbChunk(1, 0, 77, True, "cls"),
                EmbChunk(2, 0, 50, False, "last")], rows,
               draw_tokens(seed, 1, 100 + 77 + 50 + 40 + 4, cfg.vocab), gen_chunks=[GenChunk(3, 0, 40, True)])
    pair.step(b1)
    rows2 = [DecodeRow(3, 40)] + [DecodeRow(s, c + 1) for s, c in dec_ctx.items()]
    b2 = Batch([EmbChunk(2, 50, 30, True, "last")], rows2, draw_tokens(seed, 2, 30 + 5, cfg.vocab))
    pair.step(b2)
    rows3 = [DecodeRow(3, 41)] + [DecodeRow(s, c + 2) for s, c in dec_ctx.items()]
    pair.step(Batch([], rows3, draw_tokens(seed, 3, 5, cfg.vocab)))
    print(f"{dtype} hd {head_dim} group {group}: {pair.report}", flush=True)
