"""GPU parity at the edges of the batch descriptor, against the float64 oracle: one-token chunks
on page boundaries, decode rows at context 0 and on page edges, batches of one item kind, an
empty batch, a model without layers (token gather, final norm, pooling and LM head only), and a
bf16 batch of more than 1280 rows (the rotation/append kernel of large batches, with and
without a bad page).
"""
import numpy as np
import pytest
import torch

from workload import Batch, DecodeRow, EmbChunk, PagedKV, draw_tokens, make_weights, tiny_config
from tests.parity import Pair

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _boundary_pair(cfg, seed):
    """Sequences 0-2 take chunks, 3-6 decode rows at contexts 0, 15, 16 and 31 (16-token pages)."""
    W = make_weights(cfg, seed)
    n_seq, max_blocks = 8, 8
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, seed)
    pk.reserve(0, 1)
    pk.fill_random(1, 15, seed + 1)
    pk.reserve(1, 16)
    pk.fill_random(2, 16, seed + 2)
    pk.reserve(2, 33)
    for i, c in enumerate((0, 15, 16, 31)):
        if c:
            pk.fill_random(3 + i, c, seed + 3 + i)
        pk.reserve(3 + i, c + 1)
    acc_w = np.zeros(n_seq)
    acc_w[1], acc_w[2] = 15, 16
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=64, max_chunks=3, max_decode=4, max_ctx=128)
    return pair


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_one_token_chunks_and_decode_rows_on_page_edges(dtype):
    """A one-token request (first and last chunk at once), a one-token chunk on the last slot of
    a page, a 17-token chunk from a page start across the next page boundary, and decode rows at
    contexts 0, 15, 16 and 31 (their new key first, last or second-to-last in a page)."""
    cfg = tiny_config(dtype)
    pair = _boundary_pair(cfg, 31)
    chunks = [EmbChunk(0, 0, 1, True, "mean"), EmbChunk(1, 15, 1, True, "mean"),
              EmbChunk(2, 16, 17, True, "last")]
    rows = [DecodeRow(3 + i, c) for i, c in enumerate((0, 15, 16, 31))]
    pair.step(Batch(chunks, rows, draw_tokens(31, 1, 1 + 1 + 17 + 4, cfg.vocab)))
    print(pair.report, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_batches_of_one_kind_and_the_empty_batch(dtype):
    """Embedding-only (one token), decode-only (one row at context 0), then an empty batch, which
    launches nothing and leaves every cache slot and pooling state as it was."""
    cfg = tiny_config(dtype)
    pair = _boundary_pair(cfg, 41)
    pair.step(Batch([EmbChunk(0, 0, 1, True, "cls")], [], draw_tokens(41, 1, 1, cfg.vocab)))
    pair.step(Batch([], [DecodeRow(3, 0)], draw_tokens(41, 2, 1, cfg.vocab)))
    pair.step(Batch([], [], np.zeros(0, np.int32)))
    print(pair.report, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_model_without_layers(dtype):
    """n_layers = 0: the step gathers token rows, takes the final norm, pools and runs the LM
    head; nothing is appended to the (layer-less) cache."""
    cfg = tiny_config(dtype).replace(n_layers=0)
    W = make_weights(cfg, 51)
    pk = PagedKV(cfg, 20, 4, 4, 51)
    for s in range(4):
        pk.reserve(s, 40)
    acc_w = np.zeros(4)
    acc_w[1] = 7
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=64, max_chunks=2, max_decode=2, max_ctx=64)
    chunks = [EmbChunk(0, 0, 20, True, "mean"), EmbChunk(1, 7, 9, True, "mean")]
    rows = [DecodeRow(2, 5), DecodeRow(3, 0)]
    pair.step(Batch(chunks, rows, draw_tokens(51, 1, 20 + 9 + 2, cfg.vocab)))
    print(pair.report, flush=True)


def _over_1280_rows(seed=61):
    """Tiny bf16 model, one batch of 1302 rows: chunks at offsets and of lengths that are not
    multiples of 8 (a resumed one among them) and two decode rows."""
    cfg = tiny_config("bf16")
    W = make_weights(cfg, seed, qk_std=0.09)
    n_seq, max_blocks = 5, 1400 // 16 + 1
    pk = PagedKV(cfg, n_seq * max_blocks + 3, n_seq, max_blocks, seed)
    pk.reserve(0, 700)
    pk.fill_random(1, 37, seed + 1)
    pk.reserve(1, 37 + 555)
    pk.reserve(2, 45)
    pk.fill_random(3, 100, seed + 3)
    pk.reserve(3, 101)
    pk.fill_random(4, 16, seed + 4)
    pk.reserve(4, 17)
    chunks = [EmbChunk(0, 0, 700, True, "mean"), EmbChunk(1, 37, 555, False, "mean"),
              EmbChunk(2, 0, 45, True, "last")]
    rows = [DecodeRow(3, 100), DecodeRow(4, 16)]
    batch = Batch(chunks, rows, draw_tokens(seed, 1, 700 + 555 + 45 + 2, cfg.vocab))
    acc_w = np.zeros(n_seq)
    acc_w[1] = 37
    return cfg, W, pk, batch, acc_w


def test_bf16_batch_over_1280_rows():
    """More than 1280 rows of one bf16 model: the QKV projection stores fp32 rows, which the
    16-token x one-head rotation/append kernel rotates and appends (values both as 16-byte runs
    of 8 slots and one at a time where rows do not fill them).  Every output against the oracle."""
    cfg, W, pk, batch, acc_w = _over_1280_rows()
    pair = Pair(cfg, W, pk, acc_w=acc_w)
    pair.workspace(max_tokens=batch.n_tokens, max_chunks=3, max_decode=2, max_ctx=1400)
    pair.step(batch)
    print(pair.report, flush=True)


def test_bf16_batch_over_1280_rows_flags_a_bad_page():
    """The same batch with one block-table entry past the pool: the rotation/append kernel of
    more than 256 rows flags the page error and skips that page; the step completes."""
    from paper_2609_25405_amd import runtime as R
    cfg, W, pk, batch, acc_w = _over_1280_rows()
    dm = R.DeviceModel(cfg, W)
    kv = R.DeviceKV.from_paged(pk)
    bt = pk.block_table.copy()
    bt[2, 1] = pk.n_pages                 # chunk 2's rows 16..31 point past the pool
    kv.set_block_table(bt)
    ws = R.Workspace(dm, dm, batch.n_tokens, 3, 2, 1400)
    S = torch.zeros((pk.n_seq, cfg.d_model), device="cuda")
    Wc = torch.tensor(acc_w, dtype=torch.float32, device="cuda")
    out = torch.zeros((3, cfg.d_model), device="cuda")
    lg = torch.zeros((2, cfg.vocab), device="cuda")
    R.step(dm, dm, batch, kv, kv, S, Wc, lg, out, ws)
    torch.cuda.synchronize()
    assert ws.device_error() == 1
    # the requests whose pages are all valid still get finite results
    assert torch.isfinite(lg).all()
    assert torch.isfinite(out[0]).all() and abs(out[0].norm().item() - 1.0) < 1e-3
