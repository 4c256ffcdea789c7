"""orthrus_step_noalloc (the step on library-owned scratch, for callers that cannot allocate)
against orthrus_step with a caller workspace: the same batches on two identical copies of every
input, outputs and caches compared bit for bit (the same kernels in the same order).

Two calls in a row, the second with a smaller batch (the scratch keeps the first call's
contents), on one bf16 model and on two models with two caches (whose row groups run one after
the other on the caller's stream instead of concurrently); a block-table entry past the pool
reports its error bit through the caller's word and the next call starts clean; a batch that
needs more than the scratch is rejected before anything is enqueued.
"""
import numpy as np
import pytest
import torch

from paper_2609_25405_amd import _abi as A
from paper_2609_25405_amd import runtime as R
from workload import Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, draw_tokens, make_weights

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _cfg():
    return ModelConfig(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128, d_ff=1024,
                       vocab=512, dtype="bf16")


class Side:
    """One copy of a step's mutable state: caches, pooling state, outputs."""

    def __init__(self, cfg, pk_e, pk_g, n_seq_e, n_chunks, n_logits):
        self.kv_e = R.DeviceKV.from_paged(pk_e)
        self.kv_g = self.kv_e if pk_g is None else R.DeviceKV.from_paged(pk_g)
        self.S = torch.zeros((n_seq_e, cfg.d_model), device="cuda")
        self.W = torch.zeros(n_seq_e, device="cuda")
        self.logits = torch.full((max(1, n_logits), cfg.vocab), float("nan"), device="cuda")
        self.emb = torch.full((max(1, n_chunks), cfg.d_model), float("nan"), device="cuda")

    def state(self):
        t = [self.S, self.W, self.logits, self.emb, self.kv_e.k, self.kv_e.v]
        if self.kv_g is not self.kv_e:
            t += [self.kv_g.k, self.kv_g.v]
        return [x.clone() for x in t]


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def run_both(dm_e, dm_g, pk_e, pk_g, batches, n_seq_e):
    cfg = dm_e.cfg
    n_chunks = max(len(b.chunks) + len(b.gen_chunks) for b in batches)
    n_logits = max(b.n_logit_rows for b in batches)
    a = Side(cfg, pk_e, pk_g, n_seq_e, n_chunks, n_logits)
    b = Side(cfg, pk_e, pk_g, n_seq_e, n_chunks, n_logits)
    ws = R.Workspace(dm_e, dm_g, max(x.n_tokens for x in batches), n_chunks, max(len(x.rows) for x in batches),
                     2048)
    err = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    for i, batch in enumerate(batches):
        R.step(dm_e, dm_g, batch, a.kv_e, a.kv_g, a.S, a.W, a.logits, a.emb, ws)
        rc = R.step_noalloc(dm_e, dm_g, batch, b.kv_e, b.kv_g, b.S, b.W, b.logits, b.emb, err)
        assert rc == A.ORTHRUS_OK, rc
        torch.cuda.synchronize()
        assert ws.device_error() == 0
        assert int(err.item()) == 0
        for x, y in zip(a.state(), b.state()):
            assert torch.equal(_bits(x), _bits(y)), f"call {i}: outputs differ"
        print(f"call {i}: {batch.n_tokens} tokens identical", flush=True)
    return a, b, err


def test_noalloc_step_equals_workspace_step_one_model():
    cfg = _cfg()
    W = make_weights(cfg, 2301, qk_std=0.06)
    dm = R.DeviceModel(cfg, W)
    n_seq = 6
    pk = PagedKV(cfg, n_seq * 40, n_seq, 40, 2301)
    for s, c in ((3, 300), (4, 17), (5, 600)):
        pk.fill_random(s, c, 2301)
    for s, n in ((0, 400), (1, 200), (2, 60), (3, 303), (4, 20), (5, 603)):
        pk.reserve(s, n)
    big = Batch([EmbChunk(0, 0, 256, False, "mean"), EmbChunk(1, 0, 150, True, "last")],
                [DecodeRow(3, 300), DecodeRow(4, 17), DecodeRow(5, 600)], draw_tokens(2301, 1, 256 + 150 + 40 + 3, 512),
                gen_chunks=[GenChunk(2, 0, 40, True)])
    small = Batch([EmbChunk(0, 256, 20, True, "mean")], [DecodeRow(3, 301)], draw_tokens(2301, 2, 21, 512))
    run_both(dm, dm, pk, None, [big, small], n_seq)


def test_noalloc_step_equals_workspace_step_two_models():
    cfg = _cfg()
    dm_e = R.DeviceModel(cfg, make_weights(cfg, 2302, model_tag=1, qk_std=0.06))
    dm_g = R.DeviceModel(cfg, make_weights(cfg, 2302, model_tag=2, qk_std=0.06))
    pe = PagedKV(cfg, 64, 4, 16, 1)
    pg = PagedKV(cfg, 64, 4, 16, 2)
    for s in range(4):
        pe.reserve(s, 200)
        pg.fill_random(s, 40 + 30 * s, 3)
        pg.reserve(s, 42 + 30 * s)
    big = Batch([EmbChunk(0, 0, 120, True, "mean"), EmbChunk(1, 0, 64, False, "cls")],
                [DecodeRow(s, 40 + 30 * s) for s in range(4)], draw_tokens(2302, 3, 120 + 64 + 4, 512))
    small = Batch([EmbChunk(1, 64, 10, True, "cls")], [DecodeRow(2, 101)], draw_tokens(2302, 4, 11, 512))
    run_both(dm_e, dm_g, pe, pg, [big, small], 4)


def test_noalloc_two_models_wide_generator_group():
    """A generator group of 129..256 decode rows beside the embedding rows: the two-stream step gives
    that group's split-K projections 256x256 tiles, the allocation-free one-stream step 128x128;
    each output element sums the same K stages in the same order either way, so bitwise equal."""
    cfg = _cfg()
    dm_e = R.DeviceModel(cfg, make_weights(cfg, 2305, model_tag=1, qk_std=0.06))
    dm_g = R.DeviceModel(cfg, make_weights(cfg, 2305, model_tag=2, qk_std=0.06))
    n_g = 200
    pe = PagedKV(cfg, 64, 4, 16, 1)
    pg = PagedKV(cfg, n_g * 8, n_g, 8, 2)
    for s in range(4):
        pe.reserve(s, 200)
    ctx = [20 + (37 * s) % 90 for s in range(n_g)]
    for s, c in enumerate(ctx):
        pg.fill_random(s, c, 5)
        pg.reserve(s, c + 2)
    big = Batch([EmbChunk(0, 0, 180, True, "mean"), EmbChunk(1, 0, 120, False, "cls")],
                [DecodeRow(s, ctx[s]) for s in range(n_g)], draw_tokens(2305, 3, 180 + 120 + n_g, 512))
    small = Batch([EmbChunk(1, 120, 30, True, "cls")], [DecodeRow(s, ctx[s] + 1) for s in range(150)],
                  draw_tokens(2305, 4, 30 + 150, 512))
    run_both(dm_e, dm_g, pe, pg, [big, small], 4)


def test_noalloc_error_bits_and_capacity():
    cfg = _cfg()
    dm = R.DeviceModel(cfg, make_weights(cfg, 2303))
    pk = PagedKV(cfg, 300, 3, 260, 2303)
    for s in range(3):
        pk.reserve(s, 64)
    kv = R.DeviceKV.from_paged(pk)
    S = torch.zeros((3, cfg.d_model), device="cuda")
    Wc = torch.zeros(3, device="cuda")
    lg = torch.zeros((1, cfg.vocab), device="cuda")
    out = torch.zeros((1, cfg.d_model), device="cuda")
    err = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    bt = pk.block_table.copy()
    bt[1, 0] = pk.n_pages                                 # one past the pool: flagged, not read
    kv.set_block_table(bt)
    ids = draw_tokens(2303, 1, 16, cfg.vocab)
    assert R.step_noalloc(dm, dm, Batch([], [DecodeRow(1, 3)], ids[:1]), kv, kv, S, Wc, lg, None, err) == 0
    torch.cuda.synchronize()
    assert int(err.item()) == A.ORTHRUS_DEVERR_PAGE
    assert R.step_noalloc(dm, dm, Batch([], [DecodeRow(2, 3)], ids[:1]), kv, kv, S, Wc, lg, None, err) == 0
    torch.cuda.synchronize()
    assert int(err.item()) == 0                           # the next call starts clean
    # a 4096-token chunk needs more workspace than the scratch holds: rejected, nothing enqueued
    n = 4096
    need = A.orthrus_workspace_bytes(dm.handle, dm.handle, n, 1, 0, n)
    assert need > A.ORTHRUS_SCRATCH_BYTES
    pk2 = PagedKV(cfg, n // 16 + 1, 1, n // 16, 2304)
    pk2.reserve(0, n)
    kv2 = R.DeviceKV.from_paged(pk2)
    before = kv2.k.clone()
    err.fill_(-1)
    big = Batch([EmbChunk(0, 0, n, False, "none")], [], draw_tokens(2304, 1, n, cfg.vocab))
    assert R.step_noalloc(dm, dm, big, kv2, kv2, S[:1], Wc[:1], None, out, err) == A.ORTHRUS_ECAPACITY
    torch.cuda.synchronize()
    assert int(err.item()) == -1 and torch.equal(_bits(kv2.k), _bits(before))
