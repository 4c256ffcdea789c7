"""The native intra-batch scheduler (include/orthrus_sched.h) against the reference model.

Random request traces (arrivals, lengths, output lengths, pooling heads, end-of-sequence
tokens) drive liborthrus.so's scheduler and oracle.sched.IBSOracle side by side; every batch
must agree exactly: items, their order, the credit-loop picks, the credits, budget use, logits
rows and finished requests.  Beyond the model, the native batches must satisfy the step's
contract (the oracle's host validation), carry each request's tokens, and keep the block
tables consistent (live requests own disjoint pages, released rows cleared).
"""
import random

import numpy as np
import pytest

from oracle.sched import IBSOracle, SchedConfig, SchedError
from oracle.step import validate, StepError
from paper_2609_25405_amd import runtime as R
from paper_2609_25405_amd import _abi as A
from workload import Batch, DecodeRow, EmbChunk, GenChunk, tiny_config

POOLS = ("mean", "last", "cls", "wmean")


class _KVShape:
    """What the step's host validation reads of a cache."""

    def __init__(self, n_seq, max_blocks, page=16):
        self.n_seq, self.max_blocks, self.page = n_seq, max_blocks, page


def _as_step_batch(b, pools):
    chunks = [EmbChunk(s, off, n, last, pools[rid])
              for (rid, off, n, last), s in zip(b["emb_chunks"], b["slots"]["emb"])]
    gen = [GenChunk(s, off, n, last) for (rid, off, n, last), s in zip(b["gen_chunks"], b["slots"]["gen"])]
    rows = [DecodeRow(s, ctx) for (rid, ctx, k), s in zip(b["decodes"], b["slots"]["dec"])]
    return Batch(chunks, rows, b["token_ids"], gen)


def _run_pair(seed, cfg: SchedConfig, iters=80, eos_rate=0.0, vocab=50, adapters=False):
    rng = random.Random(seed)
    o = IBSOracle(cfg)
    caches = [cfg.emb_cache] if cfg.shared_cache else [cfg.emb_cache, cfg.gen_cache]
    n = R.Scheduler(cfg.budget, cfg.chunk, caches, shared=cfg.shared_cache,
                    atomic_embeddings=cfg.atomic_embeddings, decode_tokens=cfg.decode_tokens,
                    page_size=cfg.page_size, eos=cfg.eos)
    mcfg = tiny_config().replace(vocab=vocab)
    model = (mcfg, {"lm_head": np.zeros(1), "adapters": [None] * 7})
    kv_e = _KVShape(cfg.emb_cache[0], cfg.emb_cache[2])
    kv_g = kv_e if cfg.shared_cache else _KVShape(cfg.gen_cache[0], cfg.gen_cache[2])
    rid = 0
    pools, toks, history, weights = {}, {}, {}, {}
    for it in range(iters):
        for _ in range(rng.randrange(0, 4)):
            if rng.random() < 0.5:
                ln = rng.randrange(1, 300)
                pools[rid] = rng.choice(POOLS)
                toks[rid] = [rng.randrange(vocab) for _ in range(ln)]
                ad = rng.randrange(-1, 7) if adapters else -1
                wts = [rng.random() for _ in range(ln)] if pools[rid] == "wmean" else None
                weights[rid] = wts
                try:
                    o.submit_embedding(rid, ln, adapter=ad)
                    ok = True
                except SchedError:
                    ok = False
                if ok:
                    n.submit_embedding(rid, ln, toks[rid], pools[rid], weights=wts, adapter=ad)
                else:
                    with pytest.raises(A.OrthrusError):
                        n.submit_embedding(rid, ln, toks[rid], pools[rid], weights=wts, adapter=ad)
            else:
                ln, mx = rng.randrange(1, 200), rng.randrange(1, 30)
                toks[rid] = [rng.randrange(vocab) for _ in range(ln)]
                history[rid] = []
                try:
                    o.submit_generation(rid, ln, mx)
                    ok = True
                except SchedError:
                    ok = False
                if ok:
                    n.submit_generation(rid, ln, mx, toks[rid])
                else:
                    with pytest.raises(A.OrthrusError):
                        n.submit_generation(rid, ln, mx, toks[rid])
            rid += 1
        ob = o.schedule()
        nb = n.next()
        assert nb["emb_chunks"] == ob.emb_chunks
        assert nb["emb_adapters"] == ob.emb_adapters
        assert len({a for a in nb["emb_adapters"] if a >= 0}) <= A.ORTHRUS_MAX_STEP_ADAPTERS
        assert nb["gen_chunks"] == ob.gen_chunks
        assert nb["decodes"] == ob.decodes
        assert nb["order"] == ob.order
        assert nb["used"] == ob.used
        assert nb["logit_ids"] == ob.logit_ids
        assert nb["finished"] == ob.finished
        assert nb["credits"] == (o.a_e, o.a_g)
        # the batch satisfies the step's host contract and carries the requests' tokens
        sb = _as_step_batch(nb, pools)
        sb.chunk_adapter = nb["emb_adapters"]
        if any(pools[c[0]] == "wmean" for c in nb["emb_chunks"]):
            sb.token_weights = np.concatenate(
                [np.asarray(weights[c[0]][c[1]:c[1] + c[2]], np.float32) if weights[c[0]] else
                 np.ones(c[2], np.float32) for c in nb["emb_chunks"]])
        validate(model, model, sb, kv_e, kv_g)
        want = []
        for rid_, off, ln, _ in nb["emb_chunks"] + nb["gen_chunks"]:
            want += toks[rid_][off:off + ln]
        want += [history[r][-1] if history[r] else 0 for r, _, _ in nb["decodes"]]
        assert list(nb["token_ids"]) == want
        # sampled tokens, a few of them the end-of-sequence id
        sampled = [cfg.eos if (cfg.eos >= 0 and rng.random() < eos_rate) else rng.randrange(vocab)
                   for _ in nb["logit_ids"]]
        for r, t in zip(nb["logit_ids"], sampled):
            history[r].append(t)
        fin_o = o.commit(dict(zip(ob.logit_ids, sampled)))
        fin_n = n.commit(sampled if sampled else None)
        assert sorted(fin_n) == sorted(fin_o)
        _check_tables(n, cfg)
    return o, n


def _check_tables(n: R.Scheduler, cfg: SchedConfig):
    for c in range(1 if cfg.shared_cache else 2):
        bt = n.block_table(c)
        used = bt[bt >= 0]
        limits = cfg.emb_cache if c == 0 else cfg.gen_cache
        assert len(set(used.tolist())) == used.size          # pages owned once
        assert used.size == 0 or used.max() < limits[1]
        counts = n.counts()
        assert counts[f"free_pages{c}"] + used.size == limits[1]
        # rows are filled from the front: no page after a hole
        for row in bt:
            k = int((row >= 0).sum())
            assert (row[:k] >= 0).all() and (row[k:] == -1).all()


@pytest.mark.parametrize("seed", range(8))
def test_native_scheduler_matches_reference_model(seed):
    cfg = SchedConfig(budget=256, chunk=64, emb_cache=(12, 300, 40), eos=-1)
    _run_pair(seed, cfg)


@pytest.mark.parametrize("seed", range(4))
def test_native_scheduler_matches_with_adapters(seed):
    """Embedding requests naming LoRA adapters 0..5: no batch takes chunks of more than four."""
    cfg = SchedConfig(budget=256, chunk=32, emb_cache=(20, 400, 40))
    _run_pair(seed, cfg, adapters=True)


@pytest.mark.parametrize("seed", range(4))
def test_native_scheduler_matches_atomic_and_two_caches(seed):
    cfg = SchedConfig(budget=200, chunk=48, atomic_embeddings=True, shared_cache=False,
                      emb_cache=(6, 120, 20), gen_cache=(9, 150, 16))
    _run_pair(seed, cfg)


@pytest.mark.parametrize("seed", range(4))
def test_native_scheduler_matches_with_eos_and_long_decode_items(seed):
    cfg = SchedConfig(budget=96, chunk=32, decode_tokens=8, emb_cache=(10, 200, 40), eos=3)
    _run_pair(seed, cfg, eos_rate=0.15, vocab=8)


def test_native_scheduler_argument_checks():
    with pytest.raises(A.OrthrusError):
        R.Scheduler(0, 4, [(4, 10, 4)])
    s = R.Scheduler(16, 4, [(2, 8, 4)])
    with pytest.raises(A.OrthrusError) as e:
        s.submit_embedding(1, 65)                 # 5 pages > 4 block-table columns
    assert e.value.code == A.ORTHRUS_ECAPACITY
    s.submit_embedding(1, 4)
    with pytest.raises(A.OrthrusError):
        s.submit_embedding(1, 4)                  # id already live
    with pytest.raises(A.OrthrusError):
        s.submit_generation(2, 4, 0)              # max_new < 1
    s.next()
    with pytest.raises(A.OrthrusError):
        s.next()                                  # previous batch not committed
    with pytest.raises(A.OrthrusError):
        s.commit([1, 2])                          # no logits rows in this batch
    assert s.commit() == [1]
    with pytest.raises(A.OrthrusError):
        s.block_table(1)                          # shared configuration has one cache
