"""The whole loop (Algorithm 1) on the GPU: scheduler -> orthrus_step -> sampler -> emit.

Requests of both types are submitted to the native scheduler (some while others are running, so
sequence slots and pages are reused) and the native runner iterates until every request has
finished.  Each finished embedding is compared with the oracle's single-pass embedding of its
whole input (Section 3.3: chunked and single-pass pooling agree up to rounding), and each
generated token sequence is checked by teacher forcing: after the prompt and the tokens the
device produced so far, the oracle's full-recompute logits must make the device's next token
the greedy choice (or, where the oracle's top two are closer than the logits bound allows,
a token within that bound of the maximum).
"""
import numpy as np
import pytest
import torch

from oracle import decode_full_recompute, embed_single_pass, greedy_token
from tests.parity import TOL, assert_vectors_close
from workload import as_float64, draw_tokens, make_weights, tiny_config
from paper_2609_25405_amd import runtime as R

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"\n[case] {request.node.name}", flush=True)


def _check_generation(cfg, W64, prompt, toks, dtype):
    for k, t in enumerate(toks):
        lg = decode_full_recompute(cfg, W64, np.concatenate([prompt, np.asarray(toks[:k], np.int64)]))
        best = int(greedy_token(lg))
        top2 = np.sort(lg)[-2:]
        bound = 2 * TOL[dtype]["rel"] * np.abs(lg).max()
        if top2[1] - top2[0] > bound:
            assert t == best, (k, t, best)
        else:
            assert lg[t] >= lg.max() - bound, (k, t, best)


def _drive(runner, sched, late=None, max_iters=400):
    toks, embs, finished = {}, {}, []
    for it in range(max_iters):
        if late and it == late[0]:
            late[1]()
        out = runner.iterate()
        for rid, t in out["tokens"].items():
            toks.setdefault(rid, []).append(t)
        embs.update(out["embeddings"])
        finished += out["finished"]
        c = sched.counts()
        if out["n_items"] == 0 and c["queued_emb"] == c["queued_gen"] == c["running"] == 0 and it > (late[0] if late else 0):
            break
    assert runner.ws.device_error() == 0
    return toks, embs, finished


@pytest.mark.parametrize("dtype,qk_std", [("f32", None), ("bf16", 0.09)])
def test_runner_serves_mixed_requests_to_completion(dtype, qk_std):
    cfg = tiny_config(dtype)
    W = make_weights(cfg, 71, qk_std=qk_std)
    W64 = as_float64(W)
    dm = R.DeviceModel(cfg, W)
    n_seq, max_blocks = 6, 16
    n_pages = 60                        # fewer pages than 6 full rows: admission waits for pages
    kv = R.DeviceKV(cfg, n_pages, n_seq, max_blocks)
    sched = R.Scheduler(budget=96, chunk=32, caches=[(n_seq, n_pages, max_blocks)])
    runner = R.Runner(dm, dm, kv, kv, sched)
    reqs = {}

    def submit(rid, kind, n, extra):
        ids = draw_tokens(71, rid, n, cfg.vocab)
        reqs[rid] = (kind, ids, extra)
        if kind == "emb":
            sched.submit_embedding(rid, n, ids, extra)
        else:
            sched.submit_generation(rid, n, extra, ids)

    for rid, kind, n, extra in ((0, "emb", 70, "mean"), (1, "gen", 40, 6), (2, "emb", 33, "last"),
                                (3, "gen", 5, 4), (4, "emb", 100, "cls"), (5, "gen", 64, 1),
                                (6, "emb", 250, "mean"), (7, "gen", 150, 8)):
        submit(rid, kind, n, extra)

    def late():
        submit(8, "emb", 50, "mean")
        submit(9, "gen", 20, 3)

    toks, embs, finished = _drive(runner, sched, late=(3, late))
    assert sorted(finished) == sorted(reqs)
    for rid, (kind, ids, extra) in reqs.items():
        if kind == "emb":
            want = embed_single_pass(cfg, W64, ids, extra)
            assert_vectors_close(embs[rid][None], want[None], dtype, f"embedding {rid}")
        else:
            assert len(toks[rid]) == extra
            _check_generation(cfg, W64, ids, toks[rid], dtype)
    assert sched.counts()["free_pages0"] == n_pages and sched.counts()["free_slots0"] == n_seq


def test_runner_two_models_two_caches_and_end_of_sequence():
    cfg = tiny_config("bf16")
    We = make_weights(cfg, 81, model_tag=1, qk_std=0.09)
    Wg = make_weights(cfg, 81, model_tag=2, qk_std=0.09)
    We64, Wg64 = as_float64(We), as_float64(Wg)
    de, dg = R.DeviceModel(cfg, We), R.DeviceModel(cfg, Wg)
    kve = R.DeviceKV(cfg, 40, 4, 16)
    kvg = R.DeviceKV(cfg, 50, 5, 16)
    # the end-of-sequence id is the oracle's first token of request 11: it stops after one token
    p11 = draw_tokens(81, 11, 30, cfg.vocab)
    eos = int(greedy_token(decode_full_recompute(cfg, Wg64, p11)))
    sched = R.Scheduler(budget=80, chunk=24, caches=[(4, 40, 16), (5, 50, 16)], shared=False, eos=eos)
    runner = R.Runner(de, dg, kve, kvg, sched)
    reqs = {}
    for rid, kind, n, extra in ((10, "emb", 90, "mean"), (11, "gen", 30, 10), (12, "gen", 17, 5),
                                (13, "emb", 24, "last")):
        ids = p11 if rid == 11 else draw_tokens(81, rid, n, cfg.vocab)
        reqs[rid] = (kind, ids, extra)
        if kind == "emb":
            sched.submit_embedding(rid, n, ids, extra)
        else:
            sched.submit_generation(rid, n, extra, ids)
    toks, embs, finished = _drive(runner, sched)
    assert sorted(finished) == sorted(reqs)
    for rid, (kind, ids, extra) in reqs.items():
        if kind == "emb":
            assert_vectors_close(embs[rid][None], embed_single_pass(cfg, We64, ids, extra)[None], "bf16",
                                 f"embedding {rid}")
        else:
            t = toks[rid]
            _check_generation(cfg, Wg64, ids, t, "bf16")
            if rid == 11 and t[0] == eos:
                assert t == [eos]
            else:
                assert len(t) == extra or t[-1] == eos
