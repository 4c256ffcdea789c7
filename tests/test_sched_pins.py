"""Pins of the intra-batch scheduling reference model (Algorithm 2) to what the paper states.

The paper fixes the algorithm's steps and three properties (Section 4): the ratio of
embedding to generation selections converges to w_e : w_g and, for fixed weights, stays within
one scheduling opportunity of it; requests of one type are served in arrival order; persistent
credits keep a backlogged queue from starving.  It also states why chunking packs the budget:
a backlogged embedding queue leaves fewer than C tokens of the budget unused.  Each test below
checks one of these, or a hand-worked trace of the algorithm.
"""
import math
import random

import pytest

from oracle.sched import IBSOracle, SchedConfig, SchedError


def test_hand_worked_trace():
    """B = 10, C = 4; one embedding request of 6 tokens, one prompt of 5 tokens with 3 output
    tokens.  Worked by hand from the algorithm:
      iteration 1: w_e = 6, w_g = 5.  Pass 1: credits 6 vs 5 -> e (4 tokens), a_e = 6 - 11 =
        -5.  Pass 2: credits -5 + 6 = 1 vs 5 + 5 = 10, and Q_e has nothing else anyway -> g
        (4 tokens), a_g = 10 - 11 = -1.  8 tokens used; credits carried: (1, -1);
      iteration 2: w_e = 2, w_g = 1.  Pass 1: 1 + 2 = 3 >= -1 + 1 = 0 -> e (2 tokens, final),
        a_e = 3 - 3 = 0.  Pass 2: 0 + 2 = 2 vs 0 + 1 = 1, Q_e has nothing left -> g (1 token,
        final prompt chunk: first output token), a_g = 1 - 3 = -2.  Credits carried: (2, -2);
      iterations 3, 4: one decode item each, at contexts 5 and 6; the request then has its 3
      tokens and finishes."""
    s = IBSOracle(SchedConfig(budget=10, chunk=4))
    s.submit_embedding(1, 6)
    s.submit_generation(2, 5, 3)
    b = s.schedule()
    assert b.emb_chunks == [(1, 0, 4, False)] and b.gen_chunks == [(2, 0, 4, False)]
    assert b.order == ["e", "g"] and b.used == 8 and (s.a_e, s.a_g) == (1, -1)
    assert s.commit() == []
    b = s.schedule()
    assert b.emb_chunks == [(1, 4, 2, True)] and b.gen_chunks == [(2, 4, 1, True)]
    assert b.order == ["e", "g"] and (s.a_e, s.a_g) == (2, -2)
    assert b.logit_ids == [2] and b.finished == [1]
    assert s.commit() == [1]
    b = s.schedule()
    assert b.decodes == [(2, 5, 1)] and b.emb_chunks == b.gen_chunks == [] and b.used == 1
    assert (s.a_e, s.a_g) == (0, 0)      # both queues drained: credits reset
    s.commit()
    b = s.schedule()
    assert b.decodes == [(2, 6, 1)] and b.finished == [2]
    assert s.commit() == [2] and s.idle()
    assert s.schedule().used == 0


def _prefix_deviation(order, w_e, w_g):
    n_e = 0
    worst = 0.0
    for n, o in enumerate(order, 1):
        n_e += o == "e"
        worst = max(worst, abs(n_e - n * w_e / (w_e + w_g)))
    return worst


@pytest.mark.parametrize("w_e,w_g", [(300, 100), (7, 5), (1, 9), (13, 13)])
def test_proportional_share_within_one_opportunity(w_e, w_g):
    """Within one iteration the weights are fixed: one-token requests, budget large enough for
    every selection; each prefix of the selection sequence stays within one pick of w_e:w_g."""
    s = IBSOracle(SchedConfig(budget=w_e + w_g, chunk=4, emb_cache=(1000, 4096, 256)))
    for i in range(w_e):
        s.submit_embedding(i, 1)
    for i in range(w_g):
        s.submit_generation(10_000 + i, 1, 1)
    b = s.schedule()
    assert len(b.order) == w_e + w_g
    assert _prefix_deviation(b.order, w_e, w_g) <= 1.0


@pytest.mark.parametrize("w_e,w_g", [(3, 1), (1, 4), (5, 3)])
def test_persistent_credits_share_across_iterations(w_e, w_g):
    """One pick per iteration (budget 1) with queues refilled to the same weights every
    iteration: the credits carried between iterations keep the long-run ratio at w_e:w_g within
    one pick.  Credits reset every iteration would always pick the heavier queue."""
    s = IBSOracle(SchedConfig(budget=1, chunk=1))
    rid = 0
    order = []
    live_e, live_g = [], []
    for it in range(400):
        while len(live_e) < w_e:
            s.submit_embedding(rid, 1)
            live_e.append(rid)
            rid += 1
        while len(live_g) < w_g:
            s.submit_generation(rid, 1, 1)
            live_g.append(rid)
            rid += 1
        b = s.schedule()
        order += b.order
        for done in s.commit():
            (live_e if done in live_e else live_g).remove(done)
    assert len(order) == 400
    assert _prefix_deviation(order, w_e, w_g) <= 1.0
    # neither queue waits longer than its share implies
    for q, w in (("e", w_e), ("g", w_g)):
        gaps = [len(x) for x in "".join(order).split(q)[1:-1]]
        assert max(gaps, default=0) <= math.ceil((w_e + w_g) / w)


def test_one_queue_gets_all_capacity():
    for kind in ("emb", "gen"):
        s = IBSOracle(SchedConfig(budget=100, chunk=16))
        for i in range(20):
            if kind == "emb":
                s.submit_embedding(i, 10)
            else:
                s.submit_generation(i, 10, 5)
        b = s.schedule()
        assert b.used == 100
        assert len(b.emb_chunks if kind == "emb" else b.gen_chunks) == 10


def _random_trace(seed, cfg, iters=60):
    rng = random.Random(seed)
    s = IBSOracle(cfg)
    rid = 0
    log = []
    arrivals = {"emb": [], "gen": []}
    for it in range(iters):
        for _ in range(rng.randrange(0, 4)):
            if rng.random() < 0.5:
                s.submit_embedding(rid, rng.randrange(1, 300))
                arrivals["emb"].append(rid)
            else:
                s.submit_generation(rid, rng.randrange(1, 200), rng.randrange(1, 20))
                arrivals["gen"].append(rid)
            rid += 1
        b = s.schedule()
        log.append(b)
        s.commit()
    return s, log, arrivals


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("atomic", [False, True])
def test_fcfs_budget_and_chunk_invariants(seed, atomic):
    """Per type, requests are first admitted in arrival order and their chunks are contiguous;
    a request appears at most once per batch; no batch exceeds the budget; chunks never exceed
    C (whole requests in the atomic condition)."""
    cfg = SchedConfig(budget=256, chunk=64, atomic_embeddings=atomic, emb_cache=(16, 400, 32),
                      gen_cache=(16, 400, 32))
    s, log, arrivals = _random_trace(seed, cfg)
    first = {"emb": [], "gen": []}
    progress = {}
    for b in log:
        ids = [c[0] for c in b.emb_chunks + b.gen_chunks] + [d[0] for d in b.decodes]
        assert len(ids) == len(set(ids))
        assert b.used == sum(c[2] for c in b.emb_chunks + b.gen_chunks) + sum(d[2] for d in b.decodes)
        assert b.used <= cfg.budget
        for kind, chunks in (("emb", b.emb_chunks), ("gen", b.gen_chunks)):
            for rid, off, n, last in chunks:
                assert off == progress.get(rid, 0)
                if off == 0:
                    first[kind].append(rid)
                progress[rid] = off + n
                if not (kind == "emb" and atomic):
                    assert n <= cfg.chunk
                else:
                    assert off == 0 and last
    for kind in ("emb", "gen"):
        assert first[kind] == arrivals[kind][:len(first[kind])]


def test_chunking_leaves_less_than_c_unused():
    """Section 4's packing argument: with a backlogged embedding queue and capacity the only
    limit, chunks of at most C leave fewer than C budget tokens unused; whole-request
    admission can leave most of the budget idle."""
    for atomic in (False, True):
        cfg = SchedConfig(budget=256, chunk=64, atomic_embeddings=atomic, decode_tokens=8)
        s = IBSOracle(cfg)
        for i in range(25):          # running generation requests take 8 tokens each
            s.submit_generation(1000 + i, 1, 400)
        s.schedule()
        s.commit()
        for i in range(200):
            s.submit_embedding(i, 224)
        unused = []
        for _ in range(20):
            b = s.schedule()
            unused.append(cfg.budget - b.used)
            s.commit()
        if atomic:
            assert max(unused) >= 256 - 25 * 8 - 1   # a 224-token request never fits 56 tokens
        else:
            assert max(unused) < cfg.chunk


def test_cache_capacity_blocks_in_arrival_order_and_is_released():
    """A request is admitted only with a free slot and its whole page reservation; the queue
    head blocks later requests of its type (no overtaking); finishing releases the capacity."""
    cfg = SchedConfig(budget=1000, chunk=1000, emb_cache=(2, 10, 8), shared_cache=True)
    s = IBSOracle(cfg)
    s.submit_embedding(1, 100)   # 7 pages
    s.submit_embedding(2, 64)    # 4 pages: does not fit beside request 1
    s.submit_embedding(3, 16)    # 1 page: would fit, but must not overtake request 2
    b = s.schedule()
    assert [c[0] for c in b.emb_chunks] == [1]
    assert s.commit() == [1]
    b = s.schedule()
    assert [c[0] for c in b.emb_chunks] == [2, 3]
    with pytest.raises(SchedError):
        s.submit_embedding(4, 16 * 11)     # more pages than the cache holds


def test_end_of_sequence_stops_generation():
    s = IBSOracle(SchedConfig(budget=64, chunk=64, eos=7))
    s.submit_generation(1, 4, 10)
    b = s.schedule()
    assert b.logit_ids == [1]
    assert s.commit({1: 3}) == []
    b = s.schedule()
    assert b.decodes == [(1, 4, 1)]
    assert s.commit({1: 7}) == [1]
    assert s.idle()


def test_running_requests_are_served_first_in_order():
    """ScheduleRunning reserves budget for decode-phase requests before the queues get any;
    when the budget cannot hold them all, the earliest to enter the decode phase go first and
    the rest wait (no new work is admitted in front of them)."""
    s = IBSOracle(SchedConfig(budget=64, chunk=32, emb_cache=(200, 4096, 256)))
    for i in range(10):
        s.submit_generation(i, 8, 50)
    for _ in range(2):            # 80 prompt tokens: every prompt done after two iterations
        s.schedule()
        s.commit()
    for i in range(100):
        s.submit_embedding(100 + i, 300)
    seen_running = False
    for _ in range(30):
        b = s.schedule()
        running_before = [d[0] for d in b.decodes]
        if len(running_before) == 10:
            seen_running = True
            assert running_before == list(range(10))
            assert b.used == 64 and sum(c[2] for c in b.emb_chunks) == 54
        s.commit()
    assert seen_running
    # budget smaller than the decode set: the first five in phase order, nothing else
    s2 = IBSOracle(SchedConfig(budget=5, chunk=8))
    for i in range(8):
        s2.submit_generation(i, 1, 20)
    for _ in range(2):            # prompts of one token: five finish in the first iteration
        s2.schedule()
        s2.commit()
    s2.submit_embedding(99, 4)
    b = s2.schedule()
    assert [d[0] for d in b.decodes] == [0, 1, 2, 3, 4] and b.emb_chunks == [] and b.used == 5


def test_at_most_four_adapters_per_batch_in_arrival_order():
    """Six embedding requests on six adapters: the first four are admitted; the fifth would add
    a fifth adapter, so the embedding queue stops there (the sixth does not overtake it)."""
    s = IBSOracle(SchedConfig(budget=1000, chunk=64, emb_cache=(10, 400, 40)))
    for i in range(6):
        s.submit_embedding(i, 10, adapter=i)
    s.submit_embedding(6, 10, adapter=1)      # an adapter already in the batch, but behind id 4
    b = s.schedule()
    assert [c[0] for c in b.emb_chunks] == [0, 1, 2, 3] and b.emb_adapters == [0, 1, 2, 3]
    s.commit()
    b = s.schedule()
    assert [c[0] for c in b.emb_chunks] == [4, 5, 6]
