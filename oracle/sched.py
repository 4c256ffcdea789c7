"""Intra-batch scheduling (Algorithm 2) as a plain reference model (test infrastructure only).

One call of ``schedule()`` builds the batch of one iteration of the inference loop
(Algorithm 1): first ScheduleRunning reserves budget for generation requests in the decode
phase, then the credit loop of Algorithm 2 alternates between the embedding queue Q_e and the
generation queue Q_g with ScheduleOne, until the token budget B is used up or neither queue can
contribute.  ``commit()`` ends the iteration (frees what finished, applies early stops).

The model counts tokens, pages and sequence slots; it does no arithmetic of the forward pass.

Readings taken where the paper leaves a detail open (also listed in the design notes):
* ScheduleOne admits one item per request per iteration (a request appears at most once in a
  batch).  It takes the first request of its queue, in arrival order, that is not yet in the
  batch; its chunk is min(C, remaining tokens, remaining budget) tokens.  With whole-request
  embeddings (the atomic condition of the packing simulation) an embedding request is admitted
  only if all its remaining tokens fit the remaining budget.  If that request cannot be admitted
  (budget or cache capacity), the queue contributes nothing more this iteration: requests of
  one type are served in arrival order, so a later request never overtakes it.
* In the loop of Algorithm 2, "queue nonempty" means "the queue can contribute this
  iteration" as above; the credit reset at the top uses plain emptiness.  The weights w_e, w_g
  are the remaining (not yet scheduled) tokens of the queued requests, computed once per
  iteration before the loop, as the algorithm does.  Credits are exact integers.
* ScheduleRunning gives every decode-phase request its next decode item, in the order the
  requests entered that phase, while the budget holds it; the first one that does not fit waits
  with every later one (no swapping: that needs a host-side KV store).  A decode item advances
  a request by ``decode_tokens`` tokens (1 for the real step) or what remains of its output.
* Cache capacity is reserved whole at a request's first admission: a sequence slot plus the
  pages of every position it will ever write (embedding: its n tokens; generation: prompt +
  max_new - 1 positions, the last sampled token is never fed back), released when it finishes.
  Running requests therefore never wait for pages, and no preemption is needed.  With one cache
  for both models the two request types draw on the same slots and pages.
* A generation request's final prompt chunk yields its first output token; it then enters the
  decode phase (from the next iteration) unless max_new == 1.  Decode item of a request with g
  tokens generated so far: input position n + g - 1, i.e. ``ctx_len`` = n + g - 1 cached tokens.
* A sampled token equal to the end-of-sequence id (if one is set) ends the request at commit.
* An embedding request may name a LoRA adapter; a batch holds chunks of at most four distinct
  adapters (the step's limit), so an embedding request whose adapter would be a fifth cannot be
  admitted this iteration (its queue stops contributing, as for any request that does not fit).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional


@dataclass
class SchedConfig:
    budget: int                  # B: tokens per iteration
    chunk: int                   # C: most tokens of one embedding or prompt chunk
    atomic_embeddings: bool = False
    decode_tokens: int = 1
    page_size: int = 16
    emb_cache: tuple = (64, 4096, 256)   # (n_seq, n_pages, max_blocks)
    gen_cache: tuple = (64, 4096, 256)
    shared_cache: bool = True
    eos: int = -1


@dataclass
class _Req:
    id: int
    kind: str                    # "emb" or "gen"
    n: int                       # embedding input length or prompt length
    max_new: int = 0
    pool: int = 0
    adapter: int = -1
    done: int = 0                # input tokens scheduled so far
    generated: int = 0
    admitted: bool = False
    pages: int = 0

    @property
    def remaining(self) -> int:
        return self.n - self.done


@dataclass
class Schedule:
    emb_chunks: List[tuple] = field(default_factory=list)   # (id, offset, len, last)
    emb_adapters: List[int] = field(default_factory=list)   # adapter of each embedding chunk
    gen_chunks: List[tuple] = field(default_factory=list)   # (id, offset, len, last)
    decodes: List[tuple] = field(default_factory=list)      # (id, ctx_len, tokens)
    order: List[str] = field(default_factory=list)          # "e" / "g" per credit-loop pick
    used: int = 0
    logit_ids: List[int] = field(default_factory=list)      # final prompt chunks, then decodes
    finished: List[int] = field(default_factory=list)       # requests that end with this batch


class SchedError(Exception):
    pass


MAX_STEP_ADAPTERS = 4


def _pages(n_positions: int, page: int) -> int:
    return -(-n_positions // page)


class IBSOracle:
    """Reference model of Algorithm 2 with ScheduleRunning and ScheduleOne."""

    def __init__(self, cfg: SchedConfig):
        if cfg.budget < 1 or cfg.chunk < 1 or cfg.decode_tokens < 1 or cfg.page_size < 1:
            raise SchedError("bad config")
        self.cfg = cfg
        self.Qe: List[_Req] = []
        self.Qg: List[_Req] = []
        self.running: List[_Req] = []
        self.a_e = 0
        self.a_g = 0
        self.reqs: Dict[int, _Req] = {}
        # free slots and pages per cache; one shared entry when the models share a cache
        caches = [cfg.emb_cache] if cfg.shared_cache else [cfg.emb_cache, cfg.gen_cache]
        self.free_slots = [c[0] for c in caches]
        self.free_pages = [c[1] for c in caches]
        self.pending: Optional[Schedule] = None

    def _cache(self, kind: str) -> int:
        return 0 if (self.cfg.shared_cache or kind == "emb") else 1

    def _limits(self, kind: str):
        return self.cfg.emb_cache if kind == "emb" or self.cfg.shared_cache else self.cfg.gen_cache

    def _reservation(self, r: _Req) -> int:
        positions = r.n if r.kind == "emb" else r.n + r.max_new - 1
        return _pages(positions, self.cfg.page_size)

    # -- requests
    def submit_embedding(self, rid: int, n: int, pool: int = 0, adapter: int = -1) -> None:
        self._submit(_Req(rid, "emb", n, pool=pool, adapter=adapter))

    def submit_generation(self, rid: int, n: int, max_new: int) -> None:
        self._submit(_Req(rid, "gen", n, max_new=max_new))

    def _submit(self, r: _Req) -> None:
        if r.id in self.reqs or r.n < 1 or (r.kind == "gen" and r.max_new < 1):
            raise SchedError(f"bad request {r}")
        n_seq, n_pages, max_blocks = self._limits(r.kind)
        need = self._reservation(r)
        if need > max_blocks or need > n_pages:
            raise SchedError(f"request {r.id} can never fit the cache")
        self.reqs[r.id] = r
        (self.Qe if r.kind == "emb" else self.Qg).append(r)

    # -- one iteration
    def schedule(self) -> Schedule:
        if self.pending is not None:
            raise SchedError("commit the previous batch first")
        cfg = self.cfg
        out = Schedule()
        B = cfg.budget
        in_batch = set()
        # ScheduleRunning: decode-phase requests first, in the order they entered that phase
        still = []
        blocked = False
        for r in self.running:
            k = min(cfg.decode_tokens, r.max_new - r.generated)
            if blocked or k > B:
                blocked = True
                still.append(r)
                continue
            out.decodes.append((r.id, r.n + r.generated - 1, k))
            out.logit_ids.append(r.id)
            in_batch.add(r.id)
            B -= k
            r.generated += k
            if r.generated == r.max_new:
                out.finished.append(r.id)
            else:
                still.append(r)
        self.running = still
        decode_logits = list(out.logit_ids)
        out.logit_ids = []
        # Algorithm 2: proportional selection from the two queues
        w_e = sum(r.remaining for r in self.Qe)
        w_g = sum(r.remaining for r in self.Qg)
        if not self.Qe:
            self.a_e = 0
        if not self.Qg:
            self.a_g = 0
        blocked_q = {"e": False, "g": False}
        self._adapters = set()
        while B > 0:
            ce = None if blocked_q["e"] else self._candidate(self.Qe, B, in_batch)
            cg = None if blocked_q["g"] else self._candidate(self.Qg, B, in_batch)
            if ce is None:
                blocked_q["e"] = True
            if cg is None:
                blocked_q["g"] = True
            if ce is None and cg is None:
                break
            self.a_e += w_e
            self.a_g += w_g
            if cg is None or (ce is not None and self.a_e >= self.a_g):
                r, n = ce
                self._admit(r, n, out, in_batch)
                self.a_e -= w_e + w_g
                out.order.append("e")
            else:
                r, n = cg
                self._admit(r, n, out, in_batch)
                self.a_g -= w_e + w_g
                out.order.append("g")
            B -= n
        out.used = cfg.budget - B
        out.logit_ids = out.logit_ids + decode_logits
        self.pending = out
        return out

    def _candidate(self, Q: List[_Req], B: int, in_batch: set):
        """(request, chunk length) ScheduleOne would admit from Q, or None."""
        r = next((q for q in Q if q.id not in in_batch), None)
        if r is None:
            return None
        if r.kind == "emb" and self.cfg.atomic_embeddings:
            if r.remaining > B:
                return None
            n = r.remaining
        else:
            n = min(self.cfg.chunk, r.remaining, B)
        if not r.admitted:
            c = self._cache(r.kind)
            if self.free_slots[c] < 1 or self.free_pages[c] < self._reservation(r):
                return None
        if r.adapter >= 0 and r.adapter not in self._adapters and len(self._adapters) == MAX_STEP_ADAPTERS:
            return None
        return r, n

    def _admit(self, r: _Req, n: int, out: Schedule, in_batch: set) -> None:
        if not r.admitted:
            c = self._cache(r.kind)
            r.pages = self._reservation(r)
            self.free_slots[c] -= 1
            self.free_pages[c] -= r.pages
            r.admitted = True
        last = r.done + n == r.n
        item = (r.id, r.done, n, last)
        r.done += n
        in_batch.add(r.id)
        if r.kind == "emb":
            out.emb_chunks.append(item)
            out.emb_adapters.append(r.adapter)
            if r.adapter >= 0:
                self._adapters.add(r.adapter)
            if last:
                self.Qe.remove(r)
                out.finished.append(r.id)
        else:
            out.gen_chunks.append(item)
            if last:
                self.Qg.remove(r)
                out.logit_ids.append(r.id)
                r.generated = 1
                if r.generated == r.max_new:
                    out.finished.append(r.id)
                else:
                    self.running.append(r)

    def commit(self, sampled: Optional[Dict[int, int]] = None) -> List[int]:
        """End the iteration: requests whose sampled token is the end-of-sequence id stop;
        every request that finished releases its slot and pages.  Returns the finished ids."""
        if self.pending is None:
            raise SchedError("no batch to commit")
        out = self.pending
        self.pending = None
        done = list(out.finished)
        if sampled and self.cfg.eos >= 0:
            for rid, tok in sampled.items():
                r = self.reqs[rid]
                if tok == self.cfg.eos and rid not in done:
                    done.append(rid)
                    self.running = [q for q in self.running if q.id != rid]
        for rid in done:
            r = self.reqs.pop(rid)
            c = self._cache(r.kind)
            self.free_slots[c] += 1
            self.free_pages[c] += r.pages
        return done

    def idle(self) -> bool:
        return not (self.Qe or self.Qg or self.running)
