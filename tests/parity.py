"""Running the same seeded steps through the oracle and through liborthrus.so, and comparing.

Tolerances (per output vector: one logits row, one embedding, one pooling-state row):
  * fp32 path: max|gpu - oracle| / max|oracle| <= 1e-4;
  * bf16 path: cosine >= 0.999 and max|gpu - oracle| / max|oracle| <= 2e-2.
Cached key/value head vectors are intermediate state, not outputs of the step: fp32 keeps the
output bound; bf16 keeps cosine >= 0.999 with max-rel <= 4e-2.  A deeper layer's stored key is
the bf16 rounding of a projection of activations already carrying every earlier layer's bf16
rounding, and a head vector has only 64-128 entries to set its maximum; a misplaced, unrotated
or stale key is off by O(1) and fails either bound.
Bookkeeping is exact: the pooling token counts W, and the set of cache slots a step writes
(every slot the step does not own keeps its previous bytes, NaN poison included).
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import OracleKV, step_oracle
from workload import as_float64
from paper_2609_25405_amd import runtime as R

TOL = {"f32": dict(rel=1e-4, cos=None), "bf16": dict(rel=2e-2, cos=0.999)}
TOL_STATE = {"f32": dict(rel=1e-4, cos=None), "bf16": dict(rel=4e-2, cos=0.999)}


def vec_errors(g: np.ndarray, o: np.ndarray):
    g = np.asarray(g, np.float64).reshape(-1, g.shape[-1])
    o = np.asarray(o, np.float64).reshape(-1, o.shape[-1])
    rel = np.max(np.abs(g - o), axis=1) / np.maximum(np.max(np.abs(o), axis=1), 1e-30)
    cos = np.sum(g * o, axis=1) / np.maximum(np.linalg.norm(g, axis=1) * np.linalg.norm(o, axis=1), 1e-30)
    return rel, cos


def assert_vectors_close(g, o, dtype: str, what: str, tol=None):
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU values"
    rel, cos = vec_errors(g, o)
    t = (tol or TOL)[dtype]
    assert rel.max() <= t["rel"], f"{what}: max rel {rel.max():.3g} > {t['rel']}"
    if t["cos"] is not None:
        assert cos.min() >= t["cos"], f"{what}: min cos {cos.min():.6f} < {t['cos']}"
    return float(rel.max()), float(cos.min())


def written_slots(batch, block_table: np.ndarray, page: int, shared: bool):
    """(pool, page, offset) of every slot the step appends: chunk positions (embedding and
    prompt chunks) and decode positions."""
    out = []
    for c in batch.chunks:
        for p in range(c.offset, c.offset + c.len):
            out.append((0, int(block_table[0][c.seq, p // page]), p % page))
    for c in getattr(batch, "gen_chunks", []) or []:
        for p in range(c.offset, c.offset + c.len):
            out.append((0 if shared else 1, int(block_table[1][c.seq, p // page]), p % page))
    for r in batch.rows:
        p = r.ctx_len
        out.append((0 if shared else 1, int(block_table[1][r.seq, p // page]), p % page))
    return out


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


class Pair:
    """Oracle state and device state for one scenario, stepped in lockstep."""

    def __init__(self, cfg_e, W_e, paged_e, cfg_g=None, W_g=None, paged_g=None, n_seq=None,
                 acc_sum=None, acc_w=None):
        self.cfg = cfg_e
        self.dtype = cfg_e.dtype
        self.shared_model = cfg_g is None
        self.shared_kv = paged_g is None
        self.emb = (cfg_e, as_float64(W_e))
        self.gen = self.emb if self.shared_model else (cfg_g, as_float64(W_g))
        self.okv_e = OracleKV.from_paged(paged_e)
        self.okv_g = self.okv_e if self.shared_kv else OracleKV.from_paged(paged_g)
        self.dm_e = R.DeviceModel(cfg_e, W_e)
        self.dm_g = self.dm_e if self.shared_model else R.DeviceModel(cfg_g, W_g)
        self.dkv_e = R.DeviceKV.from_paged(paged_e)
        self.dkv_g = self.dkv_e if self.shared_kv else R.DeviceKV.from_paged(paged_g)
        self.bt = [paged_e.block_table, (paged_e if self.shared_kv else paged_g).block_table]
        n_seq = n_seq or paged_e.n_seq
        d = cfg_e.d_model
        self.S = np.zeros((n_seq, d)) if acc_sum is None else np.asarray(acc_sum, np.float64)
        self.W = np.zeros(n_seq) if acc_w is None else np.asarray(acc_w, np.float64)
        self.acc_sum = torch.tensor(self.S, dtype=torch.float32, device="cuda")
        self.acc_w = torch.tensor(self.W, dtype=torch.float32, device="cuda")
        self.ws = None
        self.report = []

    def workspace(self, max_tokens, max_chunks, max_decode, max_ctx):
        self.ws = R.Workspace(self.dm_e, self.dm_g, max_tokens, max_chunks, max_decode, max_ctx)

    def step(self, batch, check_kv: bool = True):
        cfg = self.cfg
        ref = step_oracle(self.emb, self.gen, batch, self.okv_e, self.okv_g, self.S, self.W)
        nc, nd = len(batch.chunks), batch.n_logit_rows
        logits = torch.full((max(1, nd), self.gen[0].vocab), float("nan"), device="cuda")
        out_emb = torch.full((max(1, nc), cfg.d_model), float("nan"), device="cuda")
        pre = [(_bits(self.dkv_e.k).clone(), _bits(self.dkv_e.v_by_position).clone())] if check_kv else None
        if check_kv and not self.shared_kv:
            pre.append((_bits(self.dkv_g.k).clone(), _bits(self.dkv_g.v_by_position).clone()))
        hidden = None
        if any(c.pool == "buffer" for c in batch.chunks):
            hidden = torch.full((self.dkv_e.n_seq, batch.hidden_stride, cfg.d_model), float("nan"),
                                device="cuda")
        R.step(self.dm_e, self.dm_g, batch, self.dkv_e, self.dkv_g, self.acc_sum, self.acc_w,
               logits, out_emb, self.ws, hidden=hidden)
        torch.cuda.synchronize()
        assert self.ws.device_error() == 0
        rec = {}
        if nd:
            rec["logits"] = assert_vectors_close(logits[:nd].cpu().numpy(), ref["logits"], self.dtype,
                                                 "logits")
        last = [i for i, c in enumerate(batch.chunks) if c.last and c.pool != "buffer"]
        if last:
            g = out_emb[last].cpu().numpy()
            o = ref["out_emb"][last]
            zero = np.all(o == 0, axis=1)     # weighted mean with all-zero weights: zero vector
            assert np.all(g[zero] == 0), "zero embedding expected"
            if (~zero).any():
                rec["emb"] = assert_vectors_close(g[~zero], o[~zero], self.dtype, "embedding")
                np.testing.assert_allclose(np.linalg.norm(g[~zero], axis=1), 1.0, rtol=1e-5)
        untouched = [i for i, c in enumerate(batch.chunks) if not c.last or c.pool == "buffer"]
        if untouched:
            assert torch.isnan(out_emb[untouched]).all(), "out_emb rows of non-final chunks written"
        if hidden is not None:
            h = hidden.cpu().numpy()
            mask = np.zeros(h.shape[:2], bool)
            for i, c in enumerate(batch.chunks):
                if c.pool == "buffer":
                    mask[c.seq, c.offset:c.offset + c.len] = True
                    rec.setdefault("hidden", [])
                    rec["hidden"].append(assert_vectors_close(h[c.seq, c.offset:c.offset + c.len],
                                                              ref["hidden"][i], self.dtype,
                                                              "buffered hidden rows"))
            assert np.isnan(h[~mask]).all(), "hidden-buffer rows outside the buffered chunks written"
        # pooling state: W exact, S per request close (rows that hold a state)
        W_gpu = self.acc_w.cpu().numpy().astype(np.float64)
        np.testing.assert_array_equal(W_gpu, ref["acc_w"])
        pooled = sorted({c.seq for c in batch.chunks if c.pool not in ("none", "buffer")})
        live = [s for s in pooled if np.any(ref["acc_sum"][s] != 0)]
        if live:
            rec["acc"] = assert_vectors_close(self.acc_sum[live].cpu().numpy(), ref["acc_sum"][live],
                                              self.dtype, "pooling state")
        self.S, self.W = ref["acc_sum"], ref["acc_w"]
        if check_kv:
            self._check_kv(batch, pre)
        self.report.append(rec)
        return ref, logits, out_emb

    def _check_kv(self, batch, pre):
        P = self.cfg.page_size
        slots = written_slots(batch, self.bt, P, self.shared_kv)
        pools = [(self.dkv_e, self.okv_e)] + ([] if self.shared_kv else [(self.dkv_g, self.okv_g)])
        for pi, (dkv, okv) in enumerate(pools):
            if dkv.k.shape[0] == 0:
                continue          # a model without layers has an empty cache
            mine = [(pg, off) for (pool, pg, off) in slots if pool == pi]
            mask = torch.zeros(dkv.k.shape[1:4], dtype=torch.bool, device="cuda")  # page, kvh, off
            if mine:
                pg = torch.tensor([m[0] for m in mine], device="cuda")
                of = torch.tensor([m[1] for m in mine], device="cuda")
                mask[pg, :, of] = True
            for which, now, before in (("k", dkv.k, pre[pi][0]), ("v", dkv.v_by_position, pre[pi][1])):
                same = _bits(now) == before
                # slots the step does not own keep their bytes in every layer
                assert bool(same[:, ~mask].all()), f"{which}: a slot outside the step changed"
                if mine:
                    # advanced indices on dims 1 and 3: results are [n, L, kvh, hd] on both sides
                    g = now[:, pg, :, of, :].float().cpu().numpy()
                    o_pool = okv.k if which == "k" else okv.v
                    o = o_pool[:, np.array([m[0] for m in mine]), :, np.array([m[1] for m in mine]), :]
                    assert_vectors_close(g, o, self.dtype, f"cached {which}", TOL_STATE)
