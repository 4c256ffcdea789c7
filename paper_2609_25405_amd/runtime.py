"""Device memory for the step, held in torch tensors, and the marshalling around orthrus_step.

PyTorch is used only to allocate device memory, copy inputs in and outputs out, and hand a
HIP stream to the library; every arithmetic step of the forward runs in liborthrus.so.
"""
from __future__ import annotations

import ctypes
from ctypes import POINTER, byref, c_int32, c_void_p
from typing import Optional

import numpy as np
import torch

from . import _abi as A

POOL_CODES = {"mean": A.ORTHRUS_POOL_MEAN, "last": A.ORTHRUS_POOL_LAST,
              "cls": A.ORTHRUS_POOL_CLS, "none": A.ORTHRUS_POOL_NONE,
              "wmean": A.ORTHRUS_POOL_WMEAN, "buffer": A.ORTHRUS_POOL_BUFFER}


def _vp(t: Optional[torch.Tensor]):
    return None if t is None else c_void_p(t.data_ptr())


def _check(rc: int, where: str) -> None:
    if rc != A.ORTHRUS_OK:
        raise A.OrthrusError(rc, where)


def torch_dtype(cfg) -> torch.dtype:
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def abi_config(cfg) -> A.orthrus_config:
    return A.orthrus_config(cfg.n_layers, cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                            cfg.d_ff, cfg.vocab, cfg.page_size, cfg.rope_base, cfg.rms_eps,
                            A.ORTHRUS_BF16 if cfg.dtype == "bf16" else A.ORTHRUS_F32)


class DeviceModel:
    """Weights uploaded to the GPU in the model dtype (norm gains fp32) plus the library handle.

    bf16 models with an LM head also get its 64 x 64 blocked copy (orthrus_block_weights), which
    the step's LM head GEMM then reads; ``block_lm_head=False`` keeps the row-major one only."""

    def __init__(self, cfg, weights, device="cuda", block_lm_head: bool = True):
        self.cfg = cfg
        dt = torch_dtype(cfg)

        def up(a, dtype=dt):
            if isinstance(a, torch.Tensor):      # already on the device (drawn there)
                return a.to(device=device, dtype=dtype).contiguous()
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device=device, dtype=dtype)

        self.tok_emb = up(weights["tok_emb"])
        self.final_norm = up(weights["final_norm"], torch.float32)
        self.lm_head = up(weights["lm_head"]) if weights.get("lm_head") is not None else None
        self.layers = []
        for lw in weights["layers"]:
            self.layers.append({k: up(v, torch.float32 if k.endswith("norm") else dt)
                                for k, v in lw.items()})
        n = max(1, len(self.layers))
        self._lw = (A.orthrus_layer_weights * n)()
        for i, lw in enumerate(self.layers):
            self._lw[i] = A.orthrus_layer_weights(*[_vp(lw[k]) for k in (
                "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")])
        self.lm_head_blocked = None
        if (block_lm_head and self.lm_head is not None and cfg.dtype == "bf16"
                and torch.device(device).type == "cuda"):
            V, d = self.lm_head.shape
            nb = A.orthrus_blocked_bytes(V, d)
            if nb == 0:
                raise A.OrthrusError(A.ORTHRUS_EINVAL, "orthrus_blocked_bytes")
            self.lm_head_blocked = torch.empty(nb // 2, dtype=torch.bfloat16, device=device)
            _check(A.orthrus_block_weights(_vp(self.lm_head), _vp(self.lm_head_blocked), V, d,
                                           c_void_p(current_stream())), "orthrus_block_weights")
            torch.cuda.current_stream().synchronize()   # steps may run on another stream
        self._w = A.orthrus_weights(_vp(self.tok_emb), _vp(self.final_norm), _vp(self.lm_head),
                                    ctypes.cast(self._lw, POINTER(A.orthrus_layer_weights)),
                                    _vp(self.lm_head_blocked))
        self._cfg = abi_config(cfg)
        h = c_void_p()
        _check(A.orthrus_model_create(byref(self._cfg), byref(self._w), byref(h)),
               "orthrus_model_create")
        self.handle = h
        self.adapters = []
        if weights.get("adapters"):
            self.set_adapters(weights["adapters"], device)

    def set_adapters(self, adapters, device="cuda"):
        """Upload LoRA adapters (workload.make_lora layout: per layer {site: (A, B) or
        (A, B_gate, B_up)}) and register them with the library."""
        dt = torch_dtype(self.cfg)

        def up(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device=device, dtype=dt)

        L = len(self.layers)
        self.adapters = []
        arr = (A.orthrus_lora * max(1, len(adapters)))()
        self._lora_keep = []
        for i, ad in enumerate(adapters):
            lls = (A.orthrus_lora_layer * max(1, L))()
            tensors = []
            ranks = [0, 0, 0, 0]
            for l, ll in enumerate(ad["layers"]):
                t = {k: tuple(up(x) for x in v) for k, v in ll.items()}
                tensors.append(t)
                f = {}
                if "qkv" in t:
                    f.update(qkv_a=_vp(t["qkv"][0]), qkv_b=_vp(t["qkv"][1]))
                    ranks[0] = t["qkv"][0].shape[0]
                if "o" in t:
                    f.update(o_a=_vp(t["o"][0]), o_b=_vp(t["o"][1]))
                    ranks[1] = t["o"][0].shape[0]
                if "gate_up" in t:
                    f.update(gate_up_a=_vp(t["gate_up"][0]), gate_b=_vp(t["gate_up"][1]),
                             up_b=_vp(t["gate_up"][2]))
                    ranks[2] = t["gate_up"][0].shape[0]
                if "down" in t:
                    f.update(down_a=_vp(t["down"][0]), down_b=_vp(t["down"][1]))
                    ranks[3] = t["down"][0].shape[0]
                lls[l] = A.orthrus_lora_layer(**f)
            arr[i].rank[:] = ranks
            arr[i].scale = float(ad["scale"])
            arr[i].layers = ctypes.cast(lls, POINTER(A.orthrus_lora_layer))
            self._lora_keep.append(lls)
            self.adapters.append(tensors)
        _check(A.orthrus_model_set_adapters(self.handle, arr, len(adapters)),
               "orthrus_model_set_adapters")

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            A.orthrus_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DeviceKV:
    """Paged KV pools and the int32 block table, on the GPU.

    Keys are [L][n_pages][n_kv][page][hd] (position-major inside a page), values
    [L][n_pages][n_kv][hd][page] (dim-major inside a page), the layouts include/orthrus.h fixes.
    ``v_by_position`` is a [L][n_pages][n_kv][page][hd] view of the values.
    """

    def __init__(self, cfg, n_pages: int, n_seq: int, max_blocks: int, device="cuda",
                 fill: float = float("nan")):
        self.cfg = cfg
        L, P, kvh, hd = cfg.n_layers, cfg.page_size, cfg.n_kv_heads, cfg.head_dim
        dt = torch_dtype(cfg)
        self.k = torch.full((L, n_pages, kvh, P, hd), fill, dtype=dt, device=device)
        self.v = torch.full((L, n_pages, kvh, hd, P), fill, dtype=dt, device=device)
        self.block_table = torch.full((n_seq, max_blocks), -1, dtype=torch.int32, device=device)
        self.n_pages, self.n_seq, self.max_blocks = n_pages, n_seq, max_blocks

    @classmethod
    def from_paged(cls, paged, device="cuda") -> "DeviceKV":
        """Upload a host image whose pools are both [L][n_pages][n_kv][page][hd]."""
        kv = cls.__new__(cls)
        kv.cfg = paged.cfg
        dt = torch_dtype(paged.cfg)
        kv.k = torch.from_numpy(paged.k).to(device=device, dtype=dt)
        kv.v = torch.from_numpy(paged.v).to(device=device, dtype=dt).transpose(-1, -2).contiguous()
        kv.block_table = torch.from_numpy(paged.block_table).to(device)
        kv.n_pages, kv.n_seq, kv.max_blocks = paged.n_pages, paged.n_seq, paged.max_blocks
        return kv

    @property
    def v_by_position(self) -> torch.Tensor:
        return self.v.transpose(-1, -2)

    def set_block_table(self, bt: np.ndarray) -> None:
        self.block_table.copy_(torch.from_numpy(np.ascontiguousarray(bt, np.int32)))

    def struct(self) -> A.orthrus_kv:
        return A.orthrus_kv(_vp(self.k), _vp(self.v), _vp(self.block_table), self.n_pages,
                            self.n_seq, self.max_blocks)


class Workspace:
    def __init__(self, emb: DeviceModel, gen: DeviceModel, max_tokens: int, max_chunks: int,
                 max_decode: int, max_ctx: int, device="cuda"):
        n = A.orthrus_workspace_bytes(emb.handle, gen.handle, max_tokens, max_chunks, max_decode,
                                      max_ctx)
        if n == 0:
            raise A.OrthrusError(A.ORTHRUS_EINVAL, "orthrus_workspace_bytes")
        self.nbytes = int(n)
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        _check(A.orthrus_workspace_init(_vp(self.buf), c_void_p(current_stream())),
               "orthrus_workspace_init")

    def device_error(self) -> int:
        bits = c_int32(0)
        rc = A.orthrus_device_error(_vp(self.buf), c_void_p(current_stream()), byref(bits))
        if rc not in (A.ORTHRUS_OK, A.ORTHRUS_EDEVICE):
            raise A.OrthrusError(rc, "orthrus_device_error")
        return bits.value


def current_stream() -> int:
    # the null stream when no GPU is present (host-side validation paths only)
    return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else 0


class PackedBatch:
    """ctypes image of a workload Batch (host memory, kept alive with this object)."""

    def __init__(self, batch):
        nc, nd = len(batch.chunks), len(batch.rows)
        self._chunks = (A.orthrus_emb_chunk * max(1, nc))()
        for i, c in enumerate(batch.chunks):
            flags = (A.ORTHRUS_CHUNK_LAST if c.last else 0) | (POOL_CODES[c.pool] << A.ORTHRUS_POOL_SHIFT)
            self._chunks[i] = A.orthrus_emb_chunk(int(c.seq), int(c.offset), int(c.len), flags)
        self._rows = (A.orthrus_decode_row * max(1, nd))()
        for j, r in enumerate(batch.rows):
            self._rows[j] = A.orthrus_decode_row(int(r.seq), int(r.ctx_len))
        gen = list(getattr(batch, "gen_chunks", []) or [])
        ng = len(gen)
        self._gen = (A.orthrus_gen_chunk * max(1, ng))()
        for i, c in enumerate(gen):
            self._gen[i] = A.orthrus_gen_chunk(int(c.seq), int(c.offset), int(c.len),
                                               A.ORTHRUS_CHUNK_LAST if c.last else 0)
        self._ids = np.ascontiguousarray(batch.token_ids, dtype=np.int32)
        # the C side reads every chunk token and one id per decode row through a bare pointer:
        # check the length here
        n_ids = sum(int(c.len) for c in batch.chunks) + sum(int(c.len) for c in gen) + nd
        if self._ids.shape != (n_ids,):
            raise A.OrthrusError(A.ORTHRUS_EDESC, "token_ids length")
        self.n_logit_rows = sum(1 for c in gen if c.last) + nd
        # per-token weights of the embedding chunks (weighted-mean heads), bounds-checked here
        tw = getattr(batch, "token_weights", None)
        n_emb = sum(int(c.len) for c in batch.chunks)
        self._w = None
        wptr = None
        if tw is not None:
            self._w = np.ascontiguousarray(tw, dtype=np.float32)
            if self._w.shape != (n_emb,):
                raise A.OrthrusError(A.ORTHRUS_EDESC, "token_weights length")
            wptr = self._w.ctypes.data_as(POINTER(ctypes.c_float))
        ca = getattr(batch, "chunk_adapter", None)
        self._ca = None
        captr = None
        if ca is not None:
            self._ca = np.ascontiguousarray(ca, dtype=np.int32)
            if self._ca.shape != (nc,):
                raise A.OrthrusError(A.ORTHRUS_EDESC, "chunk_adapter length")
            captr = self._ca.ctypes.data_as(POINTER(c_int32))
        self.c = A.orthrus_batch(nc, nd, ctypes.cast(self._chunks, POINTER(A.orthrus_emb_chunk)),
                                 ctypes.cast(self._rows, POINTER(A.orthrus_decode_row)),
                                 self._ids.ctypes.data_as(POINTER(c_int32)), ng,
                                 ctypes.cast(self._gen, POINTER(A.orthrus_gen_chunk)), wptr, None,
                                 int(getattr(batch, "hidden_stride", 0)), captr)


def step(emb: DeviceModel, gen: DeviceModel, batch, emb_kv: DeviceKV, gen_kv: DeviceKV,
         acc_sum: torch.Tensor, acc_w: torch.Tensor, out_logits: Optional[torch.Tensor],
         out_emb: Optional[torch.Tensor], ws: Workspace, stream: Optional[int] = None,
         packed: Optional[PackedBatch] = None, hidden: Optional[torch.Tensor] = None) -> None:
    """Enqueue one orthrus_step on `stream` (default: torch's current stream); raises on error.
    ``hidden``: fp32 [n_seq][hidden_stride][d] buffer that buffered-head chunks fill."""
    pb = packed if packed is not None else PackedBatch(batch)
    if hidden is not None:
        if hidden.dtype != torch.float32 or not hidden.is_contiguous() or hidden.dim() != 3 or \
                hidden.shape[0] < emb_kv.n_seq or hidden.shape[1] != pb.c.hidden_stride or \
                hidden.shape[2] != emb.cfg.d_model:
            raise A.OrthrusError(A.ORTHRUS_EINVAL, "hidden buffer shape")
        pb.c.hidden = hidden.data_ptr()
    ekv, gkv = emb_kv.struct(), (emb_kv.struct() if gen_kv is emb_kv else gen_kv.struct())
    s = current_stream() if stream is None else stream
    rc = A.orthrus_step(emb.handle, gen.handle, byref(pb.c), byref(ekv), byref(gkv), _vp(acc_sum),
                        _vp(acc_w), _vp(out_logits), _vp(out_emb), _vp(ws.buf), ws.nbytes,
                        c_void_p(s))
    _check(rc, "orthrus_step")


def step_noalloc(emb: DeviceModel, gen: DeviceModel, batch, emb_kv: DeviceKV, gen_kv: DeviceKV,
                 acc_sum: torch.Tensor, acc_w: torch.Tensor, out_logits: Optional[torch.Tensor],
                 out_emb: Optional[torch.Tensor], device_error: Optional[torch.Tensor] = None,
                 stream: Optional[int] = None) -> int:
    """Enqueue one orthrus_step_noalloc (library-owned scratch instead of a workspace); returns
    the status code (0 or a negative ORTHRUS_E* value) without raising.  ``device_error``: int32
    [1] device tensor that receives the step's device error bits."""
    pb = PackedBatch(batch)
    ekv, gkv = emb_kv.struct(), (emb_kv.struct() if gen_kv is emb_kv else gen_kv.struct())
    s = current_stream() if stream is None else stream
    return A.orthrus_step_noalloc(emb.handle, gen.handle, byref(pb.c), byref(ekv), byref(gkv), _vp(acc_sum),
                                  _vp(acc_w), _vp(out_logits), _vp(out_emb), _vp(device_error), c_void_p(s))


def sample_greedy(logits: torch.Tensor, out_tokens: torch.Tensor,
                  stream: Optional[int] = None) -> None:
    """Enqueue orthrus_sample_greedy on fp32 logits [rows][vocab] into int32 out_tokens [rows]."""
    if logits.dtype != torch.float32 or out_tokens.dtype != torch.int32:
        raise A.OrthrusError(A.ORTHRUS_EINVAL, "sample_greedy dtypes")
    if not logits.is_contiguous() or logits.dim() != 2 or out_tokens.shape != (logits.shape[0],):
        raise A.OrthrusError(A.ORTHRUS_EINVAL, "sample_greedy shapes")
    s = current_stream() if stream is None else stream
    _check(A.orthrus_sample_greedy(_vp(logits), logits.shape[0], logits.shape[1], _vp(out_tokens),
                                   c_void_p(s)), "orthrus_sample_greedy")


def plan(emb: DeviceModel, gen: DeviceModel, batch, emb_kv, gen_kv):
    """Host-side plan (no GPU work): returns (n_prefill, n_decode, items[n, 8])."""
    pb = PackedBatch(batch)
    ekv, gkv = emb_kv.struct(), gen_kv.struct()
    npre, ndec = c_int32(0), c_int32(0)
    _check(A.orthrus_plan(emb.handle, gen.handle, byref(pb.c), byref(ekv), byref(gkv), byref(npre),
                          byref(ndec), None, 0), "orthrus_plan")
    n = npre.value + ndec.value
    items = np.zeros((max(1, n), 8), np.int32)
    _check(A.orthrus_plan(emb.handle, gen.handle, byref(pb.c), byref(ekv), byref(gkv), byref(npre),
                          byref(ndec), items.ctypes.data_as(POINTER(c_int32)), n), "orthrus_plan")
    return npre.value, ndec.value, items[:n]


def profile_begin(model: DeviceModel) -> None:
    _check(A.orthrus_profile_begin(model.handle), "orthrus_profile_begin")


def profile_only(model: DeviceModel, name: str | None) -> None:
    """Time only the launches named `name` in later profiling windows (None: every launch)."""
    _check(A.orthrus_profile_only(model.handle, (name or "").encode()), "orthrus_profile_only")


def profile_end(model: DeviceModel):
    """{kernel name: (launches, total ms)} since profile_begin (synchronises the events)."""
    cap = 64
    out = (A.orthrus_kernel_time * cap)()
    n = c_int32(0)
    _check(A.orthrus_profile_end(model.handle, out, cap, byref(n)), "orthrus_profile_end")
    return {out[i].name.decode(): (out[i].launches, out[i].total_ms) for i in range(min(n.value, cap))}


class Scheduler:
    """The native intra-batch scheduler (include/orthrus_sched.h); marshalling only.

    ``caches`` holds (n_seq, n_pages, max_blocks) of the embedding (or shared) cache and, unless
    ``shared``, of the generator's cache."""

    def __init__(self, budget: int, chunk: int, caches, shared: bool = True,
                 atomic_embeddings: bool = False, decode_tokens: int = 1, page_size: int = 16,
                 eos: int = -1):
        c = A.orthrus_sched_config()
        c.budget, c.chunk, c.atomic_embeddings = budget, chunk, int(atomic_embeddings)
        c.decode_tokens, c.page_size, c.shared_cache, c.eos_token = decode_tokens, page_size, int(shared), eos
        for i, (n_seq, n_pages, max_blocks) in enumerate(caches[:1 if shared else 2]):
            c.n_seq[i], c.n_pages[i], c.max_blocks[i] = n_seq, n_pages, max_blocks
        self.cfg = c
        self.shared = shared
        h = c_void_p()
        _check(A.orthrus_sched_create(byref(c), byref(h)), "orthrus_sched_create")
        self.handle = h
        self._b = A.orthrus_sched_batch()

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            A.orthrus_sched_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def _ids(tokens, n):
        if tokens is None:
            return None, None
        a = np.ascontiguousarray(tokens, np.int32)
        if a.shape != (n,):
            raise A.OrthrusError(A.ORTHRUS_EINVAL, "token count")
        return a, c_void_p(a.ctypes.data)

    def submit_embedding(self, rid: int, n: int, tokens=None, pool: str = "mean",
                         weights=None, adapter: int = -1) -> None:
        a, p = self._ids(tokens, n)
        wp = None
        if weights is not None:
            w = np.ascontiguousarray(weights, np.float32)
            if w.shape != (n,):
                raise A.OrthrusError(A.ORTHRUS_EINVAL, "weight count")
            wp = c_void_p(w.ctypes.data)
        _check(A.orthrus_sched_submit_embedding(self.handle, rid, p, wp, n, POOL_CODES[pool], adapter),
               "orthrus_sched_submit_embedding")

    def submit_generation(self, rid: int, n: int, max_new: int, prompt=None) -> None:
        a, p = self._ids(prompt, n)
        _check(A.orthrus_sched_submit_generation(self.handle, rid, p, n, max_new),
               "orthrus_sched_submit_generation")

    def next(self) -> dict:
        """The next batch: items by request id (the fields of the scheduling reference model)
        plus the raw descriptor for orthrus_step."""
        b = self._b
        _check(A.orthrus_sched_next(self.handle, byref(b)), "orthrus_sched_next")
        bt = b.batch
        emb = [(b.chunk_ids[i], bt.chunks[i].offset, bt.chunks[i].len,
                bool(bt.chunks[i].flags & A.ORTHRUS_CHUNK_LAST)) for i in range(bt.n_chunks)]
        gen = [(b.gen_chunk_ids[i], bt.gen_chunks[i].offset, bt.gen_chunks[i].len,
                bool(bt.gen_chunks[i].flags & A.ORTHRUS_CHUNK_LAST)) for i in range(bt.n_gen_chunks)]
        dec = [(b.row_ids[j], bt.rows[j].ctx_len, b.row_tokens[j]) for j in range(bt.n_decode)]
        picks = ctypes.string_at(b.picks, b.n_picks).decode() if b.n_picks else ""
        n_tok = sum(c[2] for c in emb) + sum(c[2] for c in gen) + len(dec)
        adapters = ([bt.chunk_adapter[i] for i in range(bt.n_chunks)] if bt.chunk_adapter
                    else [-1] * bt.n_chunks)
        return {
            "emb_chunks": emb, "gen_chunks": gen, "decodes": dec, "order": list(picks),
            "emb_adapters": adapters,
            "used": b.tokens_used, "logit_ids": [b.logit_ids[i] for i in range(b.n_logit_rows)],
            "finished": [b.finishing_ids[i] for i in range(b.n_finishing)],
            "credits": (b.credit_e, b.credit_g),
            "slots": {"emb": [bt.chunks[i].seq for i in range(bt.n_chunks)],
                      "gen": [bt.gen_chunks[i].seq for i in range(bt.n_gen_chunks)],
                      "dec": [bt.rows[j].seq for j in range(bt.n_decode)]},
            "token_ids": np.ctypeslib.as_array(bt.token_ids, (n_tok,)).copy() if n_tok else
            np.zeros(0, np.int32),
            "table_rows": [(b.table_rows[2 * i], b.table_rows[2 * i + 1]) for i in range(b.n_table_rows)],
        }

    def commit(self, sampled=None):
        n_logit = self._b.n_logit_rows
        cap = self._b.n_finishing + n_logit
        fin = (ctypes.c_int64 * max(1, cap))()
        nf = c_int32(0)
        if sampled is None:
            rc = A.orthrus_sched_commit(self.handle, None, 0, byref(nf), fin, cap)
        else:
            a = np.ascontiguousarray(sampled, np.int32)
            rc = A.orthrus_sched_commit(self.handle, c_void_p(a.ctypes.data), a.size, byref(nf), fin, cap)
        _check(rc, "orthrus_sched_commit")
        return [fin[i] for i in range(nf.value)]

    def block_table(self, cache: int = 0) -> np.ndarray:
        p = A.orthrus_sched_block_table(self.handle, cache)
        if not p:
            raise A.OrthrusError(A.ORTHRUS_EINVAL, "orthrus_sched_block_table")
        i = 0 if self.shared else cache
        shape = (self.cfg.n_seq[i], self.cfg.max_blocks[i])
        return np.ctypeslib.as_array(p, shape).copy()

    def counts(self) -> dict:
        c = (ctypes.c_int64 * 7)()
        _check(A.orthrus_sched_counts(self.handle, c), "orthrus_sched_counts")
        keys = ("queued_emb", "queued_gen", "running", "free_slots0", "free_pages0", "free_slots1",
                "free_pages1")
        return dict(zip(keys, list(c)))


class Runner:
    """One GPU's iteration loop (orthrus_runner_*): device buffers in torch tensors, sized for the
    scheduler's budget."""

    def __init__(self, emb: DeviceModel, gen: DeviceModel, emb_kv: DeviceKV, gen_kv: DeviceKV,
                 sched: Scheduler, device="cuda"):
        B = sched.cfg.budget
        d, V = emb.cfg.d_model, gen.cfg.vocab
        n_seq0 = sched.cfg.n_seq[0]
        self.acc_sum = torch.zeros((n_seq0, d), dtype=torch.float32, device=device)
        self.acc_w = torch.zeros(n_seq0, dtype=torch.float32, device=device)
        self.logits = torch.zeros((B, V), dtype=torch.float32, device=device)
        self.out_emb = torch.zeros((B, d), dtype=torch.float32, device=device)
        self.tokens = torch.zeros(B, dtype=torch.int32, device=device)
        max_ctx = max(sched.cfg.max_blocks[i] for i in range(1 if sched.shared else 2)) * sched.cfg.page_size
        self.ws = Workspace(emb, gen, B, B, B, max_ctx, device=device)
        self._keep = (emb, gen, emb_kv, gen_kv, sched)
        self._ekv, self._gkv = emb_kv.struct(), (emb_kv.struct() if gen_kv is emb_kv else gen_kv.struct())
        buf = A.orthrus_runner_buffers(_vp(self.acc_sum), _vp(self.acc_w), _vp(self.logits),
                                       _vp(self.out_emb), _vp(self.tokens), _vp(self.ws.buf),
                                       self.ws.nbytes)
        self._buf = buf
        h = c_void_p()
        _check(A.orthrus_runner_create(emb.handle, gen.handle, byref(self._ekv), byref(self._gkv),
                                       sched.handle, byref(buf), byref(h)), "orthrus_runner_create")
        self.handle = h
        self.d = d
        self._out = A.orthrus_runner_output()

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            A.orthrus_runner_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def iterate(self, stream: Optional[int] = None) -> dict:
        """Run one loop iteration; returns the sampled tokens and finished embeddings by request."""
        o = self._out
        s = current_stream() if stream is None else stream
        _check(A.orthrus_runner_iterate(self.handle, c_void_p(s), byref(o)), "orthrus_runner_iterate")
        toks = {o.token_ids[i]: o.tokens[i] for i in range(o.n_tokens)}
        embs = {}
        if o.n_embeddings:
            e = np.ctypeslib.as_array(o.embeddings, (o.n_embeddings, self.d))
            embs = {o.embedding_ids[i]: e[i].copy() for i in range(o.n_embeddings)}
        return {"tokens": toks, "embeddings": embs,
                "finished": [o.finished_ids[i] for i in range(o.n_finished)],
                "used": o.tokens_used, "n_items": o.n_items}
