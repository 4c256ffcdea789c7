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
              "cls": A.ORTHRUS_POOL_CLS, "none": A.ORTHRUS_POOL_NONE}


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
    """Weights uploaded to the GPU in the model dtype (norm gains fp32) plus the library handle."""

    def __init__(self, cfg, weights, device="cuda"):
        self.cfg = cfg
        dt = torch_dtype(cfg)

        def up(a, dtype=dt):
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
        self._w = A.orthrus_weights(_vp(self.tok_emb), _vp(self.final_norm), _vp(self.lm_head),
                                    ctypes.cast(self._lw, POINTER(A.orthrus_layer_weights)))
        self._cfg = abi_config(cfg)
        h = c_void_p()
        _check(A.orthrus_model_create(byref(self._cfg), byref(self._w), byref(h)),
               "orthrus_model_create")
        self.handle = h

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
        self.c = A.orthrus_batch(nc, nd, ctypes.cast(self._chunks, POINTER(A.orthrus_emb_chunk)),
                                 ctypes.cast(self._rows, POINTER(A.orthrus_decode_row)),
                                 self._ids.ctypes.data_as(POINTER(c_int32)), ng,
                                 ctypes.cast(self._gen, POINTER(A.orthrus_gen_chunk)))


def step(emb: DeviceModel, gen: DeviceModel, batch, emb_kv: DeviceKV, gen_kv: DeviceKV,
         acc_sum: torch.Tensor, acc_w: torch.Tensor, out_logits: Optional[torch.Tensor],
         out_emb: Optional[torch.Tensor], ws: Workspace, stream: Optional[int] = None,
         packed: Optional[PackedBatch] = None) -> None:
    """Enqueue one orthrus_step on `stream` (default: torch's current stream); raises on error."""
    pb = packed if packed is not None else PackedBatch(batch)
    ekv, gkv = emb_kv.struct(), (emb_kv.struct() if gen_kv is emb_kv else gen_kv.struct())
    s = current_stream() if stream is None else stream
    rc = A.orthrus_step(emb.handle, gen.handle, byref(pb.c), byref(ekv), byref(gkv), _vp(acc_sum),
                        _vp(acc_w), _vp(out_logits), _vp(out_emb), _vp(ws.buf), ws.nbytes,
                        c_void_p(s))
    _check(rc, "orthrus_step")


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


def profile_end(model: DeviceModel):
    """{kernel name: (launches, total ms)} since profile_begin (synchronises the events)."""
    cap = 64
    out = (A.orthrus_kernel_time * cap)()
    n = c_int32(0)
    _check(A.orthrus_profile_end(model.handle, out, cap, byref(n)), "orthrus_profile_end")
    return {out[i].name.decode(): (out[i].launches, out[i].total_ms) for i in range(min(n.value, cap))}
