"""ctypes mirror of include/orthrus.h: the structs and the entry points, same names.

Argument marshalling only.  Loading fails loudly if liborthrus.so has not been built;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, c_float, c_int, c_int32, c_size_t, c_void_p, c_char_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liborthrus.so")

ORTHRUS_OK = 0
ORTHRUS_EINVAL = -1
ORTHRUS_EDESC = -2
ORTHRUS_EDUPSEQ = -3
ORTHRUS_ECAPACITY = -4
ORTHRUS_EUNSUPPORTED = -5
ORTHRUS_EHIP = -6
ORTHRUS_EDEVICE = -7
ORTHRUS_F32 = 0
ORTHRUS_BF16 = 1
ORTHRUS_CHUNK_LAST = 1
ORTHRUS_POOL_SHIFT = 1
ORTHRUS_POOL_MEAN = 0
ORTHRUS_POOL_LAST = 1
ORTHRUS_POOL_CLS = 2
ORTHRUS_POOL_NONE = 3
ORTHRUS_DEVERR_PAGE = 1
ORTHRUS_DEVERR_ACC = 2


class orthrus_config(Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("d_ff", c_int32),
                ("vocab", c_int32), ("page_size", c_int32), ("rope_base", c_float),
                ("rms_eps", c_float), ("dtype", c_int32)]


class orthrus_layer_weights(Structure):
    _fields_ = [("attn_norm", c_void_p), ("w_qkv", c_void_p), ("w_o", c_void_p),
                ("mlp_norm", c_void_p), ("w_gate", c_void_p), ("w_up", c_void_p),
                ("w_down", c_void_p)]


class orthrus_weights(Structure):
    _fields_ = [("tok_emb", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("layers", POINTER(orthrus_layer_weights))]


class orthrus_emb_chunk(Structure):
    _fields_ = [("seq", c_int32), ("offset", c_int32), ("len", c_int32), ("flags", c_int32)]


class orthrus_decode_row(Structure):
    _fields_ = [("seq", c_int32), ("ctx_len", c_int32)]


class orthrus_gen_chunk(Structure):
    _fields_ = [("seq", c_int32), ("offset", c_int32), ("len", c_int32), ("flags", c_int32)]


class orthrus_batch(Structure):
    _fields_ = [("n_chunks", c_int32), ("n_decode", c_int32),
                ("chunks", POINTER(orthrus_emb_chunk)), ("rows", POINTER(orthrus_decode_row)),
                ("token_ids", POINTER(c_int32)), ("n_gen_chunks", c_int32),
                ("gen_chunks", POINTER(orthrus_gen_chunk))]


class orthrus_kv(Structure):
    _fields_ = [("k_cache", c_void_p), ("v_cache", c_void_p), ("block_table", c_void_p),
                ("n_pages", c_int32), ("n_seq", c_int32), ("max_blocks", c_int32)]


class orthrus_kernel_time(Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", c_int32), ("total_ms", ctypes.c_double)]


# name -> (restype, argtypes); every symbol include/orthrus.h declares
SIGNATURES = {
    "orthrus_model_create": (c_int, [POINTER(orthrus_config), POINTER(orthrus_weights),
                                     POINTER(c_void_p)]),
    "orthrus_model_destroy": (None, [c_void_p]),
    "orthrus_workspace_bytes": (c_size_t, [c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                           c_int32]),
    "orthrus_step": (c_int, [c_void_p, c_void_p, POINTER(orthrus_batch), POINTER(orthrus_kv),
                             POINTER(orthrus_kv), c_void_p, c_void_p, c_void_p, c_void_p,
                             c_void_p, c_size_t, c_void_p]),
    "orthrus_sample_greedy": (c_int, [c_void_p, c_int32, c_int32, c_void_p, c_void_p]),
    "orthrus_workspace_init": (c_int, [c_void_p, c_void_p]),
    "orthrus_device_error": (c_int, [c_void_p, c_void_p, POINTER(c_int32)]),
    "orthrus_plan": (c_int, [c_void_p, c_void_p, POINTER(orthrus_batch), POINTER(orthrus_kv),
                             POINTER(orthrus_kv), POINTER(c_int32), POINTER(c_int32),
                             POINTER(c_int32), c_int32]),
    "orthrus_profile_begin": (c_int, [c_void_p]),
    "orthrus_profile_end": (c_int, [c_void_p, POINTER(orthrus_kernel_time), c_int32,
                                    POINTER(c_int32)]),
    "orthrus_strerror": (c_char_p, [c_int]),
}

_lib = None


class OrthrusError(RuntimeError):
    def __init__(self, code: int, where: str = ""):
        self.code = code
        super().__init__(f"{where}: {orthrus_strerror(code)} ({code})")


def load():
    """Load liborthrus.so (raises if it is missing: the native library is the only path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_25405_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def orthrus_model_create(cfg, weights, out):
    return load().orthrus_model_create(cfg, weights, out)


def orthrus_model_destroy(model):
    load().orthrus_model_destroy(model)


def orthrus_workspace_bytes(emb, gen, max_tokens, max_chunks, max_decode, max_ctx):
    return load().orthrus_workspace_bytes(emb, gen, max_tokens, max_chunks, max_decode, max_ctx)


def orthrus_step(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits, out_emb, workspace,
                 ws_bytes, stream):
    return load().orthrus_step(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits,
                               out_emb, workspace, ws_bytes, stream)


def orthrus_sample_greedy(logits, rows, vocab, out_tokens, stream):
    return load().orthrus_sample_greedy(logits, rows, vocab, out_tokens, stream)


def orthrus_workspace_init(workspace, stream):
    return load().orthrus_workspace_init(workspace, stream)


def orthrus_device_error(workspace, stream, bits):
    return load().orthrus_device_error(workspace, stream, bits)


def orthrus_plan(emb, gen, batch, emb_kv, gen_kv, n_prefill, n_decode, items, cap):
    return load().orthrus_plan(emb, gen, batch, emb_kv, gen_kv, n_prefill, n_decode, items, cap)


def orthrus_profile_begin(model):
    return load().orthrus_profile_begin(model)


def orthrus_profile_end(model, out, cap, n_out):
    return load().orthrus_profile_end(model, out, cap, n_out)


def orthrus_strerror(code):
    return load().orthrus_strerror(code).decode()
