"""ctypes mirror of include/orthrus.h and include/orthrus_sched.h: the structs and the entry
points, same names.

Argument marshalling only.  Loading fails loudly if liborthrus.so has not been built;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, Structure, c_char_p, c_float, c_int, c_int32, c_int64, c_size_t,
                    c_void_p)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liborthrus.so")

ORTHRUS_OK = 0
ORTHRUS_EINVAL = -1
ORTHRUS_EDESC = -2
ORTHRUS_EDUPSEQ = -3
ORTHRUS_ECAPACITY = -4
ORTHRUS_EUNSUPPORTED = -5
ORTHRUS_EHIP = -6
ORTHRUS_EDEVICE = -7
ORTHRUS_SCRATCH_BYTES = 64 << 20
ORTHRUS_F32 = 0
ORTHRUS_BF16 = 1
ORTHRUS_CHUNK_LAST = 1
ORTHRUS_POOL_SHIFT = 1
ORTHRUS_POOL_MEAN = 0
ORTHRUS_POOL_LAST = 1
ORTHRUS_POOL_CLS = 2
ORTHRUS_POOL_NONE = 3
ORTHRUS_POOL_WMEAN = 4
ORTHRUS_POOL_BUFFER = 5
ORTHRUS_POOL_MASK = 7
ORTHRUS_MAX_STEP_ADAPTERS = 4
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
                ("layers", POINTER(orthrus_layer_weights)), ("lm_head_blocked", c_void_p)]


class orthrus_lora_layer(Structure):
    _fields_ = [("qkv_a", c_void_p), ("qkv_b", c_void_p), ("o_a", c_void_p), ("o_b", c_void_p),
                ("gate_up_a", c_void_p), ("gate_b", c_void_p), ("up_b", c_void_p),
                ("down_a", c_void_p), ("down_b", c_void_p)]


class orthrus_lora(Structure):
    _fields_ = [("rank", c_int32 * 4), ("scale", c_float), ("layers", POINTER(orthrus_lora_layer))]


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
                ("gen_chunks", POINTER(orthrus_gen_chunk)), ("token_weights", POINTER(c_float)),
                ("hidden", c_void_p), ("hidden_stride", c_int32),
                ("chunk_adapter", POINTER(c_int32))]


class orthrus_kv(Structure):
    _fields_ = [("k_cache", c_void_p), ("v_cache", c_void_p), ("block_table", c_void_p),
                ("n_pages", c_int32), ("n_seq", c_int32), ("max_blocks", c_int32)]


class orthrus_kernel_time(Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", c_int32), ("total_ms", ctypes.c_double)]


class orthrus_sched_config(Structure):
    _fields_ = [("budget", c_int32), ("chunk", c_int32), ("atomic_embeddings", c_int32),
                ("decode_tokens", c_int32), ("page_size", c_int32), ("shared_cache", c_int32),
                ("eos_token", c_int32), ("n_seq", c_int32 * 2), ("n_pages", c_int32 * 2),
                ("max_blocks", c_int32 * 2)]


class orthrus_sched_batch(Structure):
    _fields_ = [("batch", orthrus_batch), ("chunk_ids", POINTER(c_int64)),
                ("gen_chunk_ids", POINTER(c_int64)), ("row_ids", POINTER(c_int64)),
                ("row_tokens", POINTER(c_int32)), ("n_logit_rows", c_int32),
                ("logit_ids", POINTER(c_int64)), ("tokens_used", c_int32), ("n_picks", c_int32),
                ("picks", c_void_p), ("n_finishing", c_int32), ("finishing_ids", POINTER(c_int64)),
                ("n_table_rows", c_int32), ("table_rows", POINTER(c_int32)), ("credit_e", c_int64),
                ("credit_g", c_int64)]


class orthrus_runner_buffers(Structure):
    _fields_ = [("acc_sum", c_void_p), ("acc_w", c_void_p), ("logits", c_void_p),
                ("out_emb", c_void_p), ("tokens", c_void_p), ("workspace", c_void_p),
                ("ws_bytes", c_size_t)]


class orthrus_runner_output(Structure):
    _fields_ = [("n_tokens", c_int32), ("token_ids", POINTER(c_int64)), ("tokens", POINTER(c_int32)),
                ("n_embeddings", c_int32), ("embedding_ids", POINTER(c_int64)),
                ("embeddings", POINTER(c_float)), ("n_finished", c_int32),
                ("finished_ids", POINTER(c_int64)), ("tokens_used", c_int32), ("n_items", c_int32)]


# name -> (restype, argtypes); every symbol include/orthrus.h and include/orthrus_sched.h declare
SIGNATURES = {
    "orthrus_model_create": (c_int, [POINTER(orthrus_config), POINTER(orthrus_weights),
                                     POINTER(c_void_p)]),
    "orthrus_model_destroy": (None, [c_void_p]),
    "orthrus_model_set_adapters": (c_int, [c_void_p, POINTER(orthrus_lora), c_int32]),
    "orthrus_workspace_bytes": (c_size_t, [c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                           c_int32]),
    "orthrus_blocked_bytes": (c_size_t, [c_int32, c_int32]),
    "orthrus_block_weights": (c_int, [c_void_p, c_void_p, c_int32, c_int32, c_void_p]),
    "orthrus_step": (c_int, [c_void_p, c_void_p, POINTER(orthrus_batch), POINTER(orthrus_kv),
                             POINTER(orthrus_kv), c_void_p, c_void_p, c_void_p, c_void_p,
                             c_void_p, c_size_t, c_void_p]),
    "orthrus_sample_greedy": (c_int, [c_void_p, c_int32, c_int32, c_void_p, c_void_p]),
    "orthrus_workspace_init": (c_int, [c_void_p, c_void_p]),
    "orthrus_step_noalloc": (c_int, [c_void_p, c_void_p, POINTER(orthrus_batch), POINTER(orthrus_kv),
                                     POINTER(orthrus_kv), c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p]),
    "orthrus_device_error": (c_int, [c_void_p, c_void_p, POINTER(c_int32)]),
    "orthrus_plan": (c_int, [c_void_p, c_void_p, POINTER(orthrus_batch), POINTER(orthrus_kv),
                             POINTER(orthrus_kv), POINTER(c_int32), POINTER(c_int32),
                             POINTER(c_int32), c_int32]),
    "orthrus_profile_begin": (c_int, [c_void_p]),
    "orthrus_profile_only": (c_int, [c_void_p, c_char_p]),
    "orthrus_profile_end": (c_int, [c_void_p, POINTER(orthrus_kernel_time), c_int32,
                                    POINTER(c_int32)]),
    "orthrus_strerror": (c_char_p, [c_int]),
    "orthrus_sched_create": (c_int, [POINTER(orthrus_sched_config), POINTER(c_void_p)]),
    "orthrus_sched_destroy": (None, [c_void_p]),
    "orthrus_sched_submit_embedding": (c_int, [c_void_p, c_int64, c_void_p, c_void_p, c_int32, c_int32,
                                               c_int32]),
    "orthrus_sched_submit_generation": (c_int, [c_void_p, c_int64, c_void_p, c_int32, c_int32]),
    "orthrus_sched_next": (c_int, [c_void_p, POINTER(orthrus_sched_batch)]),
    "orthrus_sched_commit": (c_int, [c_void_p, c_void_p, c_int32, POINTER(c_int32),
                                     POINTER(c_int64), c_int32]),
    "orthrus_sched_block_table": (POINTER(c_int32), [c_void_p, c_int32]),
    "orthrus_sched_get_config": (c_int, [c_void_p, POINTER(orthrus_sched_config)]),
    "orthrus_sched_counts": (c_int, [c_void_p, POINTER(c_int64)]),
    "orthrus_runner_create": (c_int, [c_void_p, c_void_p, POINTER(orthrus_kv), POINTER(orthrus_kv),
                                      c_void_p, POINTER(orthrus_runner_buffers), POINTER(c_void_p)]),
    "orthrus_runner_destroy": (None, [c_void_p]),
    "orthrus_runner_iterate": (c_int, [c_void_p, c_void_p, POINTER(orthrus_runner_output)]),
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


def orthrus_model_set_adapters(model, adapters, n):
    return load().orthrus_model_set_adapters(model, adapters, n)


def orthrus_workspace_bytes(emb, gen, max_tokens, max_chunks, max_decode, max_ctx):
    return load().orthrus_workspace_bytes(emb, gen, max_tokens, max_chunks, max_decode, max_ctx)


def orthrus_blocked_bytes(rows, cols):
    return load().orthrus_blocked_bytes(rows, cols)


def orthrus_block_weights(src, dst, rows, cols, stream):
    return load().orthrus_block_weights(src, dst, rows, cols, stream)


def orthrus_step(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits, out_emb, workspace,
                 ws_bytes, stream):
    return load().orthrus_step(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits,
                               out_emb, workspace, ws_bytes, stream)


def orthrus_sample_greedy(logits, rows, vocab, out_tokens, stream):
    return load().orthrus_sample_greedy(logits, rows, vocab, out_tokens, stream)


def orthrus_workspace_init(workspace, stream):
    return load().orthrus_workspace_init(workspace, stream)


def orthrus_step_noalloc(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits, out_emb,
                         device_error, stream):
    return load().orthrus_step_noalloc(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits,
                                       out_emb, device_error, stream)


def orthrus_device_error(workspace, stream, bits):
    return load().orthrus_device_error(workspace, stream, bits)


def orthrus_plan(emb, gen, batch, emb_kv, gen_kv, n_prefill, n_decode, items, cap):
    return load().orthrus_plan(emb, gen, batch, emb_kv, gen_kv, n_prefill, n_decode, items, cap)


def orthrus_profile_begin(model):
    return load().orthrus_profile_begin(model)


def orthrus_profile_only(model, name):
    return load().orthrus_profile_only(model, name)


def orthrus_profile_end(model, out, cap, n_out):
    return load().orthrus_profile_end(model, out, cap, n_out)


def orthrus_strerror(code):
    return load().orthrus_strerror(code).decode()


def orthrus_sched_create(cfg, out):
    return load().orthrus_sched_create(cfg, out)


def orthrus_sched_destroy(s):
    load().orthrus_sched_destroy(s)


def orthrus_sched_submit_embedding(s, rid, tokens, weights, n, pool, adapter):
    return load().orthrus_sched_submit_embedding(s, rid, tokens, weights, n, pool, adapter)


def orthrus_sched_submit_generation(s, rid, prompt, n, max_new):
    return load().orthrus_sched_submit_generation(s, rid, prompt, n, max_new)


def orthrus_sched_next(s, out):
    return load().orthrus_sched_next(s, out)


def orthrus_sched_commit(s, sampled, n, n_finished, finished, cap):
    return load().orthrus_sched_commit(s, sampled, n, n_finished, finished, cap)


def orthrus_sched_block_table(s, cache):
    return load().orthrus_sched_block_table(s, cache)


def orthrus_sched_get_config(s, out):
    return load().orthrus_sched_get_config(s, out)


def orthrus_sched_counts(s, counts7):
    return load().orthrus_sched_counts(s, counts7)


def orthrus_runner_create(emb, gen, emb_kv, gen_kv, sched, buf, out):
    return load().orthrus_runner_create(emb, gen, emb_kv, gen_kv, sched, buf, out)


def orthrus_runner_destroy(r):
    load().orthrus_runner_destroy(r)


def orthrus_runner_iterate(r, stream, out):
    return load().orthrus_runner_iterate(r, stream, out)
