"""The C-ABI library on the CPU: symbols, host-side validation and the attention work plan.

No GPU work happens here: every call below either only reads host memory (orthrus_plan,
model handles) or is rejected by host validation before anything is enqueued.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2609_25405_amd as P
from paper_2609_25405_amd import _abi as A
from paper_2609_25405_amd import runtime as R
from workload import (Batch, DecodeRow, EmbChunk, GenChunk, ModelConfig, PagedKV, draw_tokens,
                      make_weights, tiny_config, llm7b_config)
from oracle import OracleKV, StepError, step_oracle

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include")
HEADERS = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))


def header_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(orthrus_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    lib = P.load()
    names = header_functions()
    assert [os.path.basename(h) for h in HEADERS] == ["orthrus.h", "orthrus_sched.h"]
    assert len(names) == 16 + 12
    for n in names:
        assert hasattr(lib, n), n
        assert n in A.SIGNATURES, n
    assert set(A.SIGNATURES) == set(names)
    assert P.orthrus_strerror(A.ORTHRUS_EDUPSEQ).startswith("sequence")


def test_struct_layouts_match_header():
    # sizes follow the header's field lists (int32/float fields, 8-byte pointers)
    assert ctypes.sizeof(A.orthrus_config) == 11 * 4
    assert ctypes.sizeof(A.orthrus_emb_chunk) == 16
    assert ctypes.sizeof(A.orthrus_decode_row) == 8
    assert ctypes.sizeof(A.orthrus_kv) == 3 * 8 + 3 * 4 + 4
    assert ctypes.sizeof(A.orthrus_gen_chunk) == 16
    # n_chunks, n_decode, 3 pointers, n_gen_chunks (+4 bytes of padding), 3 pointers,
    # hidden_stride (+4 bytes of padding), 1 pointer
    assert ctypes.sizeof(A.orthrus_batch) == 8 + 3 * 8 + 8 + 3 * 8 + 8 + 8
    assert A.orthrus_batch.gen_chunks.offset == 40


STRUCTS = ["orthrus_config", "orthrus_layer_weights", "orthrus_weights", "orthrus_lora_layer",
           "orthrus_lora", "orthrus_emb_chunk",
           "orthrus_decode_row", "orthrus_gen_chunk", "orthrus_batch", "orthrus_kv",
           "orthrus_kernel_time", "orthrus_sched_config", "orthrus_sched_batch",
           "orthrus_runner_buffers", "orthrus_runner_output"]


def test_ctypes_mirror_matches_the_c_compiler(tmp_path):
    """Size and every field offset of each header struct, as a C compiler lays them out, equal
    the ctypes mirror's."""
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "orthrus_sched.h"', "int main(void) {"]
    for st in STRUCTS:
        lines.append(f'printf("{st} size %zu\\n", sizeof({st}));')
        for f, _ in getattr(A, st)._fields_:
            lines.append(f'printf("{st} {f} %zu\\n", offsetof({st}, {f}));')
    lines.append("return 0; }")
    src = tmp_path / "probe.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-std=c99", "-I", INCLUDE, str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in filter(None, out):
        st, f, v = line.split()
        want = ctypes.sizeof(getattr(A, st)) if f == "size" else getattr(getattr(A, st), f).offset
        assert int(v) == want, line


def test_model_create_validates_config():
    cfg = tiny_config()
    W = make_weights(cfg, 1)
    m = R.DeviceModel(cfg, W, device="cpu")
    assert m.handle.value
    m.close()
    for bad, code in ((dict(head_dim=32), A.ORTHRUS_EUNSUPPORTED),
                      (dict(n_kv_heads=3), A.ORTHRUS_EINVAL),
                      (dict(page_size=32), A.ORTHRUS_EUNSUPPORTED),
                      (dict(d_model=200), A.ORTHRUS_EUNSUPPORTED)):
        c = cfg.replace(**bad)
        with pytest.raises(A.OrthrusError) as e:
            R.DeviceModel(c, make_weights(c, 1) if "d_model" not in bad else W, device="cpu")
        assert e.value.code == code


def _cpu_setup(cfg=None, n_seq=6, n_pages=64, max_blocks=8):
    cfg = cfg or tiny_config()
    W = make_weights(cfg, 2)
    m = R.DeviceModel(cfg, W, device="cpu")
    pk = PagedKV(cfg, n_pages, n_seq, max_blocks, 3)
    for s in range(n_seq):
        pk.reserve(s, 40)
    kv = R.DeviceKV.from_paged(pk, device="cpu")
    return cfg, W, m, pk, kv


KIND_CODE = {"desc": A.ORTHRUS_EDESC, "dupseq": A.ORTHRUS_EDUPSEQ, "capacity": A.ORTHRUS_ECAPACITY}


def test_host_validation_matches_oracle_contract():
    cfg, W, m, pk, kv = _cpu_setup()
    ids = draw_tokens(1, 0, 12, cfg.vocab)
    bad = [
        Batch([EmbChunk(0, 0, 4, False), EmbChunk(0, 4, 4, False)], [], ids[:8]),
        Batch([EmbChunk(0, 0, 7, False)], [DecodeRow(0, 3)], ids[:8]),
        Batch([EmbChunk(6, 0, 8, False)], [], ids[:8]),
        Batch([EmbChunk(0, 0, 8, True, "none")], [], ids[:8]),
        Batch([EmbChunk(0, 0, 9, False)], [], ids[:8]),
        Batch([EmbChunk(0, 121, 8, False)], [], ids[:8]),
        Batch([], [DecodeRow(1, -1)], ids[:1]),
        Batch([], [DecodeRow(1, 128)], ids[:1]),
        Batch([EmbChunk(0, 0, 0, False)], [], ids[:0]),
        Batch([EmbChunk(0, -1, 4, False)], [], ids[:4]),
    ]
    big = ids[:8].copy()
    big[3] = cfg.vocab
    bad.append(Batch([EmbChunk(0, 0, 8, False)], [], big))
    # generation prefill chunks: same namespace as every item of the shared cache
    bad += [
        Batch([], [], ids[:4], [GenChunk(6, 0, 4, True)]),
        Batch([], [], ids[:4], [GenChunk(1, -1, 4, True)]),
        Batch([], [], ids[:0], [GenChunk(1, 0, 0, True)]),
        Batch([], [], ids[:4], [GenChunk(1, 126, 4, True)]),
        Batch([], [], ids[:8], [GenChunk(1, 0, 4, False), GenChunk(1, 4, 4, True)]),
        Batch([EmbChunk(1, 0, 4, False)], [], ids[:8], [GenChunk(1, 0, 4, True)]),
        Batch([], [DecodeRow(2, 3)], ids[:5], [GenChunk(2, 0, 4, False)]),
    ]
    big2 = ids[:6].copy()
    big2[5] = cfg.vocab
    bad.append(Batch([EmbChunk(0, 0, 2, False)], [], big2, [GenChunk(1, 0, 4, True)]))
    # weighted-mean and buffered heads
    neg = np.ones(8, np.float32)
    neg[3] = -0.5
    nan = np.ones(8, np.float32)
    nan[6] = np.nan
    bad += [
        Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids[:8]),
        Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids[:8], token_weights=neg),
        Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids[:8], token_weights=nan),
        Batch([EmbChunk(0, 0, 8, True, "wmean")], [], ids[:8], token_weights=neg[:7]),
        Batch([EmbChunk(0, 0, 8, True, "buffer")], [], ids[:8], hidden_stride=7),
        Batch([EmbChunk(0, 4, 8, True, "buffer")], [], ids[:8], hidden_stride=11),
    ]
    okv = OracleKV.from_paged(pk)
    t = R.torch
    acc, accw = t.zeros((6, cfg.d_model)), t.zeros(6)
    logits, emb = t.zeros((4, cfg.vocab)), t.zeros((4, cfg.d_model))
    ws = type("WS", (), {"buf": t.zeros(64, dtype=t.uint8), "nbytes": 64})()
    for b in bad:
        with pytest.raises(StepError) as e:
            step_oracle((cfg, W), (cfg, W), b, okv, okv, np.zeros((6, cfg.d_model)), np.zeros(6))
        want = KIND_CODE[e.value.kind]
        # descriptor checks run before the (too small) workspace is looked at
        with pytest.raises(A.OrthrusError) as g:
            R.step(m, m, b, kv, kv, acc, accw, logits, emb, ws)
        assert g.value.code == want, (b, e.value.kind, g.value.code)
        with pytest.raises(A.OrthrusError) as p:
            R.plan(m, m, b, kv, kv)
        assert p.value.code == want


def test_undersized_workspace_is_rejected_before_launch():
    cfg, W, m, pk, kv = _cpu_setup()
    ids = draw_tokens(1, 0, 8, cfg.vocab)
    b = Batch([EmbChunk(0, 0, 8, False)], [], ids)
    t = R.torch
    acc = t.zeros((6, cfg.d_model))
    accw = t.zeros(6)
    out = t.zeros((1, cfg.d_model))
    ws = type("WS", (), {"buf": t.zeros(256, dtype=t.uint8), "nbytes": 256})()
    with pytest.raises(A.OrthrusError) as e:
        R.step(m, m, b, kv, kv, acc, accw, None, out, ws)
    assert e.value.code == A.ORTHRUS_ECAPACITY


def _check_coverage(batch, cfg, npre, ndec, items):
    """Every (chunk token, kv head) in exactly one prefill tile, whose keys up to the causal bound
    are covered once (whole, or in key pieces cut on 64-key boundaries at or before the tile's
    first query, each with its own block of partial slots), and every (decode row, kv head, key)
    in exactly one decode split."""
    P_ = cfg.page_size
    group = cfg.n_q_heads // cfg.n_kv_heads
    qrows = 128 // group
    seen_q = {}
    pieces = {}
    work = []
    piece_slots = []
    allc = list(batch.chunks) + list(getattr(batch, "gen_chunks", None) or [])
    for it in items[:npre]:
        kind, ci, g, qb, qn, kb, ke, ps = it
        assert kind == 0
        c = allc[ci]
        assert 1 <= qn <= qrows and qb + qn <= c.len
        pieces.setdefault((ci, g, qb, qn), []).append((kb, ke, ps))
        work.append((ke - kb) * qn)
    for (ci, g, qb, qn), ps_ in pieces.items():
        c = allc[ci]
        ps_.sort()
        assert ps_[0][0] == 0 and ps_[-1][1] == c.offset + qb + qn
        if len(ps_) == 1:
            assert ps_[0][2] == -1
        else:
            assert 2 <= len(ps_) <= 8 and cfg.dtype == "bf16"
            for (kb, ke, ps), nxt in zip(ps_, ps_[1:] + [None]):
                assert kb % 64 == 0 and ps >= 0
                if nxt is not None:
                    assert ke == nxt[0] and ke <= c.offset + qb      # every row sees the piece
            base = ps_[0][2]
            assert [x[2] for x in ps_] == [base + k * qrows for k in range(len(ps_))]
            piece_slots += [(base + k * qrows, qrows) for k in range(len(ps_))]
        for r in range(qb, qb + qn):
            key = (ci, g, r)
            assert key not in seen_q
            seen_q[key] = True
    assert len(seen_q) == sum(c.len for c in allc) * cfg.n_kv_heads
    assert work == sorted(work, reverse=True)  # heaviest first
    seen_k = {}
    slots = set()
    # decode splits: whole 256-key chunks (the last one cut at the row's end), up to four
    # chunks per split on the bf16 path and one on the fp32 path, longest first
    max_split = 1024 if cfg.dtype == "bf16" else 256
    lengths = []
    for it in items[npre:npre + ndec]:
        kind, j, g, s, ns, kb, ke, ps = it
        assert kind == 1
        r = batch.rows[j]
        assert 0 <= s < ns and kb % 256 == 0 and kb < ke <= r.ctx_len + 1
        assert ke == r.ctx_len + 1 or ke % 256 == 0
        assert ke - kb <= max_split
        lengths.append(ke - kb)
        for k in range(kb, ke):
            assert (j, g, k) not in seen_k
            seen_k[(j, g, k)] = True
        if ns == 1:
            assert ps == -1
        else:
            assert ps not in slots
            slots.add(ps)
    assert len(seen_k) == sum(r.ctx_len + 1 for r in batch.rows) * cfg.n_kv_heads
    assert lengths == sorted(lengths, reverse=True)
    if slots:
        assert slots == set(range(len(slots)))
    # prefill pieces: disjoint blocks of qrows slots after the decode rows' slots
    taken = set(slots)
    for base, n in piece_slots:
        block = set(range(base, base + n))
        assert min(block) >= len(slots) and not (block & taken)
        taken |= block
    return len(piece_slots)


@pytest.mark.parametrize("cfgname", ["tiny", "7b", "7b-long-prefix", "7b-three-long"])
def test_plan_covers_every_key_exactly_once(cfgname):
    rng = np.random.default_rng(0)
    if cfgname == "tiny":
        cfg = tiny_config()
        chunks = [EmbChunk(0, 0, 128, False), EmbChunk(1, 256, 44, True)]
        rows = [DecodeRow(2, 0), DecodeRow(3, 255), DecodeRow(4, 256), DecodeRow(5, 1000)]
    elif cfgname == "7b":
        cfg = llm7b_config(n_layers=1)
        chunks = [EmbChunk(0, 0, 512, False, "last"), EmbChunk(1, 1536, 512, True, "last")]
        rows = [DecodeRow(2 + i, int(c)) for i, c in enumerate(rng.integers(1024, 4097, 64))]
    elif cfgname == "7b-long-prefix":
        # one chunk at the end of an 8192-token document: 128 tiles of ~8000 keys, each cut in 4
        cfg = llm7b_config(n_layers=1)
        chunks = [EmbChunk(0, 7680, 512, True, "mean")]
        rows = [DecodeRow(2 + i, 2100) for i in range(32)]
    else:
        # three chunks at 4096: 384 tiles of at most 4608 keys, under twice the mean keys per
        # workgroup slot (the launch is bound by its total work): no cuts
        cfg = llm7b_config(n_layers=1)
        chunks = [EmbChunk(i, 4096, 512, False, "mean") for i in range(3)]
        rows = [DecodeRow(3 + i, 2100) for i in range(32)]
    n_seq = 1 + max([c.seq for c in chunks] + [r.seq for r in rows])
    # planning reads no weight memory: tiny stand-in tensors carry the shapes' pointers
    small = cfg.replace(n_layers=0, vocab=64) if cfgname == "7b" else cfg
    W = make_weights(small, 0)
    m = R.DeviceModel(small.replace(vocab=cfg.vocab) if cfgname == "7b" else small, W, device="cpu")
    kv = type("KV", (), {})()
    kv.struct = lambda: A.orthrus_kv(1, 1, 1, 100000, n_seq, 600)
    ids = np.zeros(sum(c.len for c in chunks) + len(rows), np.int32)
    b = Batch(chunks, rows, ids)
    npre, ndec, items = R.plan(m, m, b, kv, kv)
    n_pieces = _check_coverage(b, cfg if cfgname == "tiny" else small, npre, ndec, items)
    # cuts only on the bf16 path, for tiles over twice the mean keys per slot, into pieces of
    # about that mean and at least 2048 keys
    assert n_pieces == {"tiny": 0, "7b": 0, "7b-long-prefix": 128 * 4, "7b-three-long": 0}[cfgname]


def _random_plan(seed):
    """Plan of a random batch checked by _check_coverage; returns the number of key pieces."""
    rng = np.random.default_rng(seed)
    if seed % 2 == 0:
        cfg = llm7b_config(n_layers=1)
        small = cfg.replace(n_layers=0, vocab=64)
    else:
        cfg = ModelConfig(n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=4, head_dim=64, d_ff=512,
                          vocab=64, dtype="bf16")
        small = cfg
    W = make_weights(small, 0)
    m = R.DeviceModel(small, W, device="cpu")
    seqs = iter(range(1000))
    def offset():
        return int(rng.choice([0, rng.integers(1, 600), rng.integers(2000, 12000)]))
    chunks = [EmbChunk(next(seqs), offset(), int(rng.integers(1, 600)), bool(rng.integers(0, 2)), "mean")
              for _ in range(int(rng.integers(0, 5)))]
    gen = [GenChunk(next(seqs), offset(), int(rng.integers(1, 300)), bool(rng.integers(0, 2)))
           for _ in range(int(rng.integers(0, 3)))]
    rows = [DecodeRow(next(seqs), int(rng.integers(0, 9000))) for _ in range(int(rng.integers(0, 40)))]
    if not (chunks or gen or rows):
        rows = [DecodeRow(next(seqs), 5)]
    n_seq = next(seqs)
    kv = type("KV", (), {})()
    kv.struct = lambda: A.orthrus_kv(1, 1, 1, 1 << 22, n_seq, 1024)
    n_tok = sum(c.len for c in chunks) + sum(c.len for c in gen) + len(rows)
    b = Batch(chunks, rows, np.zeros(n_tok, np.int32), gen)
    npre, ndec, items = R.plan(m, m, b, kv, kv)
    n_pieces = _check_coverage(b, small, npre, ndec, items)
    assert n_pieces <= 1024
    for it in items[:npre]:
        if it[7] >= 0:
            assert it[6] - it[5] >= 64
    return n_pieces


@pytest.mark.parametrize("seed", range(24))
def test_plan_invariants_on_random_batches(seed):
    """Random mixes of fresh and resuming chunks (some after long cached prefixes), prompt chunks
    and decode rows on the 7B shape and a group-2 bf16 shape: every query row and key is covered
    once, key pieces follow their rules, slot blocks are disjoint, pieces stay within budget."""
    _random_plan(seed)


def test_random_batches_exercise_key_pieces():
    """The random batches above include tiles cut into key pieces (most seeds) and plans without."""
    n = [_random_plan(s) for s in range(24)]
    assert sum(1 for x in n if x) >= 12 and 0 in n


def test_null_cache_pools_only_for_a_model_without_layers():
    """A model without layers never touches its cache pools, so they may be NULL; with layers a
    NULL pool is rejected before any device work (the block table is required either way)."""
    for n_layers, want in ((0, None), (2, A.ORTHRUS_EINVAL)):
        cfg = tiny_config().replace(n_layers=n_layers)
        m = R.DeviceModel(cfg, make_weights(cfg, 3), device="cpu")
        bt = np.zeros((2, 4), np.int32)
        kv = type("KV", (), {})()
        kv.struct = lambda: A.orthrus_kv(None, None, bt.ctypes.data, 8, 2, 4)
        b = Batch([EmbChunk(0, 0, 5, True)], [DecodeRow(1, 3)], np.zeros(6, np.int32))
        if want is None:
            npre, ndec, _ = R.plan(m, m, b, kv, kv)
            assert npre == cfg.n_kv_heads and ndec == cfg.n_kv_heads
        else:
            with pytest.raises(A.OrthrusError) as e:
                R.plan(m, m, b, kv, kv)
            assert e.value.code == want
        kv.struct = lambda: A.orthrus_kv(None, None, None, 8, 2, 4)
        with pytest.raises(A.OrthrusError) as e:
            R.plan(m, m, b, kv, kv)
        assert e.value.code == A.ORTHRUS_EINVAL


def test_prompt_chunks_need_an_lm_head_only_for_logits():
    """A final prompt chunk asks for logits; the oracle and the library both refuse it on a model
    without an LM head, and both accept a non-final prompt chunk there."""
    cfg = tiny_config()
    W = make_weights(cfg, 2)
    W["lm_head"] = None
    m = R.DeviceModel(cfg, W, device="cpu")
    pk = PagedKV(cfg, 64, 4, 8, 3)
    for s_ in range(4):
        pk.reserve(s_, 40)
    kv = R.DeviceKV.from_paged(pk, device="cpu")
    okv = OracleKV.from_paged(pk)
    ids = draw_tokens(1, 1, 4, cfg.vocab)
    b = Batch([], [], ids, [GenChunk(1, 0, 4, True)])
    with pytest.raises(StepError) as e:
        step_oracle((cfg, W), (cfg, W), b, okv, okv, np.zeros((4, cfg.d_model)), np.zeros(4))
    assert e.value.kind == "desc"
    with pytest.raises(A.OrthrusError) as g:
        R.plan(m, m, b, kv, kv)
    assert g.value.code == A.ORTHRUS_EDESC
    npre, ndec, _ = R.plan(m, m, Batch([], [], ids, [GenChunk(1, 0, 4, False)]), kv, kv)
    assert (npre, ndec) == (cfg.n_kv_heads, 0)


def test_separate_caches_keep_separate_namespaces():
    """With two caches, an embedding chunk and a prompt chunk may name the same seq index."""
    cfg, W, m, pk, kv = _cpu_setup()
    kv2 = type("KV", (), {})()
    kv2.struct = lambda: A.orthrus_kv(2, 2, 2, 64, 6, 8)
    ids = draw_tokens(1, 2, 8, cfg.vocab)
    b = Batch([EmbChunk(1, 0, 4, False)], [], ids, [GenChunk(1, 0, 4, True)])
    npre, ndec, items = R.plan(m, m, b, kv, kv2)
    assert npre == 2 * cfg.n_kv_heads and ndec == 0
    # chunk indices: the embedding chunk is 0, the prompt chunk 1
    assert sorted(set(items[:, 1])) == [0, 1]
    with pytest.raises(A.OrthrusError) as e:
        R.plan(m, m, b, kv, kv)
    assert e.value.code == A.ORTHRUS_EDUPSEQ


def test_plan_covers_prompt_chunks_with_causal_bounds():
    """Prompt chunks are tiled like embedding chunks: every (token, kv head) once, key bound =
    offset + last row + 1, heaviest first across both chunk kinds; decode rows follow."""
    cfg = tiny_config()
    W = make_weights(cfg, 0)
    m = R.DeviceModel(cfg, W, device="cpu")
    kv = type("KV", (), {})()
    kv.struct = lambda: A.orthrus_kv(1, 1, 1, 100000, 8, 600)
    chunks = [EmbChunk(0, 0, 100, True)]
    gen = [GenChunk(1, 0, 130, False), GenChunk(2, 512, 7, True)]
    rows = [DecodeRow(3, 300)]
    ids = np.zeros(100 + 137 + 1, np.int32)
    b = Batch(chunks, rows, ids, gen)
    npre, ndec, items = R.plan(m, m, b, kv, kv)
    allc = [(c.offset, c.len) for c in chunks] + [(c.offset, c.len) for c in gen]
    seen = set()
    work = []
    for it in items[:npre]:
        kind, ci, g, qb, qn, kb, ke, ps = it
        off, ln = allc[ci]
        assert kind == 0 and kb == 0 and ps == -1 and qb + qn <= ln and ke == off + qb + qn
        for r in range(qb, qb + qn):
            assert (ci, g, r) not in seen
            seen.add((ci, g, r))
        work.append(ke * qn)
    assert len(seen) == (100 + 137) * cfg.n_kv_heads
    assert work == sorted(work, reverse=True)
    assert ndec == cfg.n_kv_heads * 2  # 301 keys: two 256-key chunks, fp32 splits of one chunk


def test_sample_greedy_argument_checks():
    t = R.torch
    lg = t.zeros((2, 5))
    out = t.zeros(2, dtype=t.int32)
    for rows, vocab, code in ((-1, 5, A.ORTHRUS_EINVAL), (2, 0, A.ORTHRUS_EINVAL)):
        assert A.orthrus_sample_greedy(ctypes.c_void_p(lg.data_ptr()), rows, vocab,
                                       ctypes.c_void_p(out.data_ptr()), None) == code
    assert A.orthrus_sample_greedy(None, 2, 5, None, None) == A.ORTHRUS_EINVAL
    assert A.orthrus_sample_greedy(None, 0, 5, None, None) == A.ORTHRUS_OK
    with pytest.raises(A.OrthrusError):
        R.sample_greedy(lg.double(), out)


def test_unknown_pooling_codes_and_missing_hidden_buffer():
    cfg, W, m, pk, kv = _cpu_setup()
    t = R.torch
    ids = draw_tokens(1, 0, 8, cfg.vocab)
    acc, accw = t.zeros((6, cfg.d_model)), t.zeros(6)
    emb = t.zeros((1, cfg.d_model))
    ws = type("WS", (), {"buf": t.zeros(64, dtype=t.uint8), "nbytes": 64})()
    for code in (6, 7):
        pb = R.PackedBatch(Batch([EmbChunk(0, 0, 8, True)], [], ids))
        pb._chunks[0].flags = 1 | (code << A.ORTHRUS_POOL_SHIFT)
        with pytest.raises(A.OrthrusError) as e:
            R.step(m, m, None, kv, kv, acc, accw, None, emb, ws, packed=pb)
        assert e.value.code == A.ORTHRUS_EDESC
    # a buffered chunk without a buffer pointer
    b = Batch([EmbChunk(0, 0, 8, True, "buffer")], [], ids, hidden_stride=8)
    with pytest.raises(A.OrthrusError) as e:
        R.step(m, m, b, kv, kv, acc, accw, None, emb, ws)
    assert e.value.code == A.ORTHRUS_EINVAL


def test_adapter_registration_and_host_validation():
    from workload import make_lora
    cfg = tiny_config()
    W = make_weights(cfg, 2)
    W["adapters"] = [make_lora(cfg, 2, 16, tag=t) for t in range(6)]
    m = R.DeviceModel(cfg, W, device="cpu")
    for bad_ad, code in (([make_lora(cfg, 2, 8)], A.ORTHRUS_EUNSUPPORTED),          # qkv rank 24
                         ([make_lora(cfg, 2, 16), make_lora(cfg, 2, 32, tag=1)], A.ORTHRUS_EUNSUPPORTED),
                         ([make_lora(cfg, 2, 160)], A.ORTHRUS_EUNSUPPORTED)):        # qkv rank 480
        with pytest.raises(A.OrthrusError) as e:
            R.DeviceModel(cfg, dict(W, adapters=bad_ad), device="cpu")
        assert e.value.code == code
    pk = PagedKV(cfg, 64, 6, 8, 3)
    for s in range(6):
        pk.reserve(s, 40)
    kv = R.DeviceKV.from_paged(pk, device="cpu")
    okv = OracleKV.from_paged(pk)
    ids = draw_tokens(1, 0, 12, cfg.vocab)
    t = R.torch
    acc, accw = t.zeros((6, cfg.d_model)), t.zeros(6)
    emb = t.zeros((6, cfg.d_model))
    ws = type("WS", (), {"buf": t.zeros(64, dtype=t.uint8), "nbytes": 64})()
    We = dict(W)
    bad = [
        Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[6]),
        Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[-3]),
        Batch([EmbChunk(0, 0, 2, True)], [], ids[:2], chunk_adapter=[0, 1]),
        Batch([EmbChunk(s, 0, 2, True) for s in range(5)], [], ids[:10], chunk_adapter=[0, 1, 2, 3, 4]),
    ]
    for b in bad:
        with pytest.raises(StepError) as e:
            step_oracle((cfg, We), (cfg, We), b, okv, okv, np.zeros((6, cfg.d_model)), np.zeros(6))
        want = KIND_CODE[e.value.kind]
        with pytest.raises(A.OrthrusError) as g:
            R.step(m, m, b, kv, kv, acc, accw, None, emb, ws)
        assert g.value.code == want, (b.chunk_adapter, e.value.kind, g.value.code)
    # four distinct adapters (one of them twice) plan fine
    ok = Batch([EmbChunk(s, 0, 2, True) for s in range(5)], [], ids[:10], chunk_adapter=[3, 1, 3, 0, 5])
    R.plan(m, m, ok, kv, kv)


def test_blocked_weight_sizes():
    """The blocked copy of a [rows][cols] bf16 matrix rounds rows up to whole 64-row blocks and
    needs cols to be a multiple of 64."""
    from paper_2609_25405_amd import _abi as A
    assert A.orthrus_blocked_bytes(32000, 4096) == 32000 * 4096 * 2
    assert A.orthrus_blocked_bytes(100, 64) == 128 * 64 * 2
    assert A.orthrus_blocked_bytes(1, 128) == 64 * 128 * 2
    for rows, cols in ((0, 64), (-1, 64), (64, 0), (64, 96), (64, -64)):
        assert A.orthrus_blocked_bytes(rows, cols) == 0
    assert A.orthrus_block_weights(None, None, 64, 64, None) == A.ORTHRUS_EINVAL
