// The iteration runner: one pass of the heterogeneous-batching loop (Algorithm 1) on one GPU.
// Schedule (the intra-batch scheduler), mirror the block-table rows it assigned to the device,
// Forward + IncPooler + LM head (orthrus_step), Sampler (orthrus_sample_greedy), then Emit:
// finished embeddings and sampled tokens come back to the host and the scheduler commits.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "model.hpp"
#include "orthrus.h"
#include "orthrus_sched.h"

struct orthrus_runner {
    const orthrus_model *emb = nullptr, *gen = nullptr;
    orthrus_kv kv[2]{};   // embedding cache, generator cache (the same one when shared)
    orthrus_sched *sched = nullptr;
    orthrus_runner_buffers buf{};
    orthrus_sched_config scfg{};
    int d = 0, vocab = 0;
    // pinned host staging (grown on demand; each iteration synchronises before it is reused)
    void *rows_pin = nullptr, *tok_pin = nullptr, *emb_pin = nullptr;
    size_t rows_cap = 0, tok_cap = 0, emb_cap = 0;
    // outputs of the last iteration
    std::vector<int64_t> token_ids, emb_ids, finished;
    std::vector<int32_t> tokens;
    std::vector<float> embeddings;
};

namespace {

int grow_pinned(void **p, size_t *cap, size_t bytes) {
    if (*cap >= bytes) return ORTHRUS_OK;
    if (*p) (void)hipHostFree(*p);
    *p = nullptr;
    *cap = 0;
    if (hipHostMalloc(p, std::max<size_t>(bytes, 4096), hipHostMallocDefault) != hipSuccess) return ORTHRUS_EHIP;
    *cap = std::max<size_t>(bytes, 4096);
    return ORTHRUS_OK;
}

#define HIP_TRY(expr)                                   \
    do {                                                \
        if ((expr) != hipSuccess) return ORTHRUS_EHIP;  \
    } while (0)

}  // namespace

extern "C" {

int orthrus_runner_create(const orthrus_model *emb, const orthrus_model *gen, const orthrus_kv *emb_kv,
                          const orthrus_kv *gen_kv, orthrus_sched *sched, const orthrus_runner_buffers *buf,
                          orthrus_runner **out) {
    if (!emb || !gen || !emb_kv || !gen_kv || !sched || !buf || !out) return ORTHRUS_EINVAL;
    *out = nullptr;
    if (!buf->acc_sum || !buf->acc_w || !buf->logits || !buf->out_emb || !buf->tokens || !buf->workspace)
        return ORTHRUS_EINVAL;
    orthrus_sched_config sc{};
    if (orthrus_sched_get_config(sched, &sc)) return ORTHRUS_EINVAL;
    const bool shared = emb_kv->k_cache == gen_kv->k_cache;
    if (sc.shared_cache != (shared ? 1 : 0)) return ORTHRUS_EINVAL;
    if (sc.decode_tokens != 1 || sc.page_size != emb->cfg.page_size) return ORTHRUS_EINVAL;
    const orthrus_kv *kvs[2] = {emb_kv, gen_kv};
    int max_ctx = 0;
    for (int c = 0; c < (shared ? 1 : 2); ++c) {
        // block-table rows must have the scheduler's stride; slots and pages must exist
        if (kvs[c]->max_blocks != sc.max_blocks[c] || kvs[c]->n_seq < sc.n_seq[c] || kvs[c]->n_pages < sc.n_pages[c])
            return ORTHRUS_ECAPACITY;
        max_ctx = std::max(max_ctx, sc.max_blocks[c] * sc.page_size);
    }
    const int B = sc.budget;
    const size_t need = orthrus_workspace_bytes(emb, gen, B, B, B, max_ctx);
    if (need == 0) return ORTHRUS_EINVAL;
    if (buf->ws_bytes < need) return ORTHRUS_ECAPACITY;
    orthrus_runner *r = new (std::nothrow) orthrus_runner;
    if (!r) return ORTHRUS_EINVAL;
    r->emb = emb;
    r->gen = gen;
    r->kv[0] = *emb_kv;
    r->kv[1] = *gen_kv;
    r->sched = sched;
    r->buf = *buf;
    r->scfg = sc;
    r->d = emb->cfg.d_model;
    r->vocab = gen->cfg.vocab;
    *out = r;
    return ORTHRUS_OK;
}

void orthrus_runner_destroy(orthrus_runner *r) {
    if (!r) return;
    for (void *p : {r->rows_pin, r->tok_pin, r->emb_pin})
        if (p) (void)hipHostFree(p);
    delete r;
}

int orthrus_runner_iterate(orthrus_runner *r, void *stream, orthrus_runner_output *out) {
    if (!r || !out) return ORTHRUS_EINVAL;
    std::memset(out, 0, sizeof(*out));
    r->token_ids.clear();
    r->tokens.clear();
    r->emb_ids.clear();
    r->embeddings.clear();
    r->finished.clear();
    hipStream_t s = (hipStream_t)stream;
    orthrus_sched_batch b{};
    int rc = orthrus_sched_next(r->sched, &b);
    if (rc) return rc;
    const orthrus_batch &bt = b.batch;
    const int n_items = bt.n_chunks + bt.n_gen_chunks + bt.n_decode;
    if (n_items == 0) {
        int32_t nf = 0;
        return orthrus_sched_commit(r->sched, nullptr, 0, &nf, nullptr, 0);
    }
    // block-table rows assigned by this batch's admissions
    if (b.n_table_rows > 0) {
        size_t bytes = 0;
        for (int i = 0; i < b.n_table_rows; ++i) bytes += (size_t)r->scfg.max_blocks[b.table_rows[2 * i]] * 4;
        rc = grow_pinned(&r->rows_pin, &r->rows_cap, bytes);
        if (rc) return rc;
        char *stage = (char *)r->rows_pin;
        for (int i = 0; i < b.n_table_rows; ++i) {
            const int c = b.table_rows[2 * i], slot = b.table_rows[2 * i + 1];
            const size_t row_bytes = (size_t)r->scfg.max_blocks[c] * 4;
            const int32_t *host = orthrus_sched_block_table(r->sched, c) + (size_t)slot * r->scfg.max_blocks[c];
            std::memcpy(stage, host, row_bytes);
            char *dev = (char *)r->kv[c].block_table + (size_t)slot * row_bytes;
            HIP_TRY(hipMemcpyAsync(dev, stage, row_bytes, hipMemcpyHostToDevice, s));
            stage += row_bytes;
        }
    }
    const orthrus_kv *gkv = r->scfg.shared_cache ? &r->kv[0] : &r->kv[1];
    rc = orthrus_step(r->emb, r->gen, &bt, &r->kv[0], gkv, r->buf.acc_sum, r->buf.acc_w, r->buf.logits,
                      r->buf.out_emb, r->buf.workspace, r->buf.ws_bytes, stream);
    if (rc) return rc;
    const int nl = b.n_logit_rows;
    rc = orthrus_sample_greedy(r->buf.logits, nl, r->vocab, r->buf.tokens, stream);
    if (rc) return rc;
    rc = grow_pinned(&r->tok_pin, &r->tok_cap, (size_t)nl * 4);
    if (rc) return rc;
    if (nl > 0) HIP_TRY(hipMemcpyAsync(r->tok_pin, r->buf.tokens, (size_t)nl * 4, hipMemcpyDeviceToHost, s));
    if (bt.n_chunks > 0) {
        rc = grow_pinned(&r->emb_pin, &r->emb_cap, (size_t)bt.n_chunks * r->d * 4);
        if (rc) return rc;
        HIP_TRY(hipMemcpyAsync(r->emb_pin, r->buf.out_emb, (size_t)bt.n_chunks * r->d * 4, hipMemcpyDeviceToHost, s));
    }
    int32_t bits = 0;
    const int dev_rc = orthrus_device_error(r->buf.workspace, stream, &bits);  // synchronises
    if (dev_rc != ORTHRUS_OK && dev_rc != ORTHRUS_EDEVICE) return dev_rc;
    const int32_t *tok = (const int32_t *)r->tok_pin;
    for (int i = 0; i < nl; ++i) {
        r->token_ids.push_back(b.logit_ids[i]);
        r->tokens.push_back(tok[i]);
    }
    for (int i = 0; i < bt.n_chunks; ++i) {
        if (!(bt.chunks[i].flags & ORTHRUS_CHUNK_LAST)) continue;
        r->emb_ids.push_back(b.chunk_ids[i]);
        const float *e = (const float *)r->emb_pin + (size_t)i * r->d;
        r->embeddings.insert(r->embeddings.end(), e, e + r->d);
    }
    out->tokens_used = b.tokens_used;
    out->n_items = n_items;
    int32_t nf = 0;
    r->finished.resize((size_t)b.n_finishing + nl);
    rc = orthrus_sched_commit(r->sched, nl ? r->tokens.data() : nullptr, nl, &nf, r->finished.data(),
                              (int32_t)r->finished.size());
    if (rc) return rc;
    r->finished.resize(nf);
    out->n_tokens = nl;
    out->token_ids = r->token_ids.data();
    out->tokens = r->tokens.data();
    out->n_embeddings = (int32_t)r->emb_ids.size();
    out->embedding_ids = r->emb_ids.data();
    out->embeddings = r->embeddings.data();
    out->n_finished = nf;
    out->finished_ids = r->finished.data();
    return dev_rc;
}

}  // extern "C"
