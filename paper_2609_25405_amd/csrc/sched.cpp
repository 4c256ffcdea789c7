// Intra-batch scheduling (Algorithm 2, Section 4) with ScheduleRunning and ScheduleOne, plus the
// request life cycle around it: queues, persistent credits, sequence slots, page reservations and
// the host block tables.  Plain C++17, no device calls.
//
// One iteration: ScheduleRunning gives every decode-phase request (in phase order) its decode item
// while the budget holds it; then, with w_e / w_g = remaining tokens of the embedding / generation
// queues, both credits grow by their weight on every pass and the queue with the larger credit
// (embedding on ties) gives up one item through ScheduleOne and pays w_e + w_g.  Credits persist
// across iterations and reset when their queue is empty at the start of one.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <deque>
#include <memory>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "orthrus_sched.h"

namespace {

struct Req {
    int64_t id = 0;
    bool emb = true;
    int32_t n = 0, max_new = 0, pool = 0, adapter = -1;
    int32_t done = 0, generated = 0;
    bool admitted = false;
    int32_t cache = 0, slot = -1;
    std::vector<int32_t> pages;
    std::vector<int32_t> tokens;  // empty: zeros
    std::vector<float> weights;   // weighted-mean requests: one per token
    int32_t last_token = 0;
    int64_t batch_iter = -1;      // iteration whose batch holds this request
    int32_t remaining() const { return n - done; }
};

struct Cache {
    int32_t n_seq = 0, n_pages = 0, max_blocks = 0;
    std::deque<int32_t> free_slots, free_pages;
    std::vector<int32_t> table;  // [n_seq][max_blocks]
};

}  // namespace

struct orthrus_sched {
    orthrus_sched_config cfg{};
    std::unordered_map<int64_t, std::unique_ptr<Req>> reqs;
    std::vector<Req *> Qe, Qg, running;
    int64_t a_e = 0, a_g = 0;
    Cache caches[2];
    int64_t iter = 0;
    bool pending = false;
    // the batch of the current iteration
    std::vector<orthrus_emb_chunk> chunks;
    std::vector<orthrus_gen_chunk> gchunks;
    std::vector<orthrus_decode_row> rows;
    std::vector<int32_t> tokens, row_tokens, table_rows, chunk_adapter;
    std::vector<float> token_weights;
    std::vector<int32_t> batch_adapters;  // distinct adapters of this batch's embedding chunks
    std::vector<int64_t> chunk_ids, gen_ids, row_ids, logit_ids, finishing_ids;
    std::vector<Req *> logit_reqs, finishing;
    std::string picks;

    int cache_of(const Req &r) const { return (cfg.shared_cache || r.emb) ? 0 : 1; }
    int32_t reservation(const Req &r) const {
        const int64_t positions = r.emb ? r.n : (int64_t)r.n + r.max_new - 1;
        return (int32_t)((positions + cfg.page_size - 1) / cfg.page_size);
    }
};

namespace {

// a request submitted between orthrus_sched_next and _commit only joins its queue: the pending
// batch is not affected
int submit(orthrus_sched *s, std::unique_ptr<Req> r, const int32_t *tokens) {
    if (r->n < 1 || (!r->emb && r->max_new < 1) || s->reqs.count(r->id)) return ORTHRUS_EINVAL;
    if (!r->emb && (int64_t)r->n + r->max_new - 1 > INT32_MAX) return ORTHRUS_EINVAL;
    const Cache &c = s->caches[s->cache_of(*r)];
    const int32_t need = s->reservation(*r);
    if (need > c.max_blocks || need > c.n_pages) return ORTHRUS_ECAPACITY;
    if (tokens) r->tokens.assign(tokens, tokens + r->n);
    Req *p = r.get();
    s->reqs.emplace(r->id, std::move(r));
    (p->emb ? s->Qe : s->Qg).push_back(p);
    return ORTHRUS_OK;
}

// ScheduleOne's candidate in Q: (request, chunk length) or length 0 when Q cannot contribute
int32_t candidate(orthrus_sched *s, std::vector<Req *> &Q, int32_t B, Req **out) {
    Req *r = nullptr;
    for (Req *q : Q)
        if (q->batch_iter != s->iter) {
            r = q;
            break;
        }
    if (!r) return 0;
    int32_t n;
    if (r->emb && s->cfg.atomic_embeddings) {
        if (r->remaining() > B) return 0;
        n = r->remaining();
    } else {
        n = std::min(std::min(s->cfg.chunk, r->remaining()), B);
    }
    if (!r->admitted) {
        const Cache &c = s->caches[s->cache_of(*r)];
        if (c.free_slots.empty() || (int64_t)c.free_pages.size() < s->reservation(*r)) return 0;
    }
    if (r->adapter >= 0 &&
        std::find(s->batch_adapters.begin(), s->batch_adapters.end(), r->adapter) == s->batch_adapters.end() &&
        (int)s->batch_adapters.size() == ORTHRUS_MAX_STEP_ADAPTERS)
        return 0;
    *out = r;
    return n;
}

void admit(orthrus_sched *s, Req *r, int32_t n) {
    if (!r->admitted) {
        const int ci = s->cache_of(*r);
        Cache &c = s->caches[ci];
        r->cache = ci;
        r->slot = c.free_slots.front();
        c.free_slots.pop_front();
        const int32_t need = s->reservation(*r);
        int32_t *row = &c.table[(size_t)r->slot * c.max_blocks];
        for (int32_t b = 0; b < need; ++b) {
            r->pages.push_back(c.free_pages.front());
            c.free_pages.pop_front();
            row[b] = r->pages.back();
        }
        s->table_rows.push_back(ci);
        s->table_rows.push_back(r->slot);
        r->admitted = true;
    }
    const bool last = r->done + n == r->n;
    r->batch_iter = s->iter;
    if (r->emb) {
        orthrus_emb_chunk c{r->slot, r->done, n, (last ? ORTHRUS_CHUNK_LAST : 0) | (r->pool << ORTHRUS_POOL_SHIFT)};
        s->chunks.push_back(c);
        s->chunk_ids.push_back(r->id);
        s->chunk_adapter.push_back(r->adapter);
        if (r->adapter >= 0 &&
            std::find(s->batch_adapters.begin(), s->batch_adapters.end(), r->adapter) == s->batch_adapters.end())
            s->batch_adapters.push_back(r->adapter);
    } else {
        orthrus_gen_chunk c{r->slot, r->done, n, last ? ORTHRUS_CHUNK_LAST : 0};
        s->gchunks.push_back(c);
        s->gen_ids.push_back(r->id);
    }
    r->done += n;
    if (!last) return;
    if (r->emb) {
        s->Qe.erase(std::find(s->Qe.begin(), s->Qe.end(), r));
        s->finishing.push_back(r);
    } else {
        s->Qg.erase(std::find(s->Qg.begin(), s->Qg.end(), r));
        s->logit_reqs.push_back(r);
        r->generated = 1;
        if (r->generated == r->max_new) s->finishing.push_back(r);
        else s->running.push_back(r);
    }
}

void release(orthrus_sched *s, Req *r) {
    if (r->admitted) {
        Cache &c = s->caches[r->cache];
        int32_t *row = &c.table[(size_t)r->slot * c.max_blocks];
        for (size_t b = 0; b < r->pages.size(); ++b) row[b] = -1;
        for (int32_t p : r->pages) c.free_pages.push_back(p);
        c.free_slots.push_back(r->slot);
    }
    s->reqs.erase(r->id);
}

}  // namespace

extern "C" {

int orthrus_sched_create(const orthrus_sched_config *cfg, orthrus_sched **out) {
    if (!cfg || !out) return ORTHRUS_EINVAL;
    *out = nullptr;
    const orthrus_sched_config &c = *cfg;
    if (c.budget < 1 || c.chunk < 1 || c.decode_tokens < 1 || c.page_size < 1) return ORTHRUS_EINVAL;
    if (c.atomic_embeddings != 0 && c.atomic_embeddings != 1) return ORTHRUS_EINVAL;
    if (c.shared_cache != 0 && c.shared_cache != 1) return ORTHRUS_EINVAL;
    const int n_caches = c.shared_cache ? 1 : 2;
    for (int i = 0; i < n_caches; ++i)
        if (c.n_seq[i] < 1 || c.n_pages[i] < 1 || c.max_blocks[i] < 1) return ORTHRUS_EINVAL;
    orthrus_sched *s = new (std::nothrow) orthrus_sched;
    if (!s) return ORTHRUS_EINVAL;
    s->cfg = c;
    for (int i = 0; i < n_caches; ++i) {
        Cache &k = s->caches[i];
        k.n_seq = c.n_seq[i];
        k.n_pages = c.n_pages[i];
        k.max_blocks = c.max_blocks[i];
        for (int32_t j = 0; j < k.n_seq; ++j) k.free_slots.push_back(j);
        for (int32_t j = 0; j < k.n_pages; ++j) k.free_pages.push_back(j);
        k.table.assign((size_t)k.n_seq * k.max_blocks, -1);
    }
    *out = s;
    return ORTHRUS_OK;
}

void orthrus_sched_destroy(orthrus_sched *s) { delete s; }

int orthrus_sched_submit_embedding(orthrus_sched *s, int64_t id, const int32_t *tokens,
                                   const float *weights, int32_t n, int32_t pool, int32_t adapter) {
    if (!s || n < 1 || adapter < -1) return ORTHRUS_EINVAL;
    if (pool != ORTHRUS_POOL_MEAN && pool != ORTHRUS_POOL_LAST && pool != ORTHRUS_POOL_CLS &&
        pool != ORTHRUS_POOL_WMEAN)
        return ORTHRUS_EINVAL;
    if (pool == ORTHRUS_POOL_WMEAN) {
        if (!weights) return ORTHRUS_EINVAL;
        for (int32_t i = 0; i < n; ++i)
            if (!std::isfinite(weights[i]) || weights[i] < 0.f) return ORTHRUS_EINVAL;
    }
    std::unique_ptr<Req> r(new (std::nothrow) Req);
    if (!r) return ORTHRUS_EINVAL;
    r->id = id;
    r->emb = true;
    r->n = n;
    r->pool = pool;
    r->adapter = adapter;
    if (pool == ORTHRUS_POOL_WMEAN) r->weights.assign(weights, weights + n);
    return submit(s, std::move(r), tokens);
}

int orthrus_sched_submit_generation(orthrus_sched *s, int64_t id, const int32_t *prompt, int32_t n,
                                    int32_t max_new) {
    if (!s) return ORTHRUS_EINVAL;
    std::unique_ptr<Req> r(new (std::nothrow) Req);
    if (!r) return ORTHRUS_EINVAL;
    r->id = id;
    r->emb = false;
    r->n = n;
    r->max_new = max_new;
    return submit(s, std::move(r), prompt);
}

int orthrus_sched_next(orthrus_sched *s, orthrus_sched_batch *out) {
    if (!s || !out || s->pending) return ORTHRUS_EINVAL;
    s->iter++;
    s->chunks.clear();
    s->gchunks.clear();
    s->rows.clear();
    s->tokens.clear();
    s->token_weights.clear();
    s->chunk_adapter.clear();
    s->batch_adapters.clear();
    s->row_tokens.clear();
    s->table_rows.clear();
    s->chunk_ids.clear();
    s->gen_ids.clear();
    s->row_ids.clear();
    s->logit_ids.clear();
    s->finishing_ids.clear();
    s->logit_reqs.clear();
    s->finishing.clear();
    s->picks.clear();
    const orthrus_sched_config &cfg = s->cfg;
    int32_t B = cfg.budget;

    // ScheduleRunning
    std::vector<Req *> still, decoded;
    bool blocked = false;
    for (Req *r : s->running) {
        const int32_t k = std::min(cfg.decode_tokens, r->max_new - r->generated);
        if (blocked || k > B) {
            blocked = true;
            still.push_back(r);
            continue;
        }
        s->rows.push_back(orthrus_decode_row{r->slot, r->n + r->generated - 1});
        s->row_ids.push_back(r->id);
        s->row_tokens.push_back(k);
        decoded.push_back(r);
        r->batch_iter = s->iter;
        B -= k;
        r->generated += k;
        if (r->generated == r->max_new) s->finishing.push_back(r);
        else still.push_back(r);
    }
    s->running.swap(still);

    // Algorithm 2
    int64_t w_e = 0, w_g = 0;
    for (Req *r : s->Qe) w_e += r->remaining();
    for (Req *r : s->Qg) w_g += r->remaining();
    if (s->Qe.empty()) s->a_e = 0;
    if (s->Qg.empty()) s->a_g = 0;
    bool stop_e = false, stop_g = false;
    while (B > 0) {
        Req *re = nullptr, *rg = nullptr;
        const int32_t ne = stop_e ? 0 : candidate(s, s->Qe, B, &re);
        const int32_t ng = stop_g ? 0 : candidate(s, s->Qg, B, &rg);
        stop_e = ne == 0;
        stop_g = ng == 0;
        if (stop_e && stop_g) break;
        s->a_e += w_e;
        s->a_g += w_g;
        if (stop_g || (!stop_e && s->a_e >= s->a_g)) {
            admit(s, re, ne);
            s->a_e -= w_e + w_g;
            s->picks.push_back('e');
            B -= ne;
        } else {
            admit(s, rg, ng);
            s->a_g -= w_e + w_g;
            s->picks.push_back('g');
            B -= ng;
        }
    }

    // token ids in batch order: embedding chunks, prompt chunks, decode inputs
    for (size_t i = 0; i < s->chunks.size(); ++i) {
        const Req &r = *s->reqs[s->chunk_ids[i]];
        const orthrus_emb_chunk &c = s->chunks[i];
        if (r.tokens.empty()) s->tokens.insert(s->tokens.end(), c.len, 0);
        else s->tokens.insert(s->tokens.end(), r.tokens.begin() + c.offset, r.tokens.begin() + c.offset + c.len);
    }
    for (size_t i = 0; i < s->gchunks.size(); ++i) {
        const Req &r = *s->reqs[s->gen_ids[i]];
        const orthrus_gen_chunk &c = s->gchunks[i];
        if (r.tokens.empty()) s->tokens.insert(s->tokens.end(), c.len, 0);
        else s->tokens.insert(s->tokens.end(), r.tokens.begin() + c.offset, r.tokens.begin() + c.offset + c.len);
    }
    for (Req *r : decoded) s->tokens.push_back(r->last_token);
    // per-token weights of the embedding chunks, when a weighted-mean request is in the batch
    bool any_weighted = false;
    for (size_t i = 0; i < s->chunks.size(); ++i) any_weighted |= !s->reqs[s->chunk_ids[i]]->weights.empty();
    if (any_weighted)
        for (size_t i = 0; i < s->chunks.size(); ++i) {
            const Req &r = *s->reqs[s->chunk_ids[i]];
            const orthrus_emb_chunk &c = s->chunks[i];
            if (r.weights.empty()) s->token_weights.insert(s->token_weights.end(), c.len, 1.f);
            else s->token_weights.insert(s->token_weights.end(), r.weights.begin() + c.offset,
                                         r.weights.begin() + c.offset + c.len);
        }
    // logits rows: final prompt chunks, then decode rows
    for (Req *r : decoded) s->logit_reqs.push_back(r);
    for (Req *r : s->logit_reqs) s->logit_ids.push_back(r->id);
    for (Req *r : s->finishing) s->finishing_ids.push_back(r->id);

    std::memset(out, 0, sizeof(*out));
    out->batch.n_chunks = (int32_t)s->chunks.size();
    out->batch.n_decode = (int32_t)s->rows.size();
    out->batch.chunks = s->chunks.data();
    out->batch.rows = s->rows.data();
    out->batch.token_ids = s->tokens.data();
    out->batch.n_gen_chunks = (int32_t)s->gchunks.size();
    out->batch.gen_chunks = s->gchunks.data();
    out->batch.token_weights = any_weighted ? s->token_weights.data() : nullptr;
    out->batch.chunk_adapter = s->batch_adapters.empty() ? nullptr : s->chunk_adapter.data();
    out->chunk_ids = s->chunk_ids.data();
    out->gen_chunk_ids = s->gen_ids.data();
    out->row_ids = s->row_ids.data();
    out->row_tokens = s->row_tokens.data();
    out->n_logit_rows = (int32_t)s->logit_ids.size();
    out->logit_ids = s->logit_ids.data();
    out->tokens_used = cfg.budget - B;
    out->n_picks = (int32_t)s->picks.size();
    out->picks = s->picks.data();
    out->n_finishing = (int32_t)s->finishing_ids.size();
    out->finishing_ids = s->finishing_ids.data();
    out->n_table_rows = (int32_t)s->table_rows.size() / 2;
    out->table_rows = s->table_rows.data();
    out->credit_e = s->a_e;
    out->credit_g = s->a_g;
    s->pending = true;
    return ORTHRUS_OK;
}

int orthrus_sched_commit(orthrus_sched *s, const int32_t *sampled, int32_t n, int32_t *n_finished,
                         int64_t *finished, int32_t cap) {
    if (!s || !s->pending) return ORTHRUS_EINVAL;
    if (sampled ? n != (int32_t)s->logit_reqs.size() : n != 0) return ORTHRUS_EINVAL;
    std::vector<Req *> done = s->finishing;
    if (sampled) {
        for (int32_t i = 0; i < n; ++i) {
            Req *r = s->logit_reqs[i];
            r->last_token = sampled[i];
            if (s->cfg.eos_token >= 0 && sampled[i] == s->cfg.eos_token &&
                std::find(done.begin(), done.end(), r) == done.end()) {
                done.push_back(r);
                auto it = std::find(s->running.begin(), s->running.end(), r);
                if (it != s->running.end()) s->running.erase(it);
            }
        }
    }
    int32_t k = 0;
    for (Req *r : done) {
        if (finished && k < cap) finished[k] = r->id;
        ++k;
        release(s, r);
    }
    if (n_finished) *n_finished = k;
    s->pending = false;
    return ORTHRUS_OK;
}

const int32_t *orthrus_sched_block_table(const orthrus_sched *s, int32_t cache) {
    if (!s || cache < 0 || cache > 1 || (cache == 1 && s->cfg.shared_cache)) return nullptr;
    return s->caches[cache].table.data();
}

int orthrus_sched_get_config(const orthrus_sched *s, orthrus_sched_config *out) {
    if (!s || !out) return ORTHRUS_EINVAL;
    *out = s->cfg;
    return ORTHRUS_OK;
}

int orthrus_sched_counts(const orthrus_sched *s, int64_t *counts7) {
    if (!s || !counts7) return ORTHRUS_EINVAL;
    counts7[0] = (int64_t)s->Qe.size();
    counts7[1] = (int64_t)s->Qg.size();
    counts7[2] = (int64_t)s->running.size();
    for (int i = 0; i < 2; ++i) {
        counts7[3 + 2 * i] = (int64_t)s->caches[i].free_slots.size();
        counts7[4 + 2 * i] = (int64_t)s->caches[i].free_pages.size();
    }
    return ORTHRUS_OK;
}

}  // extern "C"
