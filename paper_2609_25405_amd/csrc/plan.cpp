// Host planner for the mixed step (Section 3.2 batch unit, Section 3.3 chunk bookkeeping).
//
// Turns the caller's descriptor into the metadata the kernels read: per token its id,
// absolute position and request; per chunk (embedding and generation prefill) its request,
// offset, length, flags and first token; per decode row its request, context and split
// layout; the attention work list; and the rows that get logits.  Validation mirrors the step
// contract: every check here runs before anything is enqueued, so a rejected batch leaves all
// caller buffers untouched.
#include "plan.hpp"

#include <algorithm>
#include <array>
#include <climits>
#include <cmath>
#include <cstring>
#include <numeric>
#include <set>
#include <utility>

namespace orthrus {

int validate_config(const orthrus_config &c) {
    if (c.n_layers < 0 || c.d_model <= 0 || c.n_q_heads <= 0 || c.n_kv_heads <= 0 ||
        c.head_dim <= 0 || c.d_ff <= 0 || c.vocab <= 0 || c.page_size <= 0 || !(c.rms_eps > 0.f) ||
        !(c.rope_base > 1.f))
        return ORTHRUS_EINVAL;
    if (c.n_q_heads % c.n_kv_heads) return ORTHRUS_EINVAL;
    if (c.dtype != ORTHRUS_F32 && c.dtype != ORTHRUS_BF16) return ORTHRUS_EINVAL;
    const int group = c.n_q_heads / c.n_kv_heads;
    if (c.head_dim != 64 && c.head_dim != 128) return ORTHRUS_EUNSUPPORTED;
    if (group != 1 && group != 2 && group != 4) return ORTHRUS_EUNSUPPORTED;
    if (c.page_size != 16) return ORTHRUS_EUNSUPPORTED;
    const int align = c.dtype == ORTHRUS_BF16 ? 256 : 64;
    if (c.d_model % align || c.d_ff % align) return ORTHRUS_EUNSUPPORTED;
    if ((c.n_q_heads * c.head_dim) % align) return ORTHRUS_EUNSUPPORTED;
    return ORTHRUS_OK;
}

int max_splits_for_ctx(int max_ctx, int page_size) {
    const int pages = (max_ctx + 1 + page_size - 1) / page_size;
    return std::max(1, (pages + kSplitPages - 1) / kSplitPages);
}

int plan_step(const Model &emb, const Model &gen, const orthrus_batch &b, const orthrus_kv &ekv,
              const orthrus_kv &gkv, StepPlan &p) {
    if (b.n_chunks < 0 || b.n_decode < 0 || b.n_gen_chunks < 0) return ORTHRUS_EINVAL;
    if ((b.n_chunks && !b.chunks) || (b.n_decode && !b.rows) || (b.n_gen_chunks && !b.gen_chunks))
        return ORTHRUS_EINVAL;
    const int P = emb.cfg.page_size;
    p = StepPlan();
    p.n_chunks = b.n_chunks;
    p.n_gen = b.n_gen_chunks;
    p.D = b.n_decode;
    p.shared_kv = ekv.k_cache == gkv.k_cache;
    // one sequence namespace per cache: generation items share the embedding one when the
    // caches are the same
    const int gen_ns = p.shared_kv ? 0 : 1;
    long long Te = 0, Tg = 0;
    int n_last_gen = 0;
    std::set<std::pair<int, int>> seen;  // (namespace, seq)
    for (int i = 0; i < b.n_chunks; ++i) {
        const orthrus_emb_chunk &c = b.chunks[i];
        const int pool = (c.flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK;
        if (c.seq < 0 || c.seq >= ekv.n_seq || c.offset < 0 || c.len < 1) return ORTHRUS_EDESC;
        if (c.flags & ~(ORTHRUS_CHUNK_LAST | (ORTHRUS_POOL_MASK << ORTHRUS_POOL_SHIFT))) return ORTHRUS_EDESC;
        if (pool > ORTHRUS_POOL_BUFFER) return ORTHRUS_EDESC;
        if (pool == ORTHRUS_POOL_NONE && (c.flags & ORTHRUS_CHUNK_LAST)) return ORTHRUS_EDESC;
        if ((long long)c.offset + c.len > (long long)ekv.max_blocks * P) return ORTHRUS_ECAPACITY;
        if (pool == ORTHRUS_POOL_BUFFER && (long long)c.offset + c.len > b.hidden_stride) return ORTHRUS_ECAPACITY;
        if (!seen.insert({0, c.seq}).second) return ORTHRUS_EDUPSEQ;
        Te += c.len;
        p.any_mean |= pool == ORTHRUS_POOL_MEAN;
        p.any_wmean |= pool == ORTHRUS_POOL_WMEAN;
        p.any_buffer |= pool == ORTHRUS_POOL_BUFFER;
    }
    if (p.any_buffer && !b.hidden) return ORTHRUS_EINVAL;
    if (p.any_buffer && (long long)ekv.n_seq * b.hidden_stride > INT32_MAX) return ORTHRUS_ECAPACITY;
    for (int i = 0; i < b.n_gen_chunks; ++i) {
        const orthrus_gen_chunk &c = b.gen_chunks[i];
        if (c.seq < 0 || c.seq >= gkv.n_seq || c.offset < 0 || c.len < 1) return ORTHRUS_EDESC;
        if (c.flags & ~ORTHRUS_CHUNK_LAST) return ORTHRUS_EDESC;
        if ((long long)c.offset + c.len > (long long)gkv.max_blocks * P) return ORTHRUS_ECAPACITY;
        if (!seen.insert({gen_ns, c.seq}).second) return ORTHRUS_EDUPSEQ;
        Tg += c.len;
        n_last_gen += c.flags & ORTHRUS_CHUNK_LAST;
    }
    for (int j = 0; j < b.n_decode; ++j) {
        const orthrus_decode_row &r = b.rows[j];
        if (r.seq < 0 || r.seq >= gkv.n_seq || r.ctx_len < 0) return ORTHRUS_EDESC;
        if ((long long)r.ctx_len + 1 > (long long)gkv.max_blocks * P) return ORTHRUS_ECAPACITY;
        if (!seen.insert({gen_ns, r.seq}).second) return ORTHRUS_EDUPSEQ;
    }
    if (Te + Tg + b.n_decode > (1LL << 30)) return ORTHRUS_ECAPACITY;
    p.Te = (int)Te;
    p.Tg = (int)Tg;
    p.T = p.Te + p.Tg + p.D;
    p.n_lm = n_last_gen + p.D;
    if (p.n_lm > 0 && !gen.w.lm_head) return ORTHRUS_EDESC;
    if (p.T > 0 && !b.token_ids) return ORTHRUS_EINVAL;
    for (int t = 0; t < p.T; ++t) {
        const int v = t < p.Te ? emb.cfg.vocab : gen.cfg.vocab;
        if (b.token_ids[t] < 0 || b.token_ids[t] >= v) return ORTHRUS_EDESC;
    }
    if (b.chunk_adapter) {
        for (int i = 0; i < b.n_chunks; ++i) {
            const int ad = b.chunk_adapter[i];
            if (ad < -1 || ad >= (int)emb.adapters.size()) return ORTHRUS_EDESC;
            if (ad < 0) continue;
            bool seen_ad = false;
            for (int u = 0; u < p.n_used; ++u) seen_ad |= p.used[u] == ad;
            if (seen_ad) continue;
            if (p.n_used == ORTHRUS_MAX_STEP_ADAPTERS) return ORTHRUS_ECAPACITY;
            p.used[p.n_used++] = ad;
        }
    }
    if (p.any_wmean) {
        if (!b.token_weights) return ORTHRUS_EDESC;
        int t = 0;
        for (int i = 0; i < b.n_chunks; ++i) {
            const orthrus_emb_chunk &c = b.chunks[i];
            if (((c.flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK) == ORTHRUS_POOL_WMEAN)
                for (int k = 0; k < c.len; ++k) {
                    const float w = b.token_weights[t + k];
                    if (!std::isfinite(w) || w < 0.f) return ORTHRUS_EDESC;
                }
            t += c.len;
        }
    }

    // chunk table entries of both chunk kinds: {seq, offset, len, flags, first token}
    const int n_all = b.n_chunks + b.n_gen_chunks;
    std::vector<int32_t> chunks(kChunkInts * n_all);
    {
        int t = 0;
        for (int i = 0; i < n_all; ++i) {
            int32_t *ch = &chunks[kChunkInts * i];
            if (i < b.n_chunks) {
                const orthrus_emb_chunk &c = b.chunks[i];
                ch[0] = c.seq, ch[1] = c.offset, ch[2] = c.len, ch[3] = c.flags;
            } else {
                const orthrus_gen_chunk &c = b.gen_chunks[i - b.n_chunks];
                ch[0] = c.seq, ch[1] = c.offset, ch[2] = c.len, ch[3] = c.flags | kChunkGen;
            }
            ch[4] = t;
            t += ch[2];
        }
    }

    const int nkv = emb.cfg.n_kv_heads;
    const int group = emb.group();
    const int qrows = kPrefillRows / group;  // tokens per prefill item

    // --- attention work list: prefill query tiles (heaviest first), then decode splits
    struct Pre { long long work; int chunk, kvh, qb, qn, k0, k1, piece; };
    std::vector<Pre> tiles;
    for (int i = 0; i < n_all; ++i) {
        const int32_t *ch = &chunks[kChunkInts * i];
        const int off = ch[1], len = ch[2];
        for (int qb = 0; qb < len; qb += qrows) {
            const int qn = std::min(qrows, len - qb);
            const int kend = off + qb + qn;
            for (int g = 0; g < nkv; ++g) tiles.push_back({(long long)kend * qn, i, g, qb, qn, 0, kend, -1});
        }
    }
    std::stable_sort(tiles.begin(), tiles.end(), [](const Pre &a, const Pre &b2) { return a.work > b2.work; });
    // key splits of the longest tiles (bf16): cuts on 64-key boundaries at or before the tile's
    // first query position, so only the last piece reaches the causal diagonal; heaviest tiles
    // first while the piece budget lasts
    std::vector<Pre> pre;
    struct Merge { int tok, qn, kvh, n, piece0; };
    std::vector<Merge> merges;
    int n_pieces = 0;
    {
        long long keys = 0;
        for (const Pre &t : tiles) keys += t.k1;
        // a tile is cut only when it is more than twice the mean keys per workgroup slot (else
        // the launch is bound by its total work, and pieces only add partial traffic), into
        // pieces of about that mean, at least kPrefillSplitKeys keys
        const long long mean = (keys + kAttnSlots - 1) / kAttnSlots;
        const long long target = std::max<long long>(kPrefillSplitKeys, mean);
        const bool may_split = emb.cfg.dtype == ORTHRUS_BF16;
        for (const Pre &t : tiles) {
            const int first_q = t.k1 - t.qn;                    // keys below it are seen by every row
            int n = may_split && t.k1 > 2 * mean
                        ? (int)std::min<long long>(kMaxPrefillSplits, (t.k1 + target - 1) / target)
                        : 1;
            std::vector<int> cuts{0};
            for (int k = 1; k < n; ++k) {
                const int c = std::min((int)((long long)k * t.k1 / n) / 64 * 64, first_q / 64 * 64);
                if (c > cuts.back()) cuts.push_back(c);
            }
            n = (int)cuts.size();
            if (n < 2 || n_pieces + n > kMaxPrefillPieces) {
                pre.push_back(t);
                continue;
            }
            cuts.push_back(t.k1);
            const int32_t *ch = &chunks[kChunkInts * t.chunk];
            merges.push_back({ch[4] + t.qb, t.qn, t.kvh, n, n_pieces});
            for (int k = 0; k < n; ++k)
                pre.push_back({(long long)(cuts[k + 1] - cuts[k]) * t.qn, t.chunk, t.kvh, t.qb, t.qn, cuts[k],
                               cuts[k + 1], n_pieces + k});
            n_pieces += n;
        }
        std::stable_sort(pre.begin(), pre.end(), [](const Pre &a, const Pre &b2) { return a.work > b2.work; });
    }
    // two distinct models: the embedding chunks' items and merge entries first (heaviest first
    // within each model), so each model's rows can be served by a launch of their own
    if (&emb != &gen) {
        const int n_emb_chunks = b.n_chunks;
        const auto emb_item = [n_emb_chunks](const Pre &t) { return t.chunk < n_emb_chunks; };
        p.n_pre_emb = (int)(std::stable_partition(pre.begin(), pre.end(), emb_item) - pre.begin());
        const int te = p.Te;
        p.n_merge_emb = (int)(std::stable_partition(merges.begin(), merges.end(),
                                                    [te](const Merge &m) { return m.tok < te; }) -
                              merges.begin());
    } else {
        p.n_pre_emb = (int)pre.size();
        p.n_merge_emb = (int)merges.size();
    }
    p.n_prefill = (int)pre.size();
    p.n_split_prefill = (int)merges.size();

    std::vector<int32_t> rows(kRowInts * p.D);
    // decode splits: whole chunks of kSplitPages pages, up to `cps` chunks per split, the
    // row's chunks dealt out evenly over its splits
    const int cps = gen.cfg.dtype == ORTHRUS_BF16 ? kDecodeChunksBf16 : 1;
    std::vector<std::array<int32_t, kItemInts>> dec;
    int partial = 0;
    for (int j = 0; j < p.D; ++j) {
        const orthrus_decode_row &r = b.rows[j];
        const int n_keys = r.ctx_len + 1;
        const int n_pages = (n_keys + P - 1) / P;
        const int n_chunk = (n_pages + kSplitPages - 1) / kSplitPages;
        const int n_splits = (n_chunk + cps - 1) / cps;
        rows[kRowInts * j + 0] = r.seq;
        rows[kRowInts * j + 1] = r.ctx_len;
        rows[kRowInts * j + 2] = p.Te + p.Tg + j;
        rows[kRowInts * j + 3] = n_splits;
        rows[kRowInts * j + 4] = n_splits > 1 ? partial : -1;
        if (n_splits > 1) p.n_split_rows++;
        for (int g = 0; g < nkv; ++g) {
            for (int s = 0; s < n_splits; ++s) {
                const int c0 = (int)((int64_t)s * n_chunk / n_splits);
                const int c1 = (int)((int64_t)(s + 1) * n_chunk / n_splits);
                std::array<int32_t, kItemInts> it{};
                it[IT_KIND] = 1;
                it[IT_INDEX] = j;
                it[IT_KVHEAD] = g;
                it[IT_A] = s;
                it[IT_B] = n_splits;
                it[IT_KEY_BEGIN] = c0 * kSplitPages * P;
                it[IT_KEY_END] = std::min(n_keys, c1 * kSplitPages * P);
                // partial slots: [first slot of row][kv head][split], each holding `group` heads
                it[IT_PARTIAL] = n_splits > 1 ? partial + g * n_splits + s : -1;
                dec.push_back(it);
            }
        }
        if (n_splits > 1) partial += nkv * n_splits;
    }
    // longest key ranges first, so the last round of the launch is short
    std::stable_sort(dec.begin(), dec.end(), [](const std::array<int32_t, kItemInts> &x,
                                                const std::array<int32_t, kItemInts> &y) {
        return x[IT_KEY_END] - x[IT_KEY_BEGIN] > y[IT_KEY_END] - y[IT_KEY_BEGIN];
    });
    // prefill pieces take partial slots after the decode rows': piece k of a split tile holds
    // its qrows tokens in consecutive slots, pieces of one tile qrows slots apart
    std::vector<int32_t> items(kItemInts * pre.size());
    std::vector<int32_t> combine(kCombineInts * merges.size());
    for (size_t k = 0; k < pre.size(); ++k) {
        int32_t *it = &items[kItemInts * k];
        it[IT_KIND] = 0;
        it[IT_INDEX] = pre[k].chunk;
        it[IT_KVHEAD] = pre[k].kvh;
        it[IT_A] = pre[k].qb;
        it[IT_B] = pre[k].qn;
        it[IT_KEY_BEGIN] = pre[k].k0;
        it[IT_KEY_END] = pre[k].k1;
        it[IT_PARTIAL] = pre[k].piece < 0 ? -1 : partial + pre[k].piece * qrows;
    }
    for (size_t i = 0; i < merges.size(); ++i) {
        int32_t *m = &combine[kCombineInts * i];
        m[0] = merges[i].tok;
        m[1] = merges[i].qn;
        m[2] = merges[i].kvh;
        m[3] = merges[i].n;
        m[4] = partial + merges[i].piece0 * qrows;
    }
    for (const auto &it : dec) items.insert(items.end(), it.begin(), it.end());
    p.n_decode_items = (int)(items.size() / kItemInts) - p.n_prefill;
    p.n_partials = partial + n_pieces * qrows;

    // --- pack
    p.off_tok = 0;
    p.off_pos = p.T;
    p.off_seq = 2 * p.T;
    p.off_chunks = 3 * p.T;
    p.off_rows = p.off_chunks + kChunkInts * n_all;
    p.off_items = p.off_rows + kRowInts * p.D;
    p.off_lm = p.off_items + (int)items.size();
    p.off_combine = p.off_lm + p.n_lm;
    p.off_split = p.off_combine + (int)combine.size();
    int end = p.off_split + p.n_split_rows;
    if (p.any_wmean) {
        p.off_wts = end;
        end += p.Te;
    }
    if (p.any_buffer) {
        p.off_hid = end;
        end += p.Te;
    }
    if (p.n_used > 0) {
        p.off_radp = end;
        end += p.Te;
    }
    p.meta.assign(end, 0);
    if (p.n_used > 0) {
        for (int i = 0, t = 0; i < b.n_chunks; t += b.chunks[i].len, ++i) {
            int slot = -1;
            for (int u = 0; u < p.n_used; ++u)
                if (p.used[u] == b.chunk_adapter[i]) slot = u;
            for (int k = 0; k < b.chunks[i].len; ++k) p.meta[p.off_radp + t + k] = slot;
        }
    }
    if (p.any_wmean) std::memcpy(&p.meta[p.off_wts], b.token_weights, (size_t)p.Te * 4);
    if (p.any_buffer) {
        for (int i = 0, t = 0; i < b.n_chunks; t += b.chunks[i].len, ++i) {
            const orthrus_emb_chunk &c = b.chunks[i];
            const bool buf = ((c.flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK) == ORTHRUS_POOL_BUFFER;
            for (int k = 0; k < c.len; ++k)
                p.meta[p.off_hid + t + k] = buf ? c.seq * b.hidden_stride + c.offset + k : -1;
        }
    }
    std::copy(b.token_ids, b.token_ids + p.T, p.meta.begin() + p.off_tok);
    int lm = 0;
    for (int i = 0; i < n_all; ++i) {
        const int32_t *ch = &chunks[kChunkInts * i];
        for (int k = 0; k < ch[2]; ++k) {
            p.meta[p.off_pos + ch[4] + k] = ch[1] + k;
            p.meta[p.off_seq + ch[4] + k] = ch[0];
        }
        if ((ch[3] & kChunkGen) && (ch[3] & ORTHRUS_CHUNK_LAST)) p.meta[p.off_lm + lm++] = ch[4] + ch[2] - 1;
    }
    for (int j = 0; j < p.D; ++j) {
        const int t = p.Te + p.Tg + j;
        p.meta[p.off_pos + t] = b.rows[j].ctx_len;
        p.meta[p.off_seq + t] = b.rows[j].seq;
        p.meta[p.off_lm + lm++] = t;
    }
    std::copy(chunks.begin(), chunks.end(), p.meta.begin() + p.off_chunks);
    std::copy(rows.begin(), rows.end(), p.meta.begin() + p.off_rows);
    std::copy(items.begin(), items.end(), p.meta.begin() + p.off_items);
    std::copy(combine.begin(), combine.end(), p.meta.begin() + p.off_combine);
    for (int j = 0, k = 0; j < p.D; ++j)
        if (rows[kRowInts * j + 3] > 1) p.meta[p.off_split + k++] = j;
    return ORTHRUS_OK;
}

}  // namespace orthrus
