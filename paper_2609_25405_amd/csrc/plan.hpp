// Host-side planning of one mixed step: descriptor validation, per-token metadata and the
// attention work list.  Plain C++17, no HIP calls, so it is exercised on machines without a GPU.
#pragma once

#include <cstdint>
#include <vector>

#include "orthrus.h"

namespace orthrus {

// Query-head rows per prefill work item; a work item covers (128 / group) tokens of one
// chunk times the `group` query heads that share one KV head.
constexpr int kPrefillRows = 128;
// Pages of one decode chunk (16 pages = 256 keys of a 16-token page): the unit a decode work
// item walks its key range in, and the whole split on the fp32 path.
constexpr int kSplitPages = 16;
// Chunks per decode split on the bf16 path (its items pipeline one chunk's loads under the
// previous chunk's arithmetic, so longer splits keep the memory pipe busier).
constexpr int kDecodeChunksBf16 = 4;
// Key splits of prefill items on the bf16 path.  A prefill item walks its keys one 32-key
// block after another, so an item over a long cached prefix can outlast the rest of the launch
// however many CUs are idle.  Items with more than twice the batch's mean prefill keys per
// workgroup slot (kAttnSlots = 256 CUs x two 256-thread workgroups) are cut into pieces of
// whole 64-key runs, about that mean long and at least kPrefillSplitKeys, at most
// kMaxPrefillSplits per item and kMaxPrefillPieces per step (their partials fit a fixed part of
// the workspace).
constexpr int kPrefillSplitKeys = 2048;
constexpr int kMaxPrefillSplits = 8;
constexpr int kMaxPrefillPieces = 1024;
constexpr int kAttnSlots = 512;
// int32 fields of one merge entry of a split prefill item: first token, tokens, kv head,
// pieces, first partial slot (piece k of row r: slot + k * (kPrefillRows / group) + r)
constexpr int kCombineInts = 5;

struct Model {
    orthrus_config cfg;
    orthrus_weights w;
    std::vector<orthrus_layer_weights> layers;
    // LoRA adapters chunks may name (orthrus_model_set_adapters); equal ranks for all of them
    std::vector<orthrus_lora> adapters;
    std::vector<std::vector<orthrus_lora_layer>> adapter_layers;
    int lora_rank[4] = {0, 0, 0, 0};
    int group() const { return cfg.n_q_heads / cfg.n_kv_heads; }
    int q_dim() const { return cfg.n_q_heads * cfg.head_dim; }
    int kv_dim() const { return cfg.n_kv_heads * cfg.head_dim; }
    int qkv_dim() const { return q_dim() + 2 * kv_dim(); }
};

// int32 fields of one attention work item
enum ItemField { IT_KIND = 0, IT_INDEX, IT_KVHEAD, IT_A, IT_B, IT_KEY_BEGIN, IT_KEY_END, IT_PARTIAL };
constexpr int kItemInts = 8;
constexpr int kChunkInts = 5;  // seq, offset, len, flags, first token
// chunk-table flag of a generation prefill chunk (reads and appends the generator's cache; the
// pooler skips it).  Caller flags use bits 0-2 only.
constexpr int kChunkGen = 1 << 8;
constexpr int kRowInts = 5;    // seq, ctx_len, token index, n_splits, first partial slot

// Token order of a step: [0, Te) embedding-chunk tokens, [Te, Te + Tg) generation prefill
// tokens, [Te + Tg, T) decode tokens.  The chunk table holds the n_chunks embedding chunks, then
// the n_gen generation chunks.
struct StepPlan {
    int T = 0, Te = 0, Tg = 0, D = 0, n_chunks = 0, n_gen = 0;
    bool shared_kv = true;
    int n_prefill = 0, n_decode_items = 0, n_partials = 0, n_split_rows = 0;
    int n_split_prefill = 0;  // prefill items cut along keys (merge entries at off_combine)
    // two distinct models: the first n_pre_emb prefill items and the first n_merge_emb merge
    // entries belong to embedding chunks (the embedding model's rows), the rest to generation
    // prefill chunks; each model's rows then get attention launches of their own
    int n_pre_emb = 0, n_merge_emb = 0;
    int n_lm = 0;  // rows that get logits: last rows of final prompt chunks, then decode rows
    // heads in the batch that need every embedding row's final norm (mean, weighted mean,
    // buffered), and the optional per-token arrays they read
    bool any_mean = false, any_wmean = false, any_buffer = false;
    // adapters the batch's embedding chunks name, in order of first use; per embedding token the
    // position of its adapter in that list or -1 (metadata at off_radp)
    int n_used = 0;
    int used[ORTHRUS_MAX_STEP_ADAPTERS] = {0, 0, 0, 0};
    int off_radp = -1;
    // packed metadata, uploaded verbatim: tok[T] pos[T] seq[T] chunks rows items lm_rows combine
    // split_rows (the n_split_rows decode rows with more than one split, in row order), then
    // (weighted mean) fp32 weights[Te] and (buffered head) hidden-buffer row[Te] (-1: none)
    std::vector<int32_t> meta;
    int off_tok = 0, off_pos = 0, off_seq = 0, off_chunks = 0, off_rows = 0, off_items = 0,
        off_lm = 0, off_combine = 0, off_split = 0, off_wts = -1, off_hid = -1;
};

int validate_config(const orthrus_config &c);
int plan_step(const Model &emb, const Model &gen, const orthrus_batch &b, const orthrus_kv &ekv,
              const orthrus_kv &gkv, StepPlan &out);
int max_splits_for_ctx(int max_ctx, int page_size);

}  // namespace orthrus
