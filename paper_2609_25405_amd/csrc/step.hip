// C ABI of the mixed step: model handles, workspace sizing, the per-step launch sequence (one
// iteration of the heterogeneous-batching loop, Algorithm 1, without scheduling; the forward is
// shared by all request types, Section 3.1; the pooler reads the embedding slice of the
// type-sorted batch, Section 3.2, and the LM head the rows that need next-token logits), and
// the greedy sampler.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "common.hpp"
#include "model.hpp"
#include "orthrus.h"
#include "plan.hpp"


namespace orthrus {
namespace {

constexpr size_t kAlign = 256;
size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Layout {
    size_t err, meta, x, act, qkv, q, o, u, inv_rms, partials, split_slabs, rope_cs, lora_u, total;
};
// split-K slabs of one residual-add projection: at most kMaxSplits fp32 [T][d] slabs
constexpr int kMaxSplits = 4;
// QKV projections of at most kQkvSplitRows rows per model, or of more than kQkvSplitMinRows and
// at most kQkvFusedMaxRows, split K in two (bf16 path): their fp32 partial sums [2][T][qkv_dim]
// get a region of qkv_slab_rows(T) rows, which the rotation/append kernel sums in split order.
// Measured on the 7B shape at 64 rows: the split projection and the rotation kernel take
// 18.6 + 6.9 us against 42.6 us fused (48 whole-head tiles); 8 splits 22.1 + 10.3 us; at 96
// rows 23.9 + 8.2 us against 44.0 us, at 128 rows 25.8 + 8.4 against 45.1 us; at 384 rows the
// fused projection is faster (54.5 us against 46.2 + 15.4 us with 4 splits).  At 1024 rows the
// split projection on 256x256 tiles (192 workgroups) takes 58 us against 79 us for the 128x128
// whole-head tiles before their fused epilogue (90 us with it in the two-model step)
constexpr int kQkvSplitRows = 128;
constexpr int kQkvSplitMinRows = 896;
constexpr int kQkvSplits = 2;
// QKV projections of more than kQkvFusedMaxRows rows per model (bf16 path) store fp32 rows
// from one round of 192x256 or 256x256 tiles and rotate them in the row kernel: whole-head
// 128x128 tiles with the fused epilogue need more than one round there (7B shape: 1568 rows
// 138 us fused against 86 + ~12 us; 2048 rows 173 us against 104 + ~15 us)
constexpr int kQkvFusedMaxRows = 1280;
size_t qkv_slab_rows(size_t T) { return (size_t)kQkvSplits * std::min<size_t>(T, 2 * kQkvFusedMaxRows); }
bool qkv_split_rows(int rows) { return rows <= kQkvSplitRows || (rows > kQkvSplitMinRows && rows <= kQkvFusedMaxRows); }

Layout make_layout(const Model &m, size_t T, size_t meta_ints, size_t n_partials) {
    const size_t es = m.cfg.dtype == ORTHRUS_BF16 ? 2 : 4;
    const size_t d = m.cfg.d_model;
    Layout L;
    size_t o = 0;
    L.err = o; o += kAlign;
    L.meta = o; o += up(meta_ints * 4);
    L.x = o; o += up(T * d * 4);
    L.act = o; o += up(T * d * es);
    // fp32 QKV rows for the separate rotation kernel: every row on the fp32 path; on the bf16
    // path (which rotates in the GEMM epilogue) the split-K partials of small projections
    L.qkv = o; o += up((m.cfg.dtype == ORTHRUS_BF16 ? std::max(T, qkv_slab_rows(T)) : T) * (size_t)m.qkv_dim() * 4);
    L.q = o; o += up(T * (size_t)m.q_dim() * es);
    L.o = o; o += up(T * (size_t)m.q_dim() * es);
    L.u = o; o += up(T * (size_t)m.cfg.d_ff * es);
    L.inv_rms = o; o += up(T * 4);
    L.partials = o; o += up(n_partials * (size_t)m.group() * (m.cfg.head_dim + 2) * 4);
    L.split_slabs = o; o += m.cfg.dtype == ORTHRUS_BF16 ? up((size_t)kMaxSplits * T * d * 4) : 0;
    L.rope_cs = o; o += m.cfg.dtype == ORTHRUS_BF16 ? up(T * (size_t)(m.cfg.head_dim / 2) * 8) : 0;
    // LoRA shrink output of one projection: [T][adapters in use x rank], the widest site
    const int max_rank = *std::max_element(m.lora_rank, m.lora_rank + 4);
    // (bf16 path: the rounding and its remainder, two arrays)
    L.lora_u = o; o += m.adapters.empty() ? 0 : up(T * (size_t)kMaxStepAdapters * max_rank * 4);
    L.total = o;
    return L;
}

bool same_shape(const orthrus_config &a, const orthrus_config &b) {
    return a.n_layers == b.n_layers && a.d_model == b.d_model && a.n_q_heads == b.n_q_heads &&
           a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim && a.d_ff == b.d_ff &&
           a.page_size == b.page_size && a.dtype == b.dtype && a.rope_base == b.rope_base &&
           a.rms_eps == b.rms_eps;
}

// a model without layers never reads or writes its cache: its pools may be NULL
bool kv_ok(const orthrus_kv *kv, const orthrus_model *m) {
    return kv && (m->cfg.n_layers == 0 || (kv->k_cache && kv->v_cache)) && kv->block_table && kv->n_pages > 0 &&
           kv->n_seq > 0 && kv->max_blocks > 0;
}

#define HIP_TRY(expr)                                   \
    do {                                                \
        if ((expr) != hipSuccess) return ORTHRUS_EHIP;  \
    } while (0)

// The step's metadata goes from pinned host memory to the workspace through this kernel on the
// step's stream, which reads the fine-grained host buffer itself.  An asynchronous host-to-device
// copy hands off to a copy engine and back: 30-50 us of idle GPU per step for a 6.8 us transfer
// of 64 KB, against a few microseconds here.
__global__ __launch_bounds__(256) void meta_upload_kernel(const int4 *src, int4 *dst, int n16) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n16; i += gridDim.x * 256) dst[i] = src[i];
}

int upload_meta(orthrus_model *m, const StepPlan &p, void *dst, hipStream_t s) {
    std::lock_guard<std::mutex> lk(m->mu);
    const int i = m->next;
    m->next ^= 1;
    const size_t bytes = p.meta.size() * 4;
    const size_t n16 = (bytes + 15) / 16;  // the destination region is rounded up to 256 bytes
    if (m->ev[i]) HIP_TRY(hipEventSynchronize(m->ev[i]));
    else HIP_TRY(hipEventCreateWithFlags(&m->ev[i], hipEventDisableTiming));
    if (m->stage_bytes[i] < n16 * 16) {
        if (m->stage[i]) m->retired.push_back(m->stage[i]);
        m->stage[i] = m->stage_dev[i] = nullptr;
        m->stage_bytes[i] = 0;
        void *h = nullptr;
        HIP_TRY(hipHostMalloc(&h, n16 * 32, hipHostMallocCoherent));
        m->stage[i] = h;
        m->stage_bytes[i] = n16 * 32;
        HIP_TRY(hipHostGetDevicePointer(&m->stage_dev[i], h, 0));
    }
    std::memcpy(m->stage[i], p.meta.data(), bytes);
    const int blocks = (int)std::min<size_t>((n16 + 255) / 256, 128);
    hipLaunchKernelGGL(meta_upload_kernel, dim3(blocks), dim3(256), 0, s, (const int4 *)m->stage_dev[i],
                       (int4 *)dst, (int)n16);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipEventRecord(m->ev[i], s));
    return ORTHRUS_OK;
}

// hipEvent pair around one launch when the model handle is profiling
struct Prof {
    orthrus_model *m;
    hipStream_t s;
    hipEvent_t a = nullptr;
    int id = -1;
    bool on() const { return m && m->profiling; }
    int begin(const std::string &name) {
        if (!on()) return ORTHRUS_OK;
        std::lock_guard<std::mutex> lk(m->mu);
        if (!m->prof_only.empty() && name != m->prof_only) {
            id = -2;   // not timed in this window
            return ORTHRUS_OK;
        }
        id = -1;
        for (size_t i = 0; i < m->prof_names.size(); ++i)
            if (m->prof_names[i] == name) id = (int)i;
        if (id < 0) {
            id = (int)m->prof_names.size();
            m->prof_names.push_back(name);
        }
        HIP_TRY(hipEventCreate(&a));
        HIP_TRY(hipEventRecord(a, s));
        return ORTHRUS_OK;
    }
    int end() {
        if (!on() || id == -2) return ORTHRUS_OK;
        hipEvent_t b = nullptr;
        HIP_TRY(hipEventCreate(&b));
        HIP_TRY(hipEventRecord(b, s));
        std::lock_guard<std::mutex> lk(m->mu);
        m->marks.push_back({id, a, b});
        return ORTHRUS_OK;
    }
};

size_t layer_stride(const Model &m, const orthrus_kv &kv) {
    const size_t es = m.cfg.dtype == ORTHRUS_BF16 ? 2 : 4;
    return (size_t)kv.n_pages * m.cfg.n_kv_heads * m.cfg.page_size * m.cfg.head_dim * es;
}

}  // namespace
}  // namespace orthrus

using namespace orthrus;

extern "C" {

const char *orthrus_strerror(int code) {
    switch (code) {
        case ORTHRUS_OK: return "ok";
        case ORTHRUS_EINVAL: return "invalid argument";
        case ORTHRUS_EDESC: return "malformed batch descriptor";
        case ORTHRUS_EDUPSEQ: return "sequence appears twice in one batch";
        case ORTHRUS_ECAPACITY: return "block table or workspace too small";
        case ORTHRUS_EUNSUPPORTED: return "unsupported shape or dtype";
        case ORTHRUS_EHIP: return "HIP runtime error";
        case ORTHRUS_EDEVICE: return "device-side check failed";
        default: return "unknown status";
    }
}

int orthrus_model_create(const orthrus_config *cfg, const orthrus_weights *w, orthrus_model **out) {
    if (!cfg || !w || !out) return ORTHRUS_EINVAL;
    *out = nullptr;
    const int rc = validate_config(*cfg);
    if (rc) return rc;
    if (!w->tok_emb || !w->final_norm || (cfg->n_layers > 0 && !w->layers)) return ORTHRUS_EINVAL;
    if (w->lm_head_blocked && !w->lm_head) return ORTHRUS_EINVAL;
    if (w->lm_head_blocked && cfg->dtype != ORTHRUS_BF16) return ORTHRUS_EUNSUPPORTED;
    for (int l = 0; l < cfg->n_layers; ++l) {
        const orthrus_layer_weights &lw = w->layers[l];
        if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.mlp_norm || !lw.w_gate || !lw.w_up || !lw.w_down)
            return ORTHRUS_EINVAL;
    }
    orthrus_model *m = new (std::nothrow) orthrus_model;
    if (!m) return ORTHRUS_EINVAL;
    m->cfg = *cfg;
    m->w = *w;
    m->layers.assign(w->layers, w->layers + cfg->n_layers);
    m->w.layers = m->layers.data();
    *out = m;
    return ORTHRUS_OK;
}

size_t orthrus_blocked_bytes(int32_t rows, int32_t cols) {
    if (rows <= 0 || cols <= 0 || cols % 64) return 0;
    return (size_t)((rows + 63) / 64) * 64 * (size_t)cols * 2;
}

int orthrus_block_weights(const void *src, void *dst, int32_t rows, int32_t cols, void *stream) {
    if (!src || !dst || orthrus_blocked_bytes(rows, cols) == 0) return ORTHRUS_EINVAL;
    return launch_block_weights(src, dst, rows, cols, (hipStream_t)stream) == hipSuccess ? ORTHRUS_OK
                                                                                          : ORTHRUS_EHIP;
}

int orthrus_model_set_adapters(orthrus_model *m, const orthrus_lora *adapters, int32_t n) {
    if (!m || n < 0 || (n > 0 && !adapters)) return ORTHRUS_EINVAL;
    for (int32_t i = 0; i < n; ++i) {
        const orthrus_lora &a = adapters[i];
        for (int k = 0; k < 4; ++k) {
            if (a.rank[k] != adapters[0].rank[k]) return ORTHRUS_EUNSUPPORTED;
            if (a.rank[k] < 0 || a.rank[k] > 256 || a.rank[k] % 16) return ORTHRUS_EUNSUPPORTED;
        }
        if (!(a.scale == a.scale) || (m->cfg.n_layers > 0 && !a.layers)) return ORTHRUS_EINVAL;
        for (int l = 0; l < m->cfg.n_layers; ++l) {
            const orthrus_lora_layer &ll = a.layers[l];
            if ((a.rank[0] && (!ll.qkv_a || !ll.qkv_b)) || (a.rank[1] && (!ll.o_a || !ll.o_b)) ||
                (a.rank[2] && (!ll.gate_up_a || !ll.gate_b || !ll.up_b)) ||
                (a.rank[3] && (!ll.down_a || !ll.down_b)))
                return ORTHRUS_EINVAL;
        }
    }
    std::lock_guard<std::mutex> lk(m->mu);
    m->adapters.assign(adapters, adapters + n);
    m->adapter_layers.clear();
    for (int32_t i = 0; i < n; ++i) {
        m->adapter_layers.emplace_back(adapters[i].layers, adapters[i].layers + m->cfg.n_layers);
        m->adapters[i].layers = m->adapter_layers.back().data();
    }
    for (int k = 0; k < 4; ++k) m->lora_rank[k] = n > 0 ? adapters[0].rank[k] : 0;
    return ORTHRUS_OK;
}

void orthrus_model_destroy(orthrus_model *m) {
    if (!m) return;
    for (int i = 0; i < 2; ++i) {
        if (m->ev[i]) {
            (void)hipEventSynchronize(m->ev[i]);
            (void)hipEventDestroy(m->ev[i]);
        }
        if (m->stage[i]) (void)hipHostFree(m->stage[i]);
    }
    for (void *r : m->retired) (void)hipHostFree(r);
    if (m->aux) {
        (void)hipStreamSynchronize(m->aux);
        (void)hipStreamDestroy(m->aux);
    }
    if (m->ev_fork) (void)hipEventDestroy(m->ev_fork);
    if (m->ev_join) (void)hipEventDestroy(m->ev_join);
    delete m;
}

size_t orthrus_workspace_bytes(const orthrus_model *emb, const orthrus_model *gen, int32_t max_tokens,
                               int32_t max_chunks, int32_t max_decode, int32_t max_ctx) {
    if (!emb || !gen || max_tokens < 0 || max_chunks < 0 || max_decode < 0 || max_ctx < 0) return 0;
    if (gen != emb && !same_shape(emb->cfg, gen->cfg)) return 0;
    const Model &m = *emb;
    const size_t nkv = m.cfg.n_kv_heads;
    const size_t qrows = kPrefillRows / m.group();
    const size_t splits = max_splits_for_ctx(max_ctx, m.cfg.page_size);
    const size_t pre_items = ((size_t)max_tokens / qrows + max_chunks) * nkv;
    const size_t dec_items = (size_t)max_decode * nkv * splits;
    // key-split prefill tiles (bf16): each piece adds at most one item and holds qrows partial
    // slots; a split tile has at least two pieces, so merge entries number at most pieces / 2
    const size_t pieces = m.cfg.dtype == ORTHRUS_BF16
                              ? std::min<size_t>(kMaxPrefillPieces, (size_t)kMaxPrefillSplits * pre_items)
                              : 0;
    const size_t meta = 3 * (size_t)max_tokens + kChunkInts * (size_t)max_chunks +
                        kRowInts * (size_t)max_decode + kItemInts * (pre_items + dec_items + pieces) +
                        kCombineInts * (pieces / 2) +
                        (size_t)max_chunks + max_decode +  // rows that get logits
                        max_decode +                       // decode rows with several splits
                        3 * (size_t)max_tokens;            // token weights, hidden-buffer rows,
                                                           // adapter positions
    return make_layout(m, max_tokens, meta, dec_items + pieces * qrows).total;
}

int orthrus_plan(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                 const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, int32_t *n_prefill_items,
                 int32_t *n_decode_items, int32_t *items, int32_t cap) {
    if (!emb || !gen || !batch || !kv_ok(emb_kv, emb) || !kv_ok(gen_kv, gen)) return ORTHRUS_EINVAL;
    if (gen != emb && !same_shape(emb->cfg, gen->cfg)) return ORTHRUS_EUNSUPPORTED;
    StepPlan p;
    const int rc = plan_step(*emb, *gen, *batch, *emb_kv, *gen_kv, p);
    if (rc) return rc;
    if (n_prefill_items) *n_prefill_items = p.n_prefill;
    if (n_decode_items) *n_decode_items = p.n_decode_items;
    if (items) {
        const int n = std::min<int>(cap, p.n_prefill + p.n_decode_items);
        std::memcpy(items, p.meta.data() + p.off_items, (size_t)n * kItemInts * 4);
    }
    return ORTHRUS_OK;
}

}  // extern "C"

namespace orthrus {
namespace {

// One step (the body of orthrus_step).  no_alloc (orthrus_step_noalloc): the metadata is copied
// with hipMemcpyAsync from host memory together with a zero error word, both row groups run on
// `stream` (no auxiliary stream, no events) and kernel timing is off, so nothing is allocated
// or created.
int step_impl(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
              const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, float *acc_sum, float *acc_w,
              float *out_logits, float *out_emb, void *workspace, size_t ws_bytes, void *stream, bool no_alloc) {
    if (!emb || !gen || !batch || !workspace || !kv_ok(emb_kv, emb) || !kv_ok(gen_kv, gen)) return ORTHRUS_EINVAL;
    if (gen != emb && !same_shape(emb->cfg, gen->cfg)) return ORTHRUS_EUNSUPPORTED;
    if (batch->n_chunks > 0 && (!acc_sum || !acc_w || !out_emb)) return ORTHRUS_EINVAL;
    if (batch->n_decode > 0 && !out_logits) return ORTHRUS_EINVAL;
    StepPlan p;
    int rc = plan_step(*emb, *gen, *batch, *emb_kv, *gen_kv, p);
    if (rc) return rc;
    if (p.n_lm > 0 && !out_logits) return ORTHRUS_EINVAL;
    if (p.T == 0) return ORTHRUS_OK;
    const Model &M = *emb;
    const orthrus_config &c = M.cfg;
    const Layout L = make_layout(M, p.T, p.meta.size(), p.n_partials);
    if (ws_bytes < L.total) return ORTHRUS_ECAPACITY;

    hipStream_t s = (hipStream_t)stream;
    Prof prof{no_alloc ? nullptr : const_cast<orthrus_model *>(emb), s};
    auto timed = [&](hipStream_t st, const std::string &name, auto &&launch) -> int {
        prof.s = st;
        int r = prof.begin(name);
        if (r) return r;
        if (launch() != hipSuccess) return ORTHRUS_EHIP;
        return prof.end();
    };
    // RUN: a launch on the step's stream; RUNG: a launch of row group g on the group's stream
#define RUN(name, expr)                                             \
    do {                                                            \
        const int r_ = timed(s, name, [&]() { return (expr); });    \
        if (r_) return r_;                                          \
    } while (0)
#define RUNG(g, name, expr)                                                                   \
    do {                                                                                      \
        const int r_ = timed((g).st, prof.on() ? std::string(name) + (g).tag : std::string(), \
                             [&]() { return (expr); });                                       \
        if (r_) return r_;                                                                    \
    } while (0)
    char *ws = (char *)workspace;
    int *err = (int *)(ws + L.err);
    const int32_t *meta = (const int32_t *)(ws + L.meta);
    if (no_alloc) {
        // [error word region (zeros) | metadata] in one copy: every call starts with no error bits
        static_assert(sizeof(int32_t) == 4, "int32 metadata");
        std::vector<int32_t> head(kAlign / 4 + p.meta.size(), 0);
        std::memcpy(head.data() + kAlign / 4, p.meta.data(), p.meta.size() * 4);
        if (L.meta != L.err + kAlign) return ORTHRUS_EHIP;
        HIP_TRY(hipMemcpyAsync(ws + L.err, head.data(), head.size() * 4, hipMemcpyHostToDevice, s));
    } else {
        rc = upload_meta(const_cast<orthrus_model *>(emb), p, ws + L.meta, s);
        if (rc) return rc;
    }

    const int dt = c.dtype;
    const size_t es = dt == ORTHRUS_BF16 ? 2 : 4;
    const int d = c.d_model, T = p.T, Te = p.Te;
    float *x = (float *)(ws + L.x);
    char *act = ws + L.act;
    float *qkv = (float *)(ws + L.qkv);
    char *qb = ws + L.q;
    char *ob = ws + L.o;
    char *ub = ws + L.u;
    const bool one_model = emb == gen;
    const int32_t *tok = meta + p.off_tok;

    // row groups: [0, Te) through the embedding model, [Te, T) (prompt chunks, then decode rows)
    // through the generator
    // (profiled launches of the generator's group carry the tag "@gen" in their names)
    struct Group { const orthrus_model *m; int r0, r1; hipStream_t st; const char *tag; };
    Group groups[2];
    int n_groups = 0;
    if (one_model) groups[n_groups++] = {emb, 0, T, s, ""};
    else {
        if (Te > 0) groups[n_groups++] = {emb, 0, Te, s, ""};
        if (T > Te) groups[n_groups++] = {gen, Te, T, s, "@gen"};
    }
    // Two row groups touch disjoint rows, weights and cache slots through every layer, so the
    // second group's launches run on the handle's auxiliary stream, concurrently with the
    // first's: forked after the plan upload, joined before the final norm (measured on the
    // two-model retrieval steps)
    orthrus_model *mh = const_cast<orthrus_model *>(emb);
    const bool concurrent = n_groups == 2 && !no_alloc;
    std::unique_lock<std::mutex> step_lock(mh->step_mu, std::defer_lock);
    if (concurrent) {
        step_lock.lock();
        if (!mh->aux) {
            HIP_TRY(hipStreamCreateWithFlags(&mh->aux, hipStreamNonBlocking));
            HIP_TRY(hipEventCreateWithFlags(&mh->ev_fork, hipEventDisableTiming));
            HIP_TRY(hipEventCreateWithFlags(&mh->ev_join, hipEventDisableTiming));
        }
        groups[1].st = mh->aux;
    }
    auto fork = [&]() -> int {
        if (!concurrent) return ORTHRUS_OK;
        HIP_TRY(hipEventRecord(mh->ev_fork, s));
        HIP_TRY(hipStreamWaitEvent(mh->aux, mh->ev_fork, 0));
        return ORTHRUS_OK;
    };
    auto join = [&]() -> int {
        if (!concurrent) return ORTHRUS_OK;
        HIP_TRY(hipEventRecord(mh->ev_join, mh->aux));
        HIP_TRY(hipStreamWaitEvent(s, mh->ev_join, 0));
        return ORTHRUS_OK;
    };
#define SYNC_GROUPS(call)            \
    do {                             \
        const int r_ = (call);       \
        if (r_) return r_;           \
    } while (0)

    // split-K slabs of the last residual-add projection, not yet added to x
    float *slabs = dt == ORTHRUS_BF16 ? (float *)(ws + L.split_slabs) : nullptr;
    float2 *rope_cs = dt == ORTHRUS_BF16 ? (float2 *)(ws + L.rope_cs) : nullptr;
    const size_t slab_stride = (size_t)T * d;
    int pending = 0;
    auto norm = [&](bool gather, const Group &g, const float *gain) -> hipError_t {
        NormArgs n{};
        n.pend = slabs ? slabs + (size_t)g.r0 * d : nullptr;
        n.pend_stride = slab_stride;
        n.npend = gather ? 0 : pending;
        n.x = x + (size_t)g.r0 * d;
        n.x_out = x + (size_t)g.r0 * d;
        n.table = g.m->w.tok_emb;
        n.tok = tok + g.r0;
        n.gain = gain;
        n.y = act + (size_t)g.r0 * d * es;
        n.rows = g.r1 - g.r0;
        n.d = d;
        n.eps = c.rms_eps;
        if (gather && rope_cs) {
            n.cs = rope_cs + (size_t)g.r0 * (c.head_dim / 2);
            n.pos = meta + p.off_pos + g.r0;
            n.hd = c.head_dim;
            n.rope_base = c.rope_base;
        }
        return launch_rmsnorm(dt, gather, n, g.st);
    };
    // LoRA: the shrink of site `site` (0 qkv, 1 o, 2 gate/up, 3 down) for the embedding rows of
    // group g in layer l, launched now on the GEMM input X; returns the GEMM's update arguments
    // (none when no chunk of the batch names an adapter or the site is not adapted)
    void *lora_u = ws + L.lora_u;
    auto lora_on = [&](int site, const Group &g) {
        return p.n_used > 0 && emb->lora_rank[site] > 0 && g.m == emb && g.r0 == 0 && Te > 0;
    };
    auto lora = [&](int site, int l, const Group &g, const char *X, int ldx, int K, LoraGemm &lg) -> hipError_t {
        lg = LoraGemm{};
        const int r = emb->lora_rank[site];
        if (!lora_on(site, g)) return hipSuccess;
        LoraShrink sh{};
        sh.x = X;
        sh.ldx = ldx;
        sh.K = K;
        sh.rows = Te;
        sh.r = r;
        sh.n = p.n_used;
        sh.row_adapter = meta + p.off_radp;
        sh.u = lora_u;
        lg.u = lora_u;
        if (dt == ORTHRUS_BF16) {
            // the remainder array follows the rounding array
            sh.u_lo = (char *)lora_u + (size_t)Te * p.n_used * r * 2;
            lg.u_lo = sh.u_lo;
        }
        lg.ldu = p.n_used * r;
        lg.rows = Te;
        lg.r = r;
        lg.n = p.n_used;
        for (int j = 0; j < p.n_used; ++j) {
            const orthrus_lora &ad = emb->adapters[p.used[j]];
            const orthrus_lora_layer &ll = emb->adapter_layers[p.used[j]][l];
            sh.scale[j] = ad.scale;
            const void *A = site == 0 ? ll.qkv_a : site == 1 ? ll.o_a : site == 2 ? ll.gate_up_a : ll.down_a;
            sh.a[j] = A;
            lg.b0[j] = site == 0 ? ll.qkv_b : site == 1 ? ll.o_b : site == 2 ? ll.gate_b : ll.down_b;
            lg.b1[j] = site == 2 ? ll.up_b : nullptr;
        }
        return launch_lora_shrink(dt, sh, g.st);
    };
    auto gemm = [&](int epi, const Group &g, const char *A, int lda, const void *B0, const void *B1,
                    void *out, int ldo, size_t out_es, int N, int K, const LoraGemm &lg) -> hipError_t {
        GemmArgs ga{};
        ga.A = A + (size_t)g.r0 * lda * es;
        ga.B0 = B0;
        ga.B1 = B1;
        ga.out = (char *)out + (size_t)g.r0 * ldo * out_es;
        ga.M = g.r1 - g.r0;
        ga.N = N;
        ga.K = K;
        ga.lda = lda;
        ga.ldo = ldo;
        ga.splits = 1;
        ga.lora = lg;
        return launch_gemm(dt, epi, ga, g.st);
    };
    // residual-add projection into x; bf16: split K when the tile count is low and leave the
    // slabs for the next row-wise kernel.  `splits` is chosen once per projection for the largest
    // row group and used by every group, so the pending slab count is the same for all rows.
    int max_rows = 0;
    for (int gi = 0; gi < n_groups; ++gi) max_rows = std::max(max_rows, groups[gi].r1 - groups[gi].r0);
    auto add_splits = [&](int K) { return slabs ? gemm_add_splits(max_rows, d, K, kMaxSplits) : 1; };
    auto add_proj = [&](const Group &g, const char *A, int lda, const void *B, int K, int splits,
                        const LoraGemm &lg) -> hipError_t {
        GemmArgs ga{};
        ga.A = A + (size_t)g.r0 * lda * es;
        ga.B0 = B;
        ga.out = x + (size_t)g.r0 * d;
        ga.M = g.r1 - g.r0;
        ga.N = d;
        ga.K = K;
        ga.lda = lda;
        ga.ldo = d;
        ga.splits = splits;
        ga.partial = slabs ? slabs + (size_t)g.r0 * d : nullptr;  // the group's rows of each slab
        ga.split_stride = slab_stride;
        ga.lora = lg;
        ga.wide = concurrent;
        return launch_gemm(dt, EPI_ADD_F32, ga, g.st);
    };

    // token gather fused with the first RMSNorm (the final norm when there are no layers)
    SYNC_GROUPS(fork());
    for (int gi = 0; gi < n_groups; ++gi) {
        const Group &g = groups[gi];
        const float *gain = c.n_layers > 0 ? g.m->layers[0].attn_norm : g.m->w.final_norm;
        RUNG(g, "gather_norm", norm(true, g, gain));
    }

    AttnArgs aa{};
    aa.q = qb;
    aa.o = ob;
    aa.chunks = meta + p.off_chunks;
    aa.rows = meta + p.off_rows;
    aa.items = meta + p.off_items;
    aa.combine = meta + p.off_combine;
    aa.split_rows = meta + p.off_split;
    aa.n_combine = p.n_split_prefill;
    aa.partials = (float *)(ws + L.partials);
    aa.n_prefill = p.n_prefill;
    aa.n_items = p.n_prefill + p.n_decode_items;
    aa.Te = Te;
    aa.nq = c.n_q_heads;
    aa.nkv = c.n_kv_heads;
    aa.hd = c.head_dim;
    aa.page = c.page_size;
    aa.err = err;
    aa.block_table[0] = emb_kv->block_table;
    aa.block_table[1] = gen_kv->block_table;
    aa.n_pages[0] = emb_kv->n_pages;
    aa.n_pages[1] = gen_kv->n_pages;
    aa.max_blocks[0] = emb_kv->max_blocks;
    aa.max_blocks[1] = gen_kv->max_blocks;

    RopeArgs ra{};
    ra.qkv = qkv;
    ra.nslab = 1;
    ra.cs = rope_cs;
    ra.q_out = qb;
    ra.pos = meta + p.off_pos;
    ra.seq = meta + p.off_seq;
    ra.Te = Te;
    ra.T = T;
    ra.nq = c.n_q_heads;
    ra.nkv = c.n_kv_heads;
    ra.hd = c.head_dim;
    ra.page = c.page_size;
    ra.rope_base = c.rope_base;
    ra.err = err;
    for (int i = 0; i < 2; ++i) {
        ra.block_table[i] = aa.block_table[i];
        ra.n_pages[i] = aa.n_pages[i];
        ra.max_blocks[i] = aa.max_blocks[i];
    }
    const size_t e_stride = layer_stride(M, *emb_kv), g_stride = layer_stride(M, *gen_kv);
    const int qd = M.q_dim(), qkvd = M.qkv_dim(), F = c.d_ff;
    // Two row groups (two models) never share a row, a work item or a cache slot: each group's
    // rotation/append, attention and merge run on the group's stream over its own rows, the
    // planner's items of its chunks (and, for the generator, the decode rows) and its merge
    // entries, so the groups' layer chains proceed independently
    auto rope_group = [&](const Group &g) -> hipError_t {
        RopeArgs r = ra;
        r.qkv = ra.qkv + (size_t)g.r0 * qkvd;
        r.cs = ra.cs ? ra.cs + (size_t)g.r0 * (c.head_dim / 2) : nullptr;
        r.q_out = qb + (size_t)g.r0 * qd * es;
        r.pos = ra.pos + g.r0;
        r.seq = ra.seq + g.r0;
        r.T = g.r1 - g.r0;
        r.Te = std::max(0, std::min(Te - g.r0, r.T));
        return launch_rope_append(dt, r, g.st);
    };
    const int merges_gen = p.n_split_prefill - p.n_merge_emb;
    auto attn_group = [&](int gi, bool combine) -> hipError_t {
        AttnArgs ag = aa;
        int n_dec = 0;
        if (gi == 0) {
            ag.n_prefill = p.n_pre_emb;
            ag.n_items = p.n_pre_emb;
            ag.n_combine = p.n_merge_emb;
        } else {
            ag.items = aa.items + kItemInts * p.n_pre_emb;
            ag.n_prefill = p.n_prefill - p.n_pre_emb;
            ag.n_items = aa.n_items - p.n_pre_emb;
            ag.combine = aa.combine + kCombineInts * p.n_merge_emb;
            ag.n_combine = merges_gen;
            n_dec = p.n_split_rows;
        }
        return combine ? launch_attn_combine(dt, ag, n_dec, groups[gi].st) : launch_attention(dt, ag, groups[gi].st);
    };

    for (int l = 0; l < c.n_layers; ++l) {
        if (l > 0) {
            for (int gi = 0; gi < n_groups; ++gi)
                RUNG(groups[gi], "rmsnorm", norm(false, groups[gi], groups[gi].m->layers[l].attn_norm));
            pending = 0;
        }
        ra.k_cache[0] = (char *)emb_kv->k_cache + l * e_stride;
        ra.v_cache[0] = (char *)emb_kv->v_cache + l * e_stride;
        ra.k_cache[1] = (char *)gen_kv->k_cache + l * g_stride;
        ra.v_cache[1] = (char *)gen_kv->v_cache + l * g_stride;
        // small bf16 projections (decode-only batches) stream their weights, and whole-head tiles
        // for the fused rotation leave too few workgroups (48 at 64 rows): they split K into fp32
        // partials, which the rotation/append row kernel sums in split order
        const int qkv_splits = dt == ORTHRUS_BF16 && qkv_split_rows(max_rows) && d % (kQkvSplits * 64) == 0 &&
                                       d / kQkvSplits >= 512 && (size_t)kQkvSplits * T <= qkv_slab_rows(T)
                                   ? kQkvSplits
                                   : 1;
        if (qkv_splits > 1) {
            for (int gi = 0; gi < n_groups; ++gi) {
                const Group &g = groups[gi];
                GemmArgs ga{};
                ga.A = act + (size_t)g.r0 * d * es;
                ga.B0 = g.m->layers[l].w_qkv;
                ga.out = qkv + (size_t)g.r0 * qkvd;
                ga.M = g.r1 - g.r0;
                ga.N = qkvd;
                ga.K = d;
                ga.lda = d;
                ga.ldo = qkvd;
                ga.splits = qkv_splits;
                ga.partial = qkv + (size_t)g.r0 * qkvd;
                ga.split_stride = (size_t)T * qkvd;
                ga.wide = concurrent;
                if (lora_on(0, g)) RUNG(g, "lora_shrink", lora(0, l, g, act, d, d, ga.lora));
                RUNG(g, "gemm_qkv", launch_gemm(dt, EPI_ADD_F32, ga, g.st));
            }
            ra.nslab = qkv_splits;
            ra.slab_stride = (size_t)T * qkvd;
            if (n_groups == 2) {
                for (int gi = 0; gi < n_groups; ++gi) RUNG(groups[gi], "rope_append", rope_group(groups[gi]));
            } else {
                RUN("rope_append", launch_rope_append(dt, ra, s));
            }
        } else if (dt == ORTHRUS_BF16 && max_rows <= kQkvFusedMaxRows) {
            // QKV projection with rotation and cache append in its epilogue
            for (int gi = 0; gi < n_groups; ++gi) {
                const Group &g = groups[gi];
                GemmArgs ga{};
                ga.A = act + (size_t)g.r0 * d * es;
                ga.B0 = g.m->layers[l].w_qkv;
                ga.M = g.r1 - g.r0;
                ga.N = qkvd;
                ga.K = d;
                ga.lda = d;
                ga.splits = 1;
                QkvRope &q = ga.rope;
                q.cs = rope_cs;
                q.pos = ra.pos;
                q.seq = ra.seq;
                q.q_out = qb;
                for (int i = 0; i < 2; ++i) {
                    q.k_cache[i] = ra.k_cache[i];
                    q.v_cache[i] = ra.v_cache[i];
                    q.block_table[i] = ra.block_table[i];
                    q.n_pages[i] = ra.n_pages[i];
                    q.max_blocks[i] = ra.max_blocks[i];
                }
                q.row0 = g.r0;
                q.Te = Te;
                q.nq = c.n_q_heads;
                q.nkv = c.n_kv_heads;
                q.hd = c.head_dim;
                q.page = c.page_size;
                q.err = err;
                if (lora_on(0, g)) RUNG(g, "lora_shrink", lora(0, l, g, act, d, d, ga.lora));
                RUNG(g, "gemm_qkv_rope", launch_gemm(dt, EPI_QKV_ROPE, ga, g.st));
            }
        } else {
            for (int gi = 0; gi < n_groups; ++gi) {
                const orthrus_layer_weights &lw = groups[gi].m->layers[l];
                LoraGemm lg{};
                if (lora_on(0, groups[gi])) RUNG(groups[gi], "lora_shrink", lora(0, l, groups[gi], act, d, d, lg));
                RUNG(groups[gi], "gemm_qkv", gemm(EPI_STORE_F32, groups[gi], act, d, lw.w_qkv, nullptr, qkv, qkvd, 4, qkvd, d, lg));
            }
            ra.nslab = 1;
            if (n_groups == 2) {
                for (int gi = 0; gi < n_groups; ++gi) RUNG(groups[gi], "rope_append", rope_group(groups[gi]));
            } else {
                RUN("rope_append", launch_rope_append(dt, ra, s));
            }
        }
        for (int i = 0; i < 2; ++i) {
            aa.k_cache[i] = ra.k_cache[i];
            aa.v_cache[i] = ra.v_cache[i];
        }
        if (n_groups == 2) {
            RUNG(groups[0], "attention", attn_group(0, false));
            if (p.n_merge_emb > 0) RUNG(groups[0], "attn_combine", attn_group(0, true));
            RUNG(groups[1], "attention", attn_group(1, false));
            if (p.n_split_rows > 0 || merges_gen > 0) RUNG(groups[1], "attn_combine", attn_group(1, true));
        } else {
            RUN("attention", launch_attention(dt, aa, s));
            if (p.n_split_rows > 0 || p.n_split_prefill > 0)
                RUN("attn_combine", launch_attn_combine(dt, aa, p.n_split_rows, s));
        }
        int splits = add_splits(qd);
        for (int gi = 0; gi < n_groups; ++gi) {
            const orthrus_layer_weights &lw = groups[gi].m->layers[l];
            LoraGemm lg{};
            if (lora_on(1, groups[gi])) RUNG(groups[gi], "lora_shrink", lora(1, l, groups[gi], ob, qd, qd, lg));
            RUNG(groups[gi], "gemm_o", add_proj(groups[gi], ob, qd, lw.w_o, qd, splits, lg));
        }
        pending = splits > 1 ? splits : 0;
        for (int gi = 0; gi < n_groups; ++gi)
            RUNG(groups[gi], "rmsnorm", norm(false, groups[gi], groups[gi].m->layers[l].mlp_norm));
        pending = 0;
        for (int gi = 0; gi < n_groups; ++gi) {
            const orthrus_layer_weights &lw = groups[gi].m->layers[l];
            LoraGemm lg{};
            if (lora_on(2, groups[gi])) RUNG(groups[gi], "lora_shrink", lora(2, l, groups[gi], act, d, d, lg));
            RUNG(groups[gi], "gemm_gate_up", gemm(EPI_SWIGLU, groups[gi], act, d, lw.w_gate, lw.w_up, ub, F, es, F, d, lg));
        }
        splits = add_splits(F);
        for (int gi = 0; gi < n_groups; ++gi) {
            const orthrus_layer_weights &lw = groups[gi].m->layers[l];
            LoraGemm lg{};
            if (lora_on(3, groups[gi])) RUNG(groups[gi], "lora_shrink", lora(3, l, groups[gi], ub, F, F, lg));
            RUNG(groups[gi], "gemm_down", add_proj(groups[gi], ub, F, lw.w_down, F, splits, lg));
        }
        pending = splits > 1 ? splits : 0;  // added by the next layer's norm or the final norm
    }

    SYNC_GROUPS(join());
    // final RMSNorm (scale of the embedding rows; LM-head input of the rows that get logits),
    // then the incremental pooler on the embedding slice and the LM head on the listed rows
    PoolArgs pa{};
    pa.x = x;
    pa.gain = emb->w.final_norm;
    pa.gen_gain = gen->w.final_norm;
    pa.act = act;  // free after the last layer: the LM-head input goes to its first n_lm rows
    pa.lm_rows = meta + p.off_lm;
    pa.chunks = meta + p.off_chunks;
    pa.inv_rms = (float *)(ws + L.inv_rms);
    pa.acc_sum = acc_sum;
    pa.acc_w = acc_w;
    pa.out_emb = out_emb;
    pa.n_chunks = p.n_chunks;
    pa.pend = slabs;
    pa.pend_stride = slab_stride;
    pa.npend = pending;
    pa.Te = Te;
    pa.d = d;
    pa.eps = c.rms_eps;
    pa.err = err;
    // Mean, weighted-mean and buffered heads need the final norm of every embedding row;
    // single-row heads normalise their one row inside the pooler.
    const bool any_rows = p.any_mean || p.any_wmean || p.any_buffer;
    pa.weights = p.any_wmean ? (const float *)(meta + p.off_wts) : nullptr;
    pa.hid_rows = p.any_buffer ? meta + p.off_hid : nullptr;
    pa.hidden = batch->hidden;
    pa.n_emb_rows = any_rows ? Te : 0;
    pa.n_lm = p.n_lm;
    if (!any_rows && p.n_chunks > 0 && p.n_lm > 0) {
        // independent work: LM rows' final norm and the single-row pooler in one launch
        RUN("final_norm_pool", launch_final_and_pool(dt, pa, s));
    } else {
        if (pa.n_emb_rows + pa.n_lm > 0) RUN("final_norm", launch_final_rows(dt, pa, s));
        // the embedding rows' pending slabs were added by the final norm when it covered them
        if (any_rows) pa.npend = 0;
        if (p.n_chunks > 0) RUN("pool", launch_pool(pa, any_rows, s));
    }
    if (p.n_lm > 0) {
        GemmArgs ga{};
        ga.A = act;
        ga.B0 = gen->w.lm_head_blocked ? gen->w.lm_head_blocked : gen->w.lm_head;
        ga.b_blocked = gen->w.lm_head_blocked != nullptr;
        ga.out = out_logits;
        ga.M = p.n_lm;
        ga.N = gen->cfg.vocab;
        ga.K = d;
        ga.lda = d;
        ga.ldo = gen->cfg.vocab;
        ga.splits = 1;
        RUN("lm_head", launch_gemm(dt, EPI_STORE_F32, ga, s));
    }
    return ORTHRUS_OK;
#undef RUN
#undef RUNG
#undef SYNC_GROUPS
}

// Scratch of orthrus_step_noalloc: a file-scope device array, one per device (zero at load).  In
// host code `scratch` names a host-side stand-in; its device address comes from
// hipGetSymbolAddress, taken once per device with that device current and kept in scratch_dev.
constexpr size_t kScratchBytes = ORTHRUS_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_dev[kMaxDevices] = {};

// the current device's scratch address, or nullptr on a HIP failure
void *scratch_address() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(scratch_mu);
    if (!scratch_dev[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        scratch_dev[dev] = ptr;
    }
    return scratch_dev[dev];
}

// hands the step's error bits to the caller's word and clears the scratch copy
__global__ void error_out_kernel(int *err, int *out) {
    if (threadIdx.x == 0) {
        if (out) out[0] = err[0];
        err[0] = 0;
    }
}

}  // namespace
}  // namespace orthrus

extern "C" {

int orthrus_step(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                 const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, float *acc_sum, float *acc_w,
                 float *out_logits, float *out_emb, void *workspace, size_t ws_bytes, void *stream) {
    return step_impl(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits, out_emb, workspace, ws_bytes,
                     stream, false);
}

int orthrus_step_noalloc(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                         const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, float *acc_sum, float *acc_w,
                         float *out_logits, float *out_emb, int32_t *device_error, void *stream) {
    if (!emb || !gen || !batch) return ORTHRUS_EINVAL;
    void *ws = scratch_address();
    if (!ws) return ORTHRUS_EHIP;
    const int rc = step_impl(emb, gen, batch, emb_kv, gen_kv, acc_sum, acc_w, out_logits, out_emb, ws,
                             kScratchBytes, stream, true);
    if (rc) return rc;
    hipLaunchKernelGGL(error_out_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, (int *)ws, (int *)device_error);
    return hipGetLastError() == hipSuccess ? ORTHRUS_OK : ORTHRUS_EHIP;
}

int orthrus_profile_begin(orthrus_model *m) {
    if (!m) return ORTHRUS_EINVAL;
    std::lock_guard<std::mutex> lk(m->mu);
    m->profiling = true;
    return ORTHRUS_OK;
}

int orthrus_profile_only(orthrus_model *m, const char *name) {
    if (!m) return ORTHRUS_EINVAL;
    std::lock_guard<std::mutex> lk(m->mu);
    m->prof_only = name ? name : "";
    return ORTHRUS_OK;
}

int orthrus_profile_end(orthrus_model *m, orthrus_kernel_time *out, int32_t cap, int32_t *n_out) {
    if (!m) return ORTHRUS_EINVAL;
    std::lock_guard<std::mutex> lk(m->mu);
    m->profiling = false;
    std::vector<double> ms(m->prof_names.size(), 0.0);
    std::vector<int> cnt(m->prof_names.size(), 0);
    int rc = ORTHRUS_OK;
    for (const auto &mk : m->marks) {
        float t = 0.f;
        if (hipEventSynchronize(mk.b) != hipSuccess || hipEventElapsedTime(&t, mk.a, mk.b) != hipSuccess)
            rc = ORTHRUS_EHIP;
        ms[mk.name] += t;
        cnt[mk.name] += 1;
        (void)hipEventDestroy(mk.a);
        (void)hipEventDestroy(mk.b);
    }
    m->marks.clear();
    const int n = (int)m->prof_names.size();
    if (n_out) *n_out = n;
    for (int i = 0; i < n && out && i < cap; ++i) {
        std::memset(out[i].name, 0, sizeof(out[i].name));
        std::strncpy(out[i].name, m->prof_names[i].c_str(), sizeof(out[i].name) - 1);
        out[i].launches = cnt[i];
        out[i].total_ms = ms[i];
    }
    m->prof_names.clear();
    return rc;
}

int orthrus_sample_greedy(const float *logits, int32_t rows, int32_t vocab, int32_t *out_tokens,
                          void *stream) {
    if (rows < 0 || vocab < 1) return ORTHRUS_EINVAL;
    if (rows == 0) return ORTHRUS_OK;
    if (!logits || !out_tokens) return ORTHRUS_EINVAL;
    if (launch_argmax(logits, rows, vocab, out_tokens, (hipStream_t)stream) != hipSuccess) return ORTHRUS_EHIP;
    return ORTHRUS_OK;
}

int orthrus_workspace_init(void *workspace, void *stream) {
    if (!workspace) return ORTHRUS_EINVAL;
    HIP_TRY(hipMemsetAsync(workspace, 0, kAlign, (hipStream_t)stream));
    return ORTHRUS_OK;
}

int orthrus_device_error(void *workspace, void *stream, int32_t *bits) {
    if (!workspace) return ORTHRUS_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    int32_t v = 0, zero = 0;
    HIP_TRY(hipStreamSynchronize(s));
    HIP_TRY(hipMemcpy(&v, workspace, 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(workspace, &zero, 4, hipMemcpyHostToDevice));
    if (bits) *bits = v;
    return v ? ORTHRUS_EDEVICE : ORTHRUS_OK;
}

}  // extern "C"
