/*
 * orthrus.h -- C ABI of the mixed embedding + generation step on one MI355X (gfx950).
 *
 * One call of orthrus_step() is the body of the heterogeneous-batching inference loop
 * (Algorithm 1) minus scheduling and sampling: a single forward pass over a type-sorted
 * batch holding embedding chunks, generation prefill chunks and generation decode tokens
 * (Section 3.2, "Batch Unit"), followed by the incremental pooler on the embedding slice
 * (Section 3.3, Eq. (1)-(2) and the positional heads) and the LM head on the rows that need
 * next-token logits.  orthrus_sample_greedy() is the sampler on those logits.  Every
 * request type shares the same attention and feed-forward layers (Section 3.1).
 *
 * Model family: pre-norm decoder with RMSNorm, rotary position embedding (half-split
 * pairs, angle = pos * base^(-2i/head_dim)), grouped-query attention (query head h reads
 * KV head h / (n_q_heads / n_kv_heads)), SwiGLU MLP, untied LM head.
 *
 * Conventions shared by every entry point:
 *   - All "device" pointers are HIP device memory on the current device; all "host"
 *     pointers are ordinary host memory.  The caller owns every buffer; the library
 *     never frees caller memory.  orthrus_step() allocates no device memory.
 *   - Matrices are row-major.  Weight matrices are [out_features][in_features].
 *   - dtype ORTHRUS_BF16: weights, KV cache, GEMM inputs in bfloat16; accumulation,
 *     softmax, norm statistics and the residual stream in fp32; logits, pooling state
 *     and embeddings in fp32.  dtype ORTHRUS_F32: everything fp32.
 *   - Return value: ORTHRUS_OK (0) or a negative ORTHRUS_E* code.  On a nonzero return
 *     nothing has been enqueued and no caller buffer has been touched.
 */
#ifndef ORTHRUS_H
#define ORTHRUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define ORTHRUS_OK 0
#define ORTHRUS_EINVAL (-1)       /* null pointer, negative count, malformed config   */
#define ORTHRUS_EDESC (-2)        /* bad seq / offset / len / ctx_len / flags / token */
#define ORTHRUS_EDUPSEQ (-3)      /* a sequence appears twice in one batch             */
#define ORTHRUS_ECAPACITY (-4)    /* block table or workspace too small for the batch  */
#define ORTHRUS_EUNSUPPORTED (-5) /* shape or dtype without a kernel instantiation     */
#define ORTHRUS_EHIP (-6)         /* a HIP runtime call failed                         */
#define ORTHRUS_EDEVICE (-7)      /* a kernel flagged bad device-side state            */

/* element types */
#define ORTHRUS_F32 0
#define ORTHRUS_BF16 1

/* orthrus_emb_chunk.flags: bit 0 = final chunk of its request; bits 1-3 = pooling head.  Every
 * pooled head (all but NONE) adds len to the request's W, which counts tokens (offset check). */
#define ORTHRUS_CHUNK_LAST 1
#define ORTHRUS_POOL_SHIFT 1
#define ORTHRUS_POOL_MASK 7
#define ORTHRUS_POOL_MEAN 0   /* S += sum of rows; emits S / W (Eq. (1)-(2), w = 1)           */
#define ORTHRUS_POOL_LAST 1   /* keeps the last row of the final chunk                        */
#define ORTHRUS_POOL_CLS 2    /* keeps the first row of the offset-0 chunk                    */
#define ORTHRUS_POOL_NONE 3   /* writes keys/values only (cache-filling prefill chunk)        */
#define ORTHRUS_POOL_WMEAN 4  /* S += sum of w_j * row_j with the batch's token_weights       */
                              /* (Eq. (1)-(2)); emits S, L2-normalised (the weight sum W of   */
                              /* Eq. (2) cancels in the L2 finish, so it is never formed)     */
#define ORTHRUS_POOL_BUFFER 5 /* writes the final-normed rows to the batch's hidden buffer    */
                              /* (the buffered arbitrary head); emits no embedding            */

/* device error bits reported by orthrus_device_error() */
#define ORTHRUS_DEVERR_PAGE 1 /* block-table entry outside [0, n_pages) on a used block     */
#define ORTHRUS_DEVERR_ACC 2  /* chunk offset > 0 but the request's W differs from offset */

/* Model shape.  Supported: head_dim 64 or 128; n_q_heads a multiple of n_kv_heads with
 * group size 1, 2 or 4; d_model and d_ff multiples of 256 (bf16) or 64 (f32); page_size 16. */
typedef struct orthrus_config {
    int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab, page_size;
    float rope_base, rms_eps;
    int32_t dtype; /* ORTHRUS_F32 or ORTHRUS_BF16 */
} orthrus_config;

/* Per-layer weights (device).  w_qkv: [(nq + 2 nkv) * hd][d] with the query heads, then the
 * key heads, then the value heads, each head hd contiguous rows.  w_o: [d][nq * hd].
 * w_gate, w_up: [d_ff][d].  w_down: [d][d_ff].  Norm gains are fp32 [d]. */
typedef struct orthrus_layer_weights {
    const float *attn_norm;
    const void *w_qkv;
    const void *w_o;
    const float *mlp_norm;
    const void *w_gate;
    const void *w_up;
    const void *w_down;
} orthrus_layer_weights;

/* Model weights.  tok_emb [vocab][d] and lm_head [vocab][d] (may be NULL for an embedding-only
 * model) are device memory of the model dtype; final_norm is fp32 [d] device memory.  `layers`
 * is a HOST array of n_layers entries, copied by orthrus_model_create().  lm_head_blocked
 * (optional, bf16 models only, else NULL): the same LM head in the 64 x 64 blocked layout
 * orthrus_block_weights() writes; when set, the LM head GEMM reads it instead of lm_head, which
 * must still be given (it marks the model as having an LM head). */
typedef struct orthrus_weights {
    const void *tok_emb;
    const float *final_norm;
    const void *lm_head;
    const orthrus_layer_weights *layers;
    const void *lm_head_blocked;
} orthrus_weights;

/* Weight layout helpers for the LM head that turns the decode rows' hidden states into logits
 * (the generation side of Algorithm 1's forward pass); a memory layout only, no arithmetic.
 * Bytes of the blocked copy of a bf16 [rows][cols] weight matrix: ceil(rows / 64) * 64 * cols * 2
 * (0 unless rows > 0 and cols is a positive multiple of 64). */
size_t orthrus_blocked_bytes(int32_t rows, int32_t cols);

/* Write the blocked copy of the bf16 row-major matrix src [rows][cols] (device) into dst (device,
 * orthrus_blocked_bytes() bytes, caller-owned): blocks of 64 rows x 64 columns, row blocks
 * outermost, each block's 64 rows of 64 values contiguous (8 KB), so the copy of one 64-deep
 * stage of a weight-streaming GEMM tile reads whole 8 KB runs; rows past `rows` in the last
 * block are zero.  Enqueued on `stream`.  EINVAL for null pointers or sizes orthrus_blocked_bytes
 * rejects. */
int orthrus_block_weights(const void *src, void *dst, int32_t rows, int32_t cols, void *stream);

typedef struct orthrus_model orthrus_model; /* opaque host-side handle */

/* LoRA adapter of an embedding model (Section 2, parameter sharing: embedding models derived from
 * generative ones by LoRA; the paper deploys Mistral-7B with the e5-mistral adapter, ranks up to
 * 64).  Per layer and adapted projection, A [rank][in] and B [out][rank] in the model dtype
 * (device); the projection computes x W^T + scale * (x A^T) B^T for the rows of every chunk that
 * names the adapter.  Sites: qkv (A [r_qkv][d], B [(nq + 2 nkv) hd][r_qkv]), o (A [r_o][nq hd],
 * B [d][r_o]), gate/up (one A [r_gu][d] shared, B_gate and B_up [d_ff][r_gu]), down
 * (A [r_down][d_ff], B [d][r_down]).  Separate q, k and v adapters are one qkv site with the three
 * A stacked and a block-diagonal B; separate gate and up adapters stack their A the same way. */
typedef struct orthrus_lora_layer {
    const void *qkv_a, *qkv_b;
    const void *o_a, *o_b;
    const void *gate_up_a, *gate_b, *up_b;
    const void *down_a, *down_b;
} orthrus_lora_layer;

typedef struct orthrus_lora {
    int32_t rank[4]; /* qkv, o, gate/up, down: multiples of 16 up to 256; 0 = site not adapted */
    float scale;     /* the update's factor (alpha / r in the usual parameterisation) */
    const orthrus_lora_layer *layers; /* HOST array of n_layers entries, copied */
} orthrus_lora;

/* Maximum distinct adapters the embedding chunks of one batch may name. */
#define ORTHRUS_MAX_STEP_ADAPTERS 4

/* One embedding chunk: tokens at positions [offset, offset + len) of request `seq`
 * (Section 3.3: the n-token input split into chunks c_1..c_K across iterations). */
typedef struct orthrus_emb_chunk {
    int32_t seq, offset, len, flags;
} orthrus_emb_chunk;

/* One generation decode token: `ctx_len` tokens of request `seq` are already cached; the
 * input token sits at position ctx_len, its key/value are appended there and it attends to
 * ctx_len + 1 keys including its own. */
typedef struct orthrus_decode_row {
    int32_t seq, ctx_len;
} orthrus_decode_row;

/* One generation prefill chunk: prompt tokens at positions [offset, offset + len) of generation
 * request `seq`, run through the generator and appended to its cache like `len` decode tokens
 * (the prompt-processing item of the Section 3.2 batch unit).  flags: ORTHRUS_CHUNK_LAST marks
 * the prompt's final chunk, whose last row gets next-token logits; no other bit may be set. */
typedef struct orthrus_gen_chunk {
    int32_t seq, offset, len, flags;
} orthrus_gen_chunk;

/* The batch (HOST memory, except `hidden`), type-sorted as in Section 3.2: token_ids holds the
 * embedding chunks' tokens in chunk order, then the generation prefill chunks' tokens in chunk
 * order, then one input token per decode row.  n_gen_chunks / gen_chunks may be 0 / NULL.
 *   token_weights: HOST fp32, one weight per embedding-chunk token (same order as token_ids);
 *     read for ORTHRUS_POOL_WMEAN chunks, whose weights must be finite and >= 0 (EDESC); may be
 *     NULL when no chunk uses that head.
 *   hidden: DEVICE fp32 [emb_kv n_seq][hidden_stride][d]: an ORTHRUS_POOL_BUFFER chunk of request
 *     s writes its final-normed hidden rows to rows s * hidden_stride + offset .. + len - 1
 *     (ECAPACITY if offset + len > hidden_stride); may be NULL when no chunk uses that head.
 *   chunk_adapter: HOST int32 per embedding chunk: index of the embedding model's LoRA adapter
 *     (orthrus_model_set_adapters) its rows go through, -1 for the base model (EDESC outside
 *     [-1, n_adapters); ECAPACITY for more than ORTHRUS_MAX_STEP_ADAPTERS distinct ones); NULL =
 *     every chunk uses the base model.  Prompt chunks and decode rows never use an adapter. */
typedef struct orthrus_batch {
    int32_t n_chunks, n_decode;
    const orthrus_emb_chunk *chunks;
    const orthrus_decode_row *rows;
    const int32_t *token_ids;
    int32_t n_gen_chunks;
    const orthrus_gen_chunk *gen_chunks;
    const float *token_weights;
    float *hidden;
    int32_t hidden_stride;
    const int32_t *chunk_adapter;
} orthrus_batch;

/* A paged KV cache (device), model dtype.  k_cache: [n_layers][n_pages][n_kv_heads][page][hd]
 * (keys stored after rotation, position-major inside a page); v_cache:
 * [n_layers][n_pages][n_kv_heads][hd][page] (dim-major inside a page, so that 8 consecutive
 * positions of one value dim are contiguous).  block_table: int32 [n_seq][max_blocks]; position
 * p of request s lives in page block_table[s][p / page] at in-page position p % page.  For a
 * model without layers the pools are never touched and may be NULL (the block table is still
 * validated). */
typedef struct orthrus_kv {
    void *k_cache;
    void *v_cache;
    const int32_t *block_table;
    int32_t n_pages, n_seq, max_blocks;
} orthrus_kv;

/* Validates `cfg` (EINVAL / EUNSUPPORTED) and `w` (EINVAL on a null pointer other than
 * lm_head) and returns a host handle that keeps copies of both.  No device work. */
int orthrus_model_create(const orthrus_config *cfg, const orthrus_weights *w, orthrus_model **out);
void orthrus_model_destroy(orthrus_model *m);

/* Registers the adapters that embedding chunks of `m` may name (index into this array), replacing
 * earlier ones; n = 0 removes them.  All adapters must have the same four ranks (EUNSUPPORTED
 * otherwise, or for a rank that is not a multiple of 16 up to 256); a null A or B of an adapted
 * site is EINVAL.  Host only; size workspaces (orthrus_workspace_bytes) after this call. */
int orthrus_model_set_adapters(orthrus_model *m, const orthrus_lora *adapters, int32_t n);

/* Device workspace bytes for steps of at most max_tokens tokens (all chunk tokens + decode
 * rows), at most max_chunks chunks (embedding plus generation prefill), at most max_decode
 * decode rows, and decode contexts of at most max_ctx tokens.  `gen` may equal `emb`.  Returns 0
 * for invalid arguments. */
size_t orthrus_workspace_bytes(const orthrus_model *emb, const orthrus_model *gen, int32_t max_tokens,
                               int32_t max_chunks, int32_t max_decode, int32_t max_ctx);

/* One mixed step, enqueued on `stream` (a hipStream_t; NULL = default stream); returns after
 * enqueueing.  Embedding chunks run through `emb` and read/append `emb_kv`; generation prefill
 * chunks and decode rows run through `gen` (needs an LM head when any row gets logits) and
 * read/append `gen_kv`.  `gen` may equal `emb` (shared backbone) and `gen_kv` may equal
 * `emb_kv` (then all three item types share one sequence namespace); two distinct models must
 * have equal configs.
 *   acc_sum  [emb_kv->n_seq][d] fp32 device, acc_w [emb_kv->n_seq] fp32 device: pooling state S,
 *            W of Eq. (1)-(2) per embedding request, updated in place.  A chunk at offset 0
 *            resets its request's state; a later chunk requires W == offset (else device error
 *            ORTHRUS_DEVERR_ACC and the chunk's pooling update is skipped).
 *   out_logits [n_logit_rows][vocab] fp32 device, n_logit_rows = (generation chunks flagged
 *            LAST) + n_decode: next-token logits of the last row of each final prompt chunk, in
 *            chunk order, then of each decode row.  May be NULL when n_logit_rows is 0.
 *   out_emb  [n_chunks][d] fp32 device: row i is written only if chunk i has ORTHRUS_CHUNK_LAST
 *            and a head that emits; it holds v / max(||v||_2, 1e-12) with v = S / W (mean) or S
 *            (weighted mean, last, CLS).
 *   workspace: device buffer of ws_bytes >= orthrus_workspace_bytes(...) for this batch.
 * Host-side validation (EINVAL, EDESC, EDUPSEQ, ECAPACITY) runs before anything is enqueued.
 * One step in flight per workspace.  Outputs are valid once the stream has synchronised.  With
 * two distinct models, the generator rows' launches run on a second stream owned by `emb`
 * (default priority), forked from and joined back to `stream` inside the enqueued work, so
 * ordering against `stream` is as for a single-stream step; calls sharing `emb` that use it
 * this way are serialised on the host. */
int orthrus_step(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                 const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, float *acc_sum, float *acc_w,
                 float *out_logits, float *out_emb, void *workspace, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (tight serving loops, harnesses that forbid
 * hipMalloc): the same step as orthrus_step() with the workspace
 * replaced by library-owned scratch, a static device array of ORTHRUS_SCRATCH_BYTES that every
 * GPU the library runs on holds until the process ends.  It calls no hipMalloc, hipFree,
 * hipHostMalloc or other allocating routine and creates no stream or event: the step's metadata
 * is copied from host memory with hipMemcpyAsync on `stream`, the two row groups of a two-model
 * step run one after the other on `stream`, and kernel timing (orthrus_profile_begin) does not
 * apply.  Results are identical to orthrus_step()'s.
 *   device_error: device int32 or NULL; once the stream has synchronised it holds this step's
 *     device error bits (ORTHRUS_DEVERR_*, 0 = none).  Every call starts with no bits set.
 * ECAPACITY when the batch needs more workspace than ORTHRUS_SCRATCH_BYTES (orthrus_workspace_bytes
 * with this batch's sizes tells in advance; nothing is enqueued then); otherwise the return codes
 * of orthrus_step().  All calls on one GPU share its scratch, which keeps the last call's
 * contents: calls that overlap on one GPU (several streams or host threads) race and corrupt each
 * other's results, so serialise them.  Not for capture into a HIP graph: the metadata copy reads
 * a host buffer that lives only for the duration of the call. */
#define ORTHRUS_SCRATCH_BYTES (64u << 20)
int orthrus_step_noalloc(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                         const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, float *acc_sum, float *acc_w,
                         float *out_logits, float *out_emb, int32_t *device_error, void *stream);

/* Greedy sampling (the sampler of Algorithm 1): out_tokens[r] = argmax over v of
 * logits[r * vocab + v] for r < rows, enqueued on `stream`.  Ties go to the lowest index; a NaN
 * counts as larger than every number (the first NaN wins), so the result equals a first-maximum
 * argmax in which NaN compares greatest.  logits: fp32 device [rows][vocab]; out_tokens: int32
 * device [rows].  EINVAL for rows < 0, vocab < 1, or a null pointer with rows > 0; rows == 0
 * is otherwise a no-op.  Launch failures return EHIP. */
int orthrus_sample_greedy(const float *logits, int32_t rows, int32_t vocab, int32_t *out_tokens,
                          void *stream);

/* Zeroes the device error word at the start of `workspace` (enqueued on `stream`).  Call once
 * on a freshly allocated workspace before its first step. */
int orthrus_workspace_init(void *workspace, void *stream);

/* Synchronises `stream`, then reads and clears the device error word of `workspace`.
 * Returns ORTHRUS_OK, ORTHRUS_EDEVICE (bits in *bits if non-NULL) or ORTHRUS_EHIP. */
int orthrus_device_error(void *workspace, void *stream, int32_t *bits);

/* Host-side plan of a batch without touching the GPU (for inspection and tests).  Counts the
 * attention work items the step would launch: n_prefill_items (query tiles of embedding and
 * generation prefill chunks), n_decode_items (key-range splits of decode rows, one per KV head
 * and split).  If `items` is non-NULL it receives up to `cap` items of 8 int32 each:
 *   {kind (0 prefill, 1 decode), chunk or row index, kv head, q_begin or split index,
 *    q_count or n_splits, key_begin, key_end (exclusive), partial slot or -1}.
 * Chunk indices count the embedding chunks first, then the generation prefill chunks.  On the
 * bf16 path a prefill tile over a long cached prefix may be cut along its keys into pieces (one
 * item each, cuts on 64-key boundaries at or before the tile's first query): a piece has a
 * partial slot, the first of 128 / group consecutive slots holding its rows. */
int orthrus_plan(const orthrus_model *emb, const orthrus_model *gen, const orthrus_batch *batch,
                 const orthrus_kv *emb_kv, const orthrus_kv *gen_kv, int32_t *n_prefill_items,
                 int32_t *n_decode_items, int32_t *items, int32_t cap);

/* Per-launch kernel timing, for measurement.  Between orthrus_profile_begin() and
 * orthrus_profile_end() every orthrus_step() whose `emb` is `m` records a hipEvent pair on its
 * stream around each kernel launch.  orthrus_profile_end() synchronises those events and writes
 * up to `cap` entries (one per kernel name, in first-launch order) with the launch count and the
 * summed event time; *n_out receives the number of names.  In a step of two distinct models the
 * launches over the generator's rows (prompt chunks and decode rows, attention included) are named
 * with the suffix "@gen" (e.g. "attention@gen"), those over the embedding model's rows without it.  Returns EHIP on a runtime failure. */
typedef struct orthrus_kernel_time {
    char name[32];
    int32_t launches;
    double total_ms;
} orthrus_kernel_time;
int orthrus_profile_begin(orthrus_model *m);
int orthrus_profile_end(orthrus_model *m, orthrus_kernel_time *out, int32_t cap, int32_t *n_out);
/* Limits the launches that profiling windows of `m` time to those named `name` (the names
 * orthrus_profile_end reports; NULL or "" = every launch, the initial state), so that a window can
 * time one kernel inside steps otherwise run as usual: two events per named launch instead of two
 * per launch.  Stays in effect until changed; EINVAL for a null model. */
int orthrus_profile_only(orthrus_model *m, const char *name);

const char *orthrus_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* ORTHRUS_H */
