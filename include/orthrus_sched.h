/*
 * orthrus_sched.h -- C ABI of the intra-batch scheduler and the iteration runner.
 *
 * The scheduler builds the batch of one iteration of the heterogeneous-batching loop
 * (Algorithm 1, Schedule): ScheduleRunning first reserves budget for generation requests in
 * the decode phase, then the credit loop of intra-batch scheduling (Algorithm 2, Section 4)
 * alternates between the embedding queue and the generation queue with ScheduleOne, admitting
 * one chunk of at most `chunk` tokens per request, until the token budget is used up or
 * neither queue can contribute.  It is host code only (no device calls): request state,
 * persistent credits, sequence slots and the paged-cache block tables.
 *
 * The runner is the whole loop body on one GPU: schedule, mirror the changed block-table rows
 * to the device, orthrus_step (forward, incremental pooler, LM head), orthrus_sample_greedy
 * (sampler), copy finished embeddings and sampled tokens back, and commit (emit).
 *
 * Semantics fixed here where the paper leaves them open:
 *   - A request appears at most once per batch.  ScheduleOne takes the first request of its
 *     queue (arrival order) not yet in the batch; its chunk is min(chunk, remaining tokens,
 *     remaining budget) tokens, or, with atomic_embeddings, an embedding request's whole
 *     remainder when it fits the remaining budget.  If that request cannot be admitted (budget
 *     or cache capacity) its queue contributes nothing more this iteration: requests of one
 *     type never overtake each other.  The loop's "queue nonempty" means "can contribute";
 *     the credit reset when a queue drains uses plain emptiness.
 *   - Weights w_e, w_g = remaining tokens of the queued requests, computed once per iteration
 *     before the loop; credits are exact 64-bit integers that persist across iterations.
 *   - ScheduleRunning serves decode-phase requests in the order they entered that phase; the
 *     first that does not fit the budget waits, with all later ones (no swapping).
 *   - Cache capacity is reserved whole at a request's first admission: one sequence slot and
 *     the pages of every position it will write (embedding: n; generation: n + max_new - 1),
 *     released when it finishes.  Running requests never wait for pages.
 *   - A generation request's final prompt chunk yields its first token; with max_new > 1 it
 *     then decodes one token per iteration (decode item at ctx_len = n + generated - 1).
 *   - A sampled token equal to eos_token (if >= 0) ends its request at commit.
 *   - A batch holds chunks of at most ORTHRUS_MAX_STEP_ADAPTERS distinct LoRA adapters; an
 *     embedding request whose adapter would exceed that cannot be admitted this iteration.
 *
 * Conventions: host pointers only in the scheduler; the caller owns every buffer it passes;
 * arrays returned by the scheduler stay valid until its next orthrus_sched_next / _commit /
 * _destroy call.  Return value: ORTHRUS_OK or a negative ORTHRUS_E* code (orthrus.h); on an
 * error nothing changes.  One thread at a time per scheduler or runner.
 */
#ifndef ORTHRUS_SCHED_H
#define ORTHRUS_SCHED_H

#include <stddef.h>
#include <stdint.h>

#include "orthrus.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct orthrus_sched_config {
    int32_t budget;            /* B: tokens per iteration, >= 1 */
    int32_t chunk;             /* C: most tokens of one embedding or prompt chunk, >= 1 */
    int32_t atomic_embeddings; /* 1: embedding requests only as one whole chunk (no cap C) */
    int32_t decode_tokens;     /* tokens one decode item advances; 1 for orthrus_step */
    int32_t page_size;         /* cache page size; 16 for orthrus_step */
    int32_t shared_cache;      /* 1: both request types use cache 0 (cache 1 fields unused) */
    int32_t eos_token;         /* -1: no end-of-sequence token */
    int32_t n_seq[2];          /* per cache (0: embedding or shared, 1: generation): slots */
    int32_t n_pages[2];        /*   pages */
    int32_t max_blocks[2];     /*   block-table columns */
} orthrus_sched_config;

typedef struct orthrus_sched orthrus_sched;

/* EINVAL for a null pointer or a field out of range. */
int orthrus_sched_create(const orthrus_sched_config *cfg, orthrus_sched **out);
void orthrus_sched_destroy(orthrus_sched *s);

/* Queue a request (arrival order = call order).  tokens: n token ids (host), copied; NULL stands
 * for n zeros (scheduling studies).  pool: ORTHRUS_POOL_MEAN / _LAST / _CLS / _WMEAN (buffered
 * heads are left to callers of orthrus_step, which own the hidden buffer); weights: with
 * ORTHRUS_POOL_WMEAN, n finite non-negative weights (host, copied), else ignored.  adapter: the
 * embedding model's LoRA adapter index or -1 (checked by orthrus_step); a batch takes chunks of at
 * most ORTHRUS_MAX_STEP_ADAPTERS distinct adapters.  EINVAL: id already live, n < 1, max_new < 1,
 * bad pool, weights or adapter; ECAPACITY: the request's reservation exceeds the block table or
 * the cache's pages (it could never be admitted). */
int orthrus_sched_submit_embedding(orthrus_sched *s, int64_t id, const int32_t *tokens,
                                   const float *weights, int32_t n, int32_t pool, int32_t adapter);
int orthrus_sched_submit_generation(orthrus_sched *s, int64_t id, const int32_t *prompt, int32_t n,
                                    int32_t max_new);

/* One iteration's batch.  `batch` is ready for orthrus_step: chunk and row `seq` fields are cache
 * slots (embedding chunks in cache 0; prompt chunks and decode rows in cache 1, or 0 when shared)
 * and token_ids holds the chunk tokens and each decode row's input token (the request's last
 * committed sampled token, 0 if none was committed). */
typedef struct orthrus_sched_batch {
    orthrus_batch batch;
    const int64_t *chunk_ids;      /* [batch.n_chunks] request of each embedding chunk */
    const int64_t *gen_chunk_ids;  /* [batch.n_gen_chunks] request of each prompt chunk */
    const int64_t *row_ids;        /* [batch.n_decode] request of each decode row */
    const int32_t *row_tokens;     /* [batch.n_decode] tokens each decode item advances */
    int32_t n_logit_rows;          /* final prompt chunks, then decode rows */
    const int64_t *logit_ids;      /* [n_logit_rows] */
    int32_t tokens_used;           /* budget tokens the batch takes */
    int32_t n_picks;               /* credit-loop selections, in order: 'e' or 'g' */
    const char *picks;
    int32_t n_finishing;           /* requests whose last item is in this batch */
    const int64_t *finishing_ids;
    int32_t n_table_rows;          /* block-table rows assigned since the previous batch */
    const int32_t *table_rows;     /* [n_table_rows][2]: cache, slot */
    int64_t credit_e, credit_g;    /* credits after the loop */
} orthrus_sched_batch;

/* Build the next batch (an empty one when nothing can run).  EINVAL if the previous batch has
 * not been committed. */
int orthrus_sched_next(orthrus_sched *s, orthrus_sched_batch *out);

/* End the iteration.  sampled: the token of each logits row of the batch (n == n_logit_rows), or
 * NULL with n == 0 (no tokens: decode inputs stay 0, no end-of-sequence check).  Requests that
 * finished (last item scheduled, or end-of-sequence sampled) release their slot and pages; up to
 * `cap` of their ids go to finished (may be NULL), their count to *n_finished (may be NULL). */
int orthrus_sched_commit(orthrus_sched *s, const int32_t *sampled, int32_t n, int32_t *n_finished,
                         int64_t *finished, int32_t cap);

/* Host block table of cache c (0 or 1): [n_seq][max_blocks] int32, -1 where unassigned.  NULL for
 * a bad cache index (or cache 1 of a shared configuration). */
const int32_t *orthrus_sched_block_table(const orthrus_sched *s, int32_t cache);

/* The configuration the scheduler was created with. */
int orthrus_sched_get_config(const orthrus_sched *s, orthrus_sched_config *out);

/* Queue and phase counts: queued embedding requests, queued generation requests (prompt not
 * finished), decode-phase requests, free slots and free pages of cache 0 and 1 (7 values). */
int orthrus_sched_counts(const orthrus_sched *s, int64_t *counts7);

/* ------------------------------------------------------------------------------- runner */

/* Device buffers of the runner (caller-owned, current device):
 *   acc_sum [n_seq(cache 0)][d] and acc_w [n_seq(cache 0)] fp32: pooling state by cache slot;
 *   logits [budget][vocab] fp32; out_emb [budget][d] fp32; tokens [budget] int32;
 *   workspace of ws_bytes >= orthrus_workspace_bytes(emb, gen, budget, budget, budget,
 *   max_blocks * page_size of the larger cache), initialised with orthrus_workspace_init.
 * The caches' block_table pointers must have the scheduler's shapes; the runner overwrites the
 * rows the scheduler assigns. */
typedef struct orthrus_runner_buffers {
    float *acc_sum, *acc_w, *logits, *out_emb;
    int32_t *tokens;
    void *workspace;
    size_t ws_bytes;
} orthrus_runner_buffers;

typedef struct orthrus_runner orthrus_runner;

/* Checks that the scheduler fits the models and caches (page size, decode_tokens == 1, slot and
 * block counts, workspace size): EINVAL / ECAPACITY.  Allocates pinned host staging only. */
int orthrus_runner_create(const orthrus_model *emb, const orthrus_model *gen, const orthrus_kv *emb_kv,
                          const orthrus_kv *gen_kv, orthrus_sched *sched, const orthrus_runner_buffers *buf,
                          orthrus_runner **out);
void orthrus_runner_destroy(orthrus_runner *r);

/* What one iteration produced (host arrays owned by the runner, valid until its next call). */
typedef struct orthrus_runner_output {
    int32_t n_tokens;              /* sampled tokens, one per logits row */
    const int64_t *token_ids;      /*   request of each */
    const int32_t *tokens;
    int32_t n_embeddings;          /* finished embeddings (L2-normalised, fp32) */
    const int64_t *embedding_ids;
    const float *embeddings;       /*   [n_embeddings][d] */
    int32_t n_finished;            /* requests that ended this iteration */
    const int64_t *finished_ids;
    int32_t tokens_used;           /* budget tokens of the batch */
    int32_t n_items;               /* batch items (0: nothing to run) */
} orthrus_runner_output;

/* One loop iteration (Algorithm 1): schedule, step, sample, emit.  Synchronises `stream`.  A
 * device-side error (orthrus_device_error) returns EDEVICE after the commit. */
int orthrus_runner_iterate(orthrus_runner *r, void *stream, orthrus_runner_output *out);

#ifdef __cplusplus
}
#endif
#endif /* ORTHRUS_SCHED_H */
