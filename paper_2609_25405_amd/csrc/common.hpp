// Device helpers shared by the gfx950 kernels: bf16 conversion, MFMA operand types,
// wave reductions and the launcher declarations each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "orthrus.h"

namespace orthrus {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// float -> bf16, round to nearest even: gfx950's v_cvt_pk_bf16_f32 (two values per instruction)
__device__ __forceinline__ uint32_t f2bf_bits(float f) {
    return __builtin_bit_cast(uint16_t, (bf16)f);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2 v;
    v[0] = (bf16)lo;
    v[1] = (bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16>(bf16 v) {
    return __uint_as_float((uint32_t)__builtin_bit_cast(uint16_t, v) << 16);
}
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// sticky device error word (vector atomics only)
__device__ __forceinline__ void flag_error(int *err, int bit) { atomicOr(err, bit); }

// ---------------------------------------------------------------------------------------
// launchers (host functions defined next to their kernels)
// ---------------------------------------------------------------------------------------
enum GemmEpilogue { EPI_STORE_F32 = 0, EPI_ADD_F32 = 1, EPI_SWIGLU = 2, EPI_QKV_ROPE = 3 };

// QKV projection epilogue (bf16 path): rotate q and k at each token's position, store q for
// attention and append rotated k and raw v to the paged cache (Section 3.2's cache writes)
struct QkvRope {
    const float2 *cs;          // [T][hd/2] (cos, sin) of each token's position
    const int32_t *pos, *seq;  // per token (global token index)
    void *q_out;               // [T][nq][hd]
    void *k_cache[2], *v_cache[2];          // layer base per pool
    const int32_t *block_table[2];
    int n_pages[2], max_blocks[2];
    int row0;                  // global token index of the launch's row 0
    int Te;                    // tokens < Te use pool 0, others pool 1
    int nq, nkv, hd, page;
    int *err;
};

// LoRA update of a projection (rows [0, rows) of the launch): out += U B^T, with U [rows][ldu]
// the scaled, per-row-masked shrink x A^T of the n adapters in use side by side (adapter j owns
// columns j*r .. j*r + r - 1) and B_j [N][r].  SwiGLU launches read b0 for gate, b1 for up.
constexpr int kMaxStepAdapters = ORTHRUS_MAX_STEP_ADAPTERS;
struct LoraGemm {
    const void *u;
    const void *u_lo;          // bf16 path: U = u + u_lo (u the bf16 rounding, u_lo the rest)
    int ldu, rows, r, n;       // n = 0: no update
    const void *b0[kMaxStepAdapters], *b1[kMaxStepAdapters];
};

struct GemmArgs {
    const void *A;   // [M][K] activations, row stride lda (elements)
    const void *B0;  // [N][K] weights (gate for SwiGLU)
    const void *B1;  // [N][K] up-projection weights (SwiGLU only)
    void *out;       // fp32 [M][N] (store/add) or activation dtype [M][N] (SwiGLU)
    int M, N, K, lda, ldo;
    // split-K (bf16 path, EPI_ADD_F32 only): with splits > 1 split s writes its fp32 share of
    // rows [0, M) to partial + s * split_stride (row stride ldo) instead of adding into out
    int splits;
    float *partial;
    size_t split_stride;
    QkvRope rope;    // EPI_QKV_ROPE only
    LoraGemm lora;   // adds the low-rank update before the epilogue (split 0 of a split-K launch)
    // B0 in the 64 x 64 blocked layout ([ceil(N/64)][K/64][64][64]; bf16 path, not SwiGLU):
    // one tile stage reads whole 8 KB runs instead of 128-byte pieces of 64 rows
    int b_blocked;
    // 1: the launch runs concurrently with another stream's launches, so the workgroup time it
    // takes from the shared CUs, not its own length, is what it costs; the bf16 dispatch then
    // gives split-K projections of 129..256 rows the largest tiles
    int wide;
};
hipError_t launch_gemm(int dtype, int epilogue, const GemmArgs &a, hipStream_t s);
// bf16 [rows][cols] -> the 64 x 64 blocked layout GemmArgs::b_blocked reads (cols % 64 == 0)
hipError_t launch_block_weights(const void *src, void *dst, int rows, int cols, hipStream_t s);
// split-K factor (<= max_splits; each split a run of whole 64-deep stages, the stages dealt as
// evenly as the count allows) for a bf16 residual-add projection of this shape; launch_gemm
// ignores a requested split count larger than K's number of stages
int gemm_add_splits(int M, int N, int K, int max_splits);

// LoRA shrink: u[row][j*r + k] = scale[j] * sum_i x[row][i] a_j[k][i] for the adapter j of the
// row (row_adapter[row]), 0 in the other adapters' columns.  x [rows][K] with row stride ldx,
// a_j [r][K], u [rows][n*r] (bf16 on the bf16 path, with u_lo; fp32 on the fp32 path).
struct LoraShrink {
    const void *x;
    int ldx, K, rows, r, n;
    const void *a[kMaxStepAdapters];
    float scale[kMaxStepAdapters];
    const int32_t *row_adapter;
    void *u;
    void *u_lo;                // bf16 path: the rounding remainder of u (u + u_lo = U to ~16 bits)
};
hipError_t launch_lora_shrink(int dtype, const LoraShrink &p, hipStream_t s);

struct NormArgs {
    const float *x;         // fp32 residual rows [rows][d]
    const float *pend;      // pending split-K slabs added to x first (npend of them, or none)
    size_t pend_stride;     // floats between slabs
    int npend;
    float *x_out;           // gather mode: fp32 rows written here
    const void *table;      // gather mode: token table [vocab][d] of the model dtype
    const int32_t *tok;     // gather mode: token per row
    const float *gain;      // [d]
    void *y;                // normalised rows [rows][d], model dtype
    int rows, d;
    float eps;
    // gather mode, optional: per row (cos, sin) of pos * base^(-2i/hd), i < hd/2, into cs
    float2 *cs;
    const int32_t *pos;
    int hd;
    float rope_base;
};
hipError_t launch_rmsnorm(int dtype, bool gather, const NormArgs &a, hipStream_t s);

struct RopeArgs {
    const float *qkv;        // fp32 [T][qkv_dim]: nslab partial sums slab_stride floats apart,
    int nslab;               // added in order (split-K of the QKV projection); 1 = plain rows
    size_t slab_stride;
    const float2 *cs;        // per-token (cos, sin) table [T][hd/2], or null: computed here
    void *q_out;             // [T][nq][hd] model dtype
    const int32_t *pos, *seq;
    void *k_cache[2], *v_cache[2];          // layer base per pool
    const int32_t *block_table[2];
    int n_pages[2], max_blocks[2];
    int Te;                  // tokens < Te use pool 0, others pool 1
    int T, nq, nkv, hd, page;
    float rope_base;
    int *err;
};
hipError_t launch_rope_append(int dtype, const RopeArgs &a, hipStream_t s);

struct AttnArgs {
    const void *q;            // [T][nq][hd]
    void *o;                  // [T][nq * hd]
    const void *k_cache[2], *v_cache[2];
    const int32_t *block_table[2];
    int n_pages[2], max_blocks[2];
    const int32_t *chunks, *rows, *items;
    const int32_t *split_rows;  // indices of the decode rows with more than one split
    const int32_t *combine;   // merge entries of key-split prefill tiles
    float *partials;          // [slot][group][hd + 2]
    // n_prefill: prefill items at the head of `items` (0: decode items only, served by the
    // decode-only kernel on the bf16 path); n_items: all items of the launch
    int n_prefill, n_items, n_combine, Te, nq, nkv, hd, page;
    int *err;
};
hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t s);
// merges the partials of the n_decode decode rows listed in a.split_rows (0 = none) and of the
// a.n_combine key-split prefill tiles
hipError_t launch_attn_combine(int dtype, const AttnArgs &a, int n_decode, hipStream_t s);

struct PoolArgs {
    const float *x;           // fp32 residual rows [T][d]
    const float *gain;        // embedding model's final norm gain [d]
    const float *gen_gain;    // generator's final norm gain [d] (rows that get logits)
    void *act;                // LM-head input [n_lm][d], model dtype
    const int32_t *lm_rows;   // [n_lm] token rows that get logits
    const int32_t *chunks;    // chunk table; the first n_chunks entries are embedding chunks
    float *inv_rms;           // [Te] scratch: final-norm scale of the embedding rows
    float *acc_sum, *acc_w, *out_emb;
    const float *pend;        // pending split-K slabs added to x first (npend of them, or none)
    size_t pend_stride;
    int npend;
    const float *weights;     // [Te] per-token weights (weighted-mean chunks), or null
    const int32_t *hid_rows;  // [Te] hidden-buffer row of each embedding token (-1: none), or null
    float *hidden;            // buffered-head output [rows][d] fp32
    int n_chunks, Te, d;
    int n_emb_rows, n_lm;     // final-norm launch: embedding rows [0, n_emb_rows), lm_rows
    float eps;
    int *err;
};
// final RMSNorm: 1/rms of embedding rows [0, n_emb_rows) (and the normalised row into the
// hidden buffer for buffered-head tokens), then the n_lm rows listed in lm_rows normalised into act
hipError_t launch_final_rows(int dtype, const PoolArgs &a, hipStream_t s);
// greedy sampler: out[r] = first index of the largest logits[r][.] (NaN compares greatest)
hipError_t launch_argmax(const float *logits, int rows, int vocab, int32_t *out, hipStream_t s);
// incremental pooler update and finished embeddings.  Single-row heads (last token, CLS) take
// their row's final norm themselves (adding npend slabs); with any_rows, mean, weighted-mean and
// buffered chunks are handled too and need launch_final_rows over the embedding rows first.
hipError_t launch_pool(const PoolArgs &a, bool any_rows, hipStream_t s);
// both at once when no chunk needs every embedding row's norm (n_emb_rows == 0): the LM rows'
// final norm and the single-row pooler in one launch
hipError_t launch_final_and_pool(int dtype, const PoolArgs &a, hipStream_t s);

}  // namespace orthrus
