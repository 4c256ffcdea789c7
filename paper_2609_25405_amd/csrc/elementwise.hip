// Row-wise kernels of the step: token gather + RMSNorm, RMSNorm, rotary embedding with
// KV-cache append, the incremental pooler (Section 3.3) with the final L2 normalisation, and the
// greedy sampler of Algorithm 1 (argmax over each logits row).
#include "common.hpp"
#include "plan.hpp"

namespace orthrus {

namespace {

__device__ __forceinline__ float block_sum(float v, float *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float s = 0.f;
    for (int w = 0; w < nw; ++w) s += red[w];
    return s;
}

// 4 consecutive elements of the model dtype <-> float4
__device__ __forceinline__ float4 load4(const float *p) { return *(const float4 *)p; }
__device__ __forceinline__ float4 load4(const bf16 *p) {
    const uint2 u = *(const uint2 *)p;
    return float4{bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y)};
}
__device__ __forceinline__ void store4(float *p, float4 v) { *(float4 *)p = v; }
__device__ __forceinline__ void store4(bf16 *p, float4 v) {
    *(uint2 *)p = uint2{pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)};
}

// Rows of up to RV * 256 float4 (RV = 4 for d <= 4096, 8 for d <= 8192) are held in registers
// between the sum of squares and the scaled write; longer rows take a strided loop.
constexpr int kMaxPend = 4;  // split-K slabs a row kernel adds (the step splits K at most 4 ways)

// x row plus its pending split-K slabs into registers, x + slab 0 + slab 1 + ... in that order:
// every load is issued before the first add, so the row costs one memory latency whatever the
// number of slabs (a loop that adds each slab as it arrives waits once per slab)
template <int RV>
__device__ __forceinline__ void load_row_pend(float4 (&xv)[RV], const float *xrow, const float *pend,
                                              size_t pend_stride, int npend, int nv) {
    float4 p[kMaxPend][RV];
#pragma unroll
    for (int i = 0; i < RV; ++i) {
        const int v = threadIdx.x + i * 256;
        if (v < nv) xv[i] = load4(xrow + 4 * v);
    }
#pragma unroll
    for (int sp = 0; sp < kMaxPend; ++sp) {
        if (sp < npend) {
#pragma unroll
            for (int i = 0; i < RV; ++i) {
                const int v = threadIdx.x + i * 256;
                if (v < nv) p[sp][i] = load4(pend + sp * pend_stride + 4 * v);
            }
        }
    }
#pragma unroll
    for (int sp = 0; sp < kMaxPend; ++sp) {
        if (sp < npend) {
#pragma unroll
            for (int i = 0; i < RV; ++i) {
                const int v = threadIdx.x + i * 256;
                if (v < nv) xv[i] = float4{xv[i].x + p[sp][i].x, xv[i].y + p[sp][i].y, xv[i].z + p[sp][i].z,
                                           xv[i].w + p[sp][i].w};
            }
        }
    }
}

// y = x / sqrt(mean(x^2) + eps) * gain over one row per block (d a multiple of 4); gather mode
// first sets x = table[tok] (the fp32 copy is kept as the residual stream)
template <typename T, bool GATHER, int RV>
__global__ __launch_bounds__(256) void rmsnorm_kernel(NormArgs a) {
    __shared__ float red[4];
    const int r = blockIdx.x;
    const int nv = a.d / 4;
    float *xrow = (GATHER ? a.x_out : const_cast<float *>(a.x)) + (size_t)r * a.d;
    float ss = 0.f;
    if (nv <= RV * 256) {
        float4 xv[RV], gv[RV];
        // the gain first: its loads complete under the row's
#pragma unroll
        for (int i = 0; i < RV; ++i) {
            const int v = threadIdx.x + i * 256;
            if (v < nv) gv[i] = load4(a.gain + 4 * v);
        }
        if (GATHER) {
            const T *src = (const T *)a.table + (size_t)a.tok[r] * a.d;
#pragma unroll
            for (int i = 0; i < RV; ++i) {
                const int v = threadIdx.x + i * 256;
                if (v < nv) xv[i] = load4(src + 4 * v);
            }
        } else {
            load_row_pend<RV>(xv, xrow, a.pend + (size_t)r * a.d, a.pend_stride, a.npend, nv);
        }
        if (GATHER && a.cs && (int)threadIdx.x < a.hd / 2) {
            // rotation table of this token for the QKV epilogue (angle evaluated in double)
            const double inv_freq = pow((double)a.rope_base, -2.0 * (double)threadIdx.x / (double)a.hd);
            double sv, cv;
            sincos((double)a.pos[r] * inv_freq, &sv, &cv);
            a.cs[(size_t)r * (a.hd / 2) + threadIdx.x] = float2{(float)cv, (float)sv};
        }
#pragma unroll
        for (int i = 0; i < RV; ++i) {
            const int v = threadIdx.x + i * 256;
            if (v < nv) {
                if (GATHER || a.npend > 0) store4(xrow + 4 * v, xv[i]);
                ss += xv[i].x * xv[i].x + xv[i].y * xv[i].y + xv[i].z * xv[i].z + xv[i].w * xv[i].w;
            }
        }
        const float inv = rsqrtf(block_sum(ss, red) / (float)a.d + a.eps);
        T *y = (T *)a.y + (size_t)r * a.d;
#pragma unroll
        for (int i = 0; i < RV; ++i) {
            const int v = threadIdx.x + i * 256;
            if (v < nv) {
                const float4 g = gv[i];
                store4(y + 4 * v, float4{xv[i].x * inv * g.x, xv[i].y * inv * g.y, xv[i].z * inv * g.z,
                                         xv[i].w * inv * g.w});
            }
        }
        return;
    }
    if (GATHER && a.cs && (int)threadIdx.x < a.hd / 2) {
        // rotation table of this token for the QKV epilogue (angle evaluated in double)
        const double inv_freq = pow((double)a.rope_base, -2.0 * (double)threadIdx.x / (double)a.hd);
        double sv, cv;
        sincos((double)a.pos[r] * inv_freq, &sv, &cv);
        a.cs[(size_t)r * (a.hd / 2) + threadIdx.x] = float2{(float)cv, (float)sv};
    }
    if (GATHER) {
        const T *src = (const T *)a.table + (size_t)a.tok[r] * a.d;
        for (int v = threadIdx.x; v < nv; v += 256) {
            const float4 x = load4(src + 4 * v);
            store4(xrow + 4 * v, x);
            ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
        }
    } else {
        for (int v = threadIdx.x; v < nv; v += 256) {
            float4 x = load4(xrow + 4 * v);
            if (a.npend > 0) {
                // finish a split-K residual add: x += slab 0 + slab 1 + ... in order
                for (int sp = 0; sp < a.npend; ++sp) {
                    const float4 p = load4(a.pend + sp * a.pend_stride + (size_t)r * a.d + 4 * v);
                    x = float4{x.x + p.x, x.y + p.y, x.z + p.z, x.w + p.w};
                }
                store4(xrow + 4 * v, x);
            }
            ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
        }
    }
    const float inv = rsqrtf(block_sum(ss, red) / (float)a.d + a.eps);
    T *y = (T *)a.y + (size_t)r * a.d;
    for (int v = threadIdx.x; v < nv; v += 256) {
        const float4 x = load4(xrow + 4 * v), g = load4(a.gain + 4 * v);
        store4(y + 4 * v, float4{x.x * inv * g.x, x.y * inv * g.y, x.z * inv * g.z, x.w * inv * g.w});
    }
}

// q, k rotated at their absolute positions (pairs (i, i + hd/2), angle pos * base^(-2i/hd),
// evaluated in double), q stored for attention, rotated k and raw v appended at position
// pos % page of page block_table[seq][pos / page] (keys [kv head][slot][dim], values
// [kv head][dim][slot]).
template <typename T>
// One token per blockIdx.x; its work items (rotation quads of the q and k heads, then value
// quads) are dealt over gridDim.y blocks.  Angles come from the per-token table when the step
// built one (the same values the fused GEMM epilogue uses), else in double here.
__global__ __launch_bounds__(256) void rope_append_kernel(RopeArgs a) {
    __shared__ __attribute__((aligned(16))) float cs[64], sn[64];
    const int t = blockIdx.x;
    const int half = a.hd / 2;
    const int pos = a.pos[t];
    if ((int)threadIdx.x < half) {
        if (a.cs) {
            const float2 v = a.cs[(size_t)t * half + threadIdx.x];
            cs[threadIdx.x] = v.x;
            sn[threadIdx.x] = v.y;
        } else {
            const double inv_freq = pow((double)a.rope_base, -2.0 * (double)threadIdx.x / (double)a.hd);
            double sv, cv;
            sincos((double)pos * inv_freq, &sv, &cv);
            cs[threadIdx.x] = (float)cv;
            sn[threadIdx.x] = (float)sv;
        }
    }
    __syncthreads();
    const int p = t < a.Te ? 0 : 1;
    const int seq = a.seq[t];
    const int page = a.block_table[p][(size_t)seq * a.max_blocks[p] + pos / a.page];
    const bool ok = page >= 0 && page < a.n_pages[p];
    if (!ok && threadIdx.x == 0 && blockIdx.y == 0) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
    const int qkv_dim = (a.nq + 2 * a.nkv) * a.hd;
    const float *src = a.qkv + (size_t)t * qkv_dim;
    // four values of the row: the sum of the split-K partials, in split order
    auto slab4 = [&](const float *p) {
        float4 v = *(const float4 *)p;
        for (int k = 1; k < a.nslab; ++k) {
            const float4 w = *(const float4 *)(p + k * a.slab_stride);
            v.x += w.x;
            v.y += w.y;
            v.z += w.z;
            v.w += w.w;
        }
        return v;
    };
    const size_t slot = ok ? (((size_t)page * a.nkv) * a.page + pos % a.page) * a.hd : 0;
    // rotations: (nq + nkv) heads x (half / 4) quads of pairs (i..i+3, i+half..i+half+3); then
    // values, stored dim-major inside a page: [kv head][dim][slot]
    const int quads = half / 4;
    const int n_rot = (a.nq + a.nkv) * quads, n_all = n_rot + a.nkv * a.hd / 4;
    const float *vs = src + (size_t)(a.nq + a.nkv) * a.hd;
    T *v = ok ? (T *)a.v_cache[p] + (size_t)page * a.nkv * a.hd * a.page + pos % a.page : nullptr;
    for (int w = blockIdx.y * 256 + threadIdx.x; w < n_all; w += gridDim.y * 256) {
        if (w >= n_rot) {
            if (!ok) continue;
            const int u = w - n_rot;
            const float4 x = slab4(vs + 4 * u);
            v[(size_t)(4 * u + 0) * a.page] = from_f32<T>(x.x);
            v[(size_t)(4 * u + 1) * a.page] = from_f32<T>(x.y);
            v[(size_t)(4 * u + 2) * a.page] = from_f32<T>(x.z);
            v[(size_t)(4 * u + 3) * a.page] = from_f32<T>(x.w);
            continue;
        }
        const int head = w / quads, i = 4 * (w % quads);
        const float4 x1 = slab4(src + head * a.hd + i);
        const float4 x2 = slab4(src + head * a.hd + i + half);
        const float4 c = *(const float4 *)(cs + i), sn4 = *(const float4 *)(sn + i);
        const float4 y1 = {x1.x * c.x - x2.x * sn4.x, x1.y * c.y - x2.y * sn4.y, x1.z * c.z - x2.z * sn4.z,
                           x1.w * c.w - x2.w * sn4.w};
        const float4 y2 = {x2.x * c.x + x1.x * sn4.x, x2.y * c.y + x1.y * sn4.y, x2.z * c.z + x1.z * sn4.z,
                           x2.w * c.w + x1.w * sn4.w};
        T *dst;
        if (head < a.nq) {
            dst = (T *)a.q_out + ((size_t)t * a.nq + head) * a.hd;
        } else {
            if (!ok) continue;
            dst = (T *)a.k_cache[p] + slot + (size_t)(head - a.nq) * a.page * a.hd;
        }
        store4(dst + i, y1);
        store4(dst + i + half, y2);
    }
}

// The same rotation and append for batches of more than 256 tokens with the per-token rotation
// table given (bf16 path): 16 consecutive tokens and one head per block (grid: token groups x
// (nq + 2 nkv) heads).  Each thread's rows are read before the block's page lookups are
// waited for, and a value head's 16 rows leave dim by dim, 8 consecutive slots of one dim (16
// bytes) per store wherever 8 rows fill them, adjacent lanes taking the two 8-row halves of one
// dim (one token per block writes each value as its own 2-byte store).  7B layer: 1568 rows of
// 512-token chunks 23.2 -> 19.1 us, 2048 rows of short queries 27.4 -> 24.3 us; on decode
// batches (one token per sequence) the one-token blocks are faster (6.6 against 9.5 us at 64
// rows), and four heads per block measured slower (30 us at 1568 rows).
constexpr int kRopeGroup = 16;

__global__ __launch_bounds__(256) void rope_append_group_kernel(RopeArgs a) {
    using T = bf16;
    __shared__ int4 meta[kRopeGroup];  // per row {slot, page or -1, pool, -}
    const int head = blockIdx.y, t0 = blockIdx.x * kRopeGroup;
    const int hd = a.hd, half = hd / 2, quads = half / 4;
    const size_t qkv_dim = (size_t)(a.nq + 2 * a.nkv) * hd;
    const bool is_v = head >= a.nq + a.nkv;
    // one item per thread (hd <= 128): a q/k item is (row, quad of pairs (i..i+3,
    // i+half..i+half+3)), a value item (dim, 8-row half of the group)
    const int it = threadIdx.x;
    const bool has = is_v ? it < 2 * hd : it < kRopeGroup * quads;
    const int r = is_v ? (it & 1) * 8 : it / quads, i = is_v ? it >> 1 : 4 * (it % quads);
    float4 x1{}, x2{}, c{}, sn4{};
    float v[8];
    if (has && !is_v && t0 + r < a.T) {
        const float *src = a.qkv + (size_t)(t0 + r) * qkv_dim + (size_t)head * hd;
        x1 = *(const float4 *)(src + i);
        x2 = *(const float4 *)(src + i + half);
        for (int k = 1; k < a.nslab; ++k) {   // split-K partials, in split order
            const float4 w1 = *(const float4 *)(src + k * a.slab_stride + i);
            const float4 w2 = *(const float4 *)(src + k * a.slab_stride + i + half);
            x1 = float4{x1.x + w1.x, x1.y + w1.y, x1.z + w1.z, x1.w + w1.w};
            x2 = float4{x2.x + w2.x, x2.y + w2.y, x2.z + w2.z, x2.w + w2.w};
        }
        const float2 *csr = a.cs + (size_t)(t0 + r) * half + i;
        const float2 c0 = csr[0], c1 = csr[1], c2 = csr[2], c3 = csr[3];
        c = float4{c0.x, c1.x, c2.x, c3.x};
        sn4 = float4{c0.y, c1.y, c2.y, c3.y};
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        v[k] = 0.f;
        if (has && is_v && t0 + r + k < a.T) {
            const float *p = a.qkv + (size_t)(t0 + r + k) * qkv_dim + (size_t)head * hd + i;
            float x = p[0];
            for (int sl = 1; sl < a.nslab; ++sl) x += p[sl * a.slab_stride];
            v[k] = x;
        }
    }
    if (threadIdx.x < kRopeGroup) {
        const int t = t0 + threadIdx.x;
        int4 md{0, -1, 0, 0};
        if (t < a.T) {
            const int pos = a.pos[t], p = t < a.Te ? 0 : 1;
            const int page = a.block_table[p][(size_t)a.seq[t] * a.max_blocks[p] + pos / a.page];
            const bool ok = page >= 0 && page < a.n_pages[p];
            if (!ok && head == 0) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
            md = int4{pos % a.page, ok ? page : -1, p, 0};
        }
        meta[threadIdx.x] = md;
    }
    __syncthreads();
    if (!has) return;
    if (!is_v) {
        const int t = t0 + r;
        if (t >= a.T) return;
        const bool is_q = head < a.nq;
        const int4 md = meta[r];
        if (!is_q && md.y < 0) return;
        const float4 y1 = {x1.x * c.x - x2.x * sn4.x, x1.y * c.y - x2.y * sn4.y, x1.z * c.z - x2.z * sn4.z,
                           x1.w * c.w - x2.w * sn4.w};
        const float4 y2 = {x2.x * c.x + x1.x * sn4.x, x2.y * c.y + x1.y * sn4.y, x2.z * c.z + x1.z * sn4.z,
                           x2.w * c.w + x1.w * sn4.w};
        T *dst = is_q ? (T *)a.q_out + ((size_t)t * a.nq + head) * hd
                      : (T *)a.k_cache[md.z] + (((size_t)md.y * a.nkv + (head - a.nq)) * a.page + md.x) * hd;
        store4(dst + i, y1);
        store4(dst + i + half, y2);
        return;
    }
    // value head: dim i of rows r..r+7, one 16-byte store where they fill 8 aligned slots of a page
    const int kvh = head - a.nq - a.nkv;
    const int4 m0 = meta[r];
    bool run = t0 + r + 7 < a.T && m0.y >= 0 && (m0.x & 7) == 0;
#pragma unroll
    for (int k = 1; k < 8; ++k) {
        const int4 mk = meta[r + k];
        run = run && mk.y == m0.y && mk.z == m0.z && mk.x == m0.x + k;
    }
    if (run) {
        T *dst = (T *)a.v_cache[m0.z] + (((size_t)m0.y * a.nkv + kvh) * hd + i) * a.page + m0.x;
        *(uint4 *)dst = uint4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                              pack_bf16x2(v[6], v[7])};
        return;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int4 mk = meta[r + k];
        if (t0 + r + k >= a.T || mk.y < 0) continue;
        ((T *)a.v_cache[mk.z])[(((size_t)mk.y * a.nkv + kvh) * hd + i) * a.page + mk.x] = from_f32<T>(v[k]);
    }
}

// ---------------------------------------------------------------------- incremental pooler
// Final RMSNorm, one row per block.  Blocks [0, n_emb_rows) take embedding rows 0.. and keep
// only the scale 1/rms (the pooler applies it); the following blocks take the rows listed in
// lm_rows and write them, normalised with the generator's gain, as consecutive rows of the LM
// head's input.
template <typename T, int RV>
__device__ void final_row_block(const PoolArgs &a, int b, float *red) {
    const bool emb_row = b < a.n_emb_rows;
    const int lm = b - a.n_emb_rows;
    const int r = emb_row ? b : a.lm_rows[lm];
    const int nv = a.d / 4;
    float *x = const_cast<float *>(a.x) + (size_t)r * a.d;
    float ss = 0.f;
    if (nv <= RV * 256) {
        float4 xv[RV], gv[RV];
        // an LM row's gain first: its loads complete under the row's
        if (!emb_row) {
#pragma unroll
            for (int i = 0; i < RV; ++i) {
                const int v = threadIdx.x + i * 256;
                if (v < nv) gv[i] = load4(a.gen_gain + 4 * v);
            }
        }
        load_row_pend<RV>(xv, x, a.pend + (size_t)r * a.d, a.pend_stride, a.npend, nv);
#pragma unroll
        for (int i = 0; i < RV; ++i) {
            const int v = threadIdx.x + i * 256;
            if (v < nv) {
                if (a.npend > 0) store4(x + 4 * v, xv[i]);
                ss += xv[i].x * xv[i].x + xv[i].y * xv[i].y + xv[i].z * xv[i].z + xv[i].w * xv[i].w;
            }
        }
        const float inv = rsqrtf(block_sum(ss, red) / (float)a.d + a.eps);
        if (emb_row && threadIdx.x == 0) a.inv_rms[r] = inv;
        const int hr = emb_row && a.hid_rows ? a.hid_rows[r] : -1;
        if (emb_row && hr < 0) return;
        if (emb_row) {
#pragma unroll
            for (int i = 0; i < RV; ++i) {
                const int v = threadIdx.x + i * 256;
                if (v < nv) gv[i] = load4(a.gain + 4 * v);
            }
        }
#pragma unroll
        for (int i = 0; i < RV; ++i) {
            const int v = threadIdx.x + i * 256;
            if (v < nv) {
                const float4 g = gv[i];
                const float4 o{xv[i].x * inv * g.x, xv[i].y * inv * g.y, xv[i].z * inv * g.z, xv[i].w * inv * g.w};
                if (emb_row) store4(a.hidden + (size_t)hr * a.d + 4 * v, o);
                else store4((T *)a.act + (size_t)lm * a.d + 4 * v, o);
            }
        }
        return;
    }
    for (int v = threadIdx.x; v < nv; v += 256) {
        float4 q = load4(x + 4 * v);
        if (a.npend > 0) {
            // finish the last layer's split-K residual add (slabs in order)
            for (int sp = 0; sp < a.npend; ++sp) {
                const float4 p = load4(a.pend + sp * a.pend_stride + (size_t)r * a.d + 4 * v);
                q = float4{q.x + p.x, q.y + p.y, q.z + p.z, q.w + p.w};
            }
            store4(x + 4 * v, q);
        }
        ss += q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
    }
    const float inv = rsqrtf(block_sum(ss, red) / (float)a.d + a.eps);
    if (emb_row) {
        if (threadIdx.x == 0) a.inv_rms[r] = inv;
        const int hr = a.hid_rows ? a.hid_rows[r] : -1;
        if (hr >= 0) {
            float *h = a.hidden + (size_t)hr * a.d;
            for (int v = threadIdx.x; v < nv; v += 256) {
                const float4 q = load4(x + 4 * v), g = load4(a.gain + 4 * v);
                store4(h + 4 * v, float4{q.x * inv * g.x, q.y * inv * g.y, q.z * inv * g.z, q.w * inv * g.w});
            }
        }
        return;
    }
    T *y = (T *)a.act + (size_t)lm * a.d;
    for (int v = threadIdx.x; v < nv; v += 256) {
        const float4 q = load4(x + 4 * v), g = load4(a.gen_gain + 4 * v);
        store4(y + 4 * v, float4{q.x * inv * g.x, q.y * inv * g.y, q.z * inv * g.z, q.w * inv * g.w});
    }
}

template <typename T, int RV>
__global__ __launch_bounds__(256) void final_rows_kernel(PoolArgs a) {
    __shared__ float red[4];
    final_row_block<T, RV>(a, blockIdx.x, red);
}

__device__ __forceinline__ bool chunk_state_ok(const int32_t *ch, const float *acc_w) {
    const int seq = ch[0], off = ch[1];
    return off == 0 || acc_w[seq] == (float)off;
}

// S update of Eq. (1) for mean (w = 1) and weighted-mean pooling.  Block = 64 columns x 4 row
// slices; grid = (chunks, d / 64).  Needs the final-norm scales of the chunk's rows
// (final_rows_kernel).
__global__ __launch_bounds__(256) void pool_accum_kernel(PoolArgs a) {
    __shared__ float part[4][64];
    const int ci = blockIdx.x;
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], len = ch[2], flags = ch[3], t0 = ch[4];
    const int pool = (flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK;
    // single-row heads are done by pool_rows_kernel; buffered rows need no S
    if (pool != ORTHRUS_POOL_MEAN && pool != ORTHRUS_POOL_WMEAN) return;
    const float *w = pool == ORTHRUS_POOL_WMEAN ? a.weights + t0 : nullptr;
    if (!chunk_state_ok(ch, a.acc_w)) {
        if (blockIdx.y == 0 && threadIdx.x == 0) flag_error(a.err, ORTHRUS_DEVERR_ACC);
        return;
    }
    const int c = blockIdx.y * 64 + (threadIdx.x & 63), slice = threadIdx.x >> 6;
    const float gc = a.gain[c];
    float *S = a.acc_sum + (size_t)seq * a.d + c;
    float s = 0.f;
    if (w) {
        for (int r = slice; r < len; r += 4) s += a.x[(size_t)(t0 + r) * a.d + c] * (a.inv_rms[t0 + r] * w[r]);
    } else {
        for (int r = slice; r < len; r += 4) s += a.x[(size_t)(t0 + r) * a.d + c] * a.inv_rms[t0 + r];
    }
    part[slice][threadIdx.x & 63] = s;
    __syncthreads();
    if (slice == 0) {
        const float tot = ((part[0][c & 63] + part[1][c & 63]) + part[2][c & 63]) + part[3][c & 63];
        *S = (off == 0 ? 0.f : *S) + tot * gc;
    }
}

// Token count W (Eq. (2) for w = 1; the offset check for every head) and, for a request's final
// chunk, v / max(||v||, 1e-12) with v = S / W (mean) or S (weighted mean: the weight sum of
// Eq. (2) cancels in the L2 finish).  Buffered chunks only advance W (and flag a state mismatch).
__global__ __launch_bounds__(256) void pool_finish_kernel(PoolArgs a) {
    __shared__ float red[4];
    const int ci = blockIdx.x;
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], len = ch[2], flags = ch[3];
    const int pool = (flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK;
    if (pool != ORTHRUS_POOL_MEAN && pool != ORTHRUS_POOL_WMEAN && pool != ORTHRUS_POOL_BUFFER) return;
    const bool ok = chunk_state_ok(ch, a.acc_w);
    if (!ok && pool == ORTHRUS_POOL_BUFFER && threadIdx.x == 0) flag_error(a.err, ORTHRUS_DEVERR_ACC);
    __syncthreads();
    if (!ok) return;
    const float W = (off == 0 ? 0.f : a.acc_w[seq]) + (float)len;
    __syncthreads();  // every thread has read the old W
    if (threadIdx.x == 0) a.acc_w[seq] = W;
    if (!(flags & ORTHRUS_CHUNK_LAST) || pool == ORTHRUS_POOL_BUFFER) return;
    const float *S = a.acc_sum + (size_t)seq * a.d;
    const float div = pool == ORTHRUS_POOL_MEAN ? W : 1.f;
    float ss = 0.f;
    for (int i = threadIdx.x; i < a.d; i += 256) {
        const float v = S[i] / div;
        ss += v * v;
    }
    const float nrm = sqrtf(block_sum(ss, red));
    const float inv = 1.f / fmaxf(nrm, 1e-12f);
    float *out = a.out_emb + (size_t)ci * a.d;
    for (int i = threadIdx.x; i < a.d; i += 256) out[i] = (S[i] / div) * inv;
}

// Single-row heads (last token, CLS): one block per chunk does the whole update.  The pooled
// row (the chunk's last row on its request's final chunk; row 0 of a request's first chunk)
// gets its final RMSNorm here (after the pending split-K slabs, if any), S of Eq. (1) takes
// that row (last: an offset-0 chunk without it clears S), W of Eq. (2) grows by the chunk
// length, and a final chunk writes S / max(||S||, 1e-12).
__device__ void pool_rows_block(const PoolArgs &a, int ci, float *red) {
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], len = ch[2], flags = ch[3], t0 = ch[4];
    const int pool = (flags >> ORTHRUS_POOL_SHIFT) & ORTHRUS_POOL_MASK;
    const bool last = flags & ORTHRUS_CHUNK_LAST;
    if (pool != ORTHRUS_POOL_LAST && pool != ORTHRUS_POOL_CLS) return;
    const float w_old = a.acc_w[seq];
    if (!(off == 0 || w_old == (float)off)) {
        if (threadIdx.x == 0) flag_error(a.err, ORTHRUS_DEVERR_ACC);
        return;
    }
    const int r = pool == ORTHRUS_POOL_LAST ? (last ? t0 + len - 1 : -1) : (off == 0 ? t0 : -1);
    float *S = a.acc_sum + (size_t)seq * a.d;
    const int nv = a.d / 4;
    if (r >= 0) {
        const float *xr = a.x + (size_t)r * a.d;
        auto row = [&](int v) {
            float4 q = load4(xr + 4 * v);
            for (int sp = 0; sp < a.npend; ++sp) {
                const float4 p = load4(a.pend + sp * a.pend_stride + (size_t)r * a.d + 4 * v);
                q = float4{q.x + p.x, q.y + p.y, q.z + p.z, q.w + p.w};
            }
            return q;
        };
        float ss = 0.f;
        for (int v = threadIdx.x; v < nv; v += 256) {
            const float4 q = row(v);
            ss += q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
        }
        const float inv = rsqrtf(block_sum(ss, red) / (float)a.d + a.eps);
        for (int v = threadIdx.x; v < nv; v += 256) {
            const float4 q = row(v), g = load4(a.gain + 4 * v);
            store4(S + 4 * v, float4{q.x * inv * g.x, q.y * inv * g.y, q.z * inv * g.z, q.w * inv * g.w});
        }
    } else if (pool == ORTHRUS_POOL_LAST && off == 0) {
        for (int v = threadIdx.x; v < nv; v += 256) store4(S + 4 * v, float4{0.f, 0.f, 0.f, 0.f});
    }
    __syncthreads();  // S complete; every thread has read the old W
    if (threadIdx.x == 0) a.acc_w[seq] = (off == 0 ? 0.f : w_old) + (float)len;
    if (!last) return;
    float nn = 0.f;
    for (int v = threadIdx.x; v < nv; v += 256) {
        const float4 q = load4(S + 4 * v);
        nn += q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
    }
    const float sc = 1.f / fmaxf(sqrtf(block_sum(nn, red)), 1e-12f);
    float *out = a.out_emb + (size_t)ci * a.d;
    for (int v = threadIdx.x; v < nv; v += 256) {
        const float4 q = load4(S + 4 * v);
        store4(out + 4 * v, float4{q.x * sc, q.y * sc, q.z * sc, q.w * sc});
    }
}

__global__ __launch_bounds__(256) void pool_rows_kernel(PoolArgs a) {
    __shared__ float red[4];
    pool_rows_block(a, blockIdx.x, red);
}

// With no head that needs every embedding row's norm, the final norm of the rows that get
// logits and the single-row pooler are independent: one launch, blocks [0, n_lm) normalise the
// LM rows, the following n_chunks blocks pool one chunk each.
template <typename T, int RV>
__global__ __launch_bounds__(256) void final_and_pool_rows_kernel(PoolArgs a) {
    __shared__ float red[4];
    if ((int)blockIdx.x < a.n_lm) final_row_block<T, RV>(a, blockIdx.x, red);
    else pool_rows_block(a, (int)blockIdx.x - a.n_lm, red);
}

// ------------------------------------------------------------------------- greedy sampler
// (v, i) beats (bv, bi) when it comes first in "NaN greatest, then larger value, then lower index"
__device__ __forceinline__ bool argmax_better(float v, int i, float bv, int bi) {
    const bool vn = v != v, bn = bv != bv;
    if (vn || bn) return vn && (!bn || i < bi);
    return v > bv || (v == bv && i < bi);
}

// One block per row; each thread scans a strided slice (16-byte loads when the row allows),
// then the block reduces its 256 candidates.  The result does not depend on the scan order.
__global__ __launch_bounds__(256) void argmax_kernel(const float *logits, int vocab, int32_t *out) {
    __shared__ float bvs[4];
    __shared__ int bis[4];
    const float *row = logits + (size_t)blockIdx.x * vocab;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    const bool vec = (vocab % 4 == 0) && ((uintptr_t)logits % 16 == 0);
    if (vec) {
        for (int v = threadIdx.x; v < vocab / 4; v += 256) {
            const float4 q = load4(row + 4 * v);
            if (argmax_better(q.x, 4 * v, bv, bi)) bv = q.x, bi = 4 * v;
            if (argmax_better(q.y, 4 * v + 1, bv, bi)) bv = q.y, bi = 4 * v + 1;
            if (argmax_better(q.z, 4 * v + 2, bv, bi)) bv = q.z, bi = 4 * v + 2;
            if (argmax_better(q.w, 4 * v + 3, bv, bi)) bv = q.w, bi = 4 * v + 3;
        }
    } else {
        for (int v = threadIdx.x; v < vocab; v += 256)
            if (argmax_better(row[v], v, bv, bi)) bv = row[v], bi = v;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (argmax_better(ov, oi, bv, bi)) bv = ov, bi = oi;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) bvs[wave] = bv, bis[wave] = bi;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 4; ++w)
            if (argmax_better(bvs[w], bis[w], bv, bi)) bv = bvs[w], bi = bis[w];
        out[blockIdx.x] = bi;
    }
}

}  // namespace

hipError_t launch_argmax(const float *logits, int rows, int vocab, int32_t *out, hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(argmax_kernel, dim3(rows), dim3(256), 0, s, logits, vocab, out);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, bool gather, const NormArgs &a, hipStream_t s) {
    if (a.rows <= 0) return hipSuccess;
    if (a.npend < 0 || a.npend > kMaxPend) return hipErrorInvalidValue;
    const bool rv4 = a.d <= 4096;
    auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(a.rows), dim3(256), 0, s, a); };
    if (dtype == 1) {
        if (gather) rv4 ? go(rmsnorm_kernel<bf16, true, 4>) : go(rmsnorm_kernel<bf16, true, 8>);
        else rv4 ? go(rmsnorm_kernel<bf16, false, 4>) : go(rmsnorm_kernel<bf16, false, 8>);
    } else {
        if (gather) rv4 ? go(rmsnorm_kernel<float, true, 4>) : go(rmsnorm_kernel<float, true, 8>);
        else rv4 ? go(rmsnorm_kernel<float, false, 4>) : go(rmsnorm_kernel<float, false, 8>);
    }
    return hipGetLastError();
}

hipError_t launch_rope_append(int dtype, const RopeArgs &a, hipStream_t s) {
    if (a.T <= 0) return hipSuccess;
    if (dtype == 1 && a.cs && a.T > 256) {
        if (a.page != 16 || a.hd % 8 || a.hd > 128) return hipErrorInvalidValue;
        const dim3 grid((a.T + kRopeGroup - 1) / kRopeGroup, a.nq + 2 * a.nkv);
        hipLaunchKernelGGL(rope_append_group_kernel, grid, dim3(256), 0, s, a);
        return hipGetLastError();
    }
    // enough blocks per token to spread its work items over the CUs (at least 4 x 256 blocks)
    const int items = (a.nq + a.nkv) * (a.hd / 8) + a.nkv * a.hd / 4;
    const int per_tok = std::max(1, std::min((items + 255) / 256, (1024 + a.T - 1) / std::max(a.T, 1)));
    const dim3 grid(a.T, per_tok);
    if (dtype == 1) hipLaunchKernelGGL(rope_append_kernel<bf16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(rope_append_kernel<float>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_final_rows(int dtype, const PoolArgs &a, hipStream_t s) {
    const int rows = a.n_emb_rows + a.n_lm;
    if (rows <= 0) return hipSuccess;
    if (a.npend < 0 || a.npend > kMaxPend) return hipErrorInvalidValue;
    const bool rv4 = a.d <= 4096;
    auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, a); };
    if (dtype == 1) rv4 ? go(final_rows_kernel<bf16, 4>) : go(final_rows_kernel<bf16, 8>);
    else rv4 ? go(final_rows_kernel<float, 4>) : go(final_rows_kernel<float, 8>);
    return hipGetLastError();
}

hipError_t launch_final_and_pool(int dtype, const PoolArgs &a, hipStream_t s) {
    if (a.n_emb_rows != 0) return hipErrorInvalidValue;
    if (a.npend < 0 || a.npend > kMaxPend) return hipErrorInvalidValue;
    const int blocks = a.n_lm + a.n_chunks;
    if (blocks <= 0) return hipSuccess;
    const bool rv4 = a.d <= 4096;
    auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, s, a); };
    if (dtype == 1) rv4 ? go(final_and_pool_rows_kernel<bf16, 4>) : go(final_and_pool_rows_kernel<bf16, 8>);
    else rv4 ? go(final_and_pool_rows_kernel<float, 4>) : go(final_and_pool_rows_kernel<float, 8>);
    return hipGetLastError();
}

hipError_t launch_pool(const PoolArgs &a, bool any_rows, hipStream_t s) {
    if (a.n_chunks <= 0) return hipSuccess;
    hipLaunchKernelGGL(pool_rows_kernel, dim3(a.n_chunks), dim3(256), 0, s, a);
    if (any_rows) {
        hipLaunchKernelGGL(pool_accum_kernel, dim3(a.n_chunks, a.d / 64), dim3(256), 0, s, a);
        hipLaunchKernelGGL(pool_finish_kernel, dim3(a.n_chunks), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace orthrus
