// Ragged attention over the mixed batch in one launch (Section 3.2: every batch item goes
// through the same attention layer, differing only in length).
//
// The host planner emits a work list; block b runs item b:
//   * prefill items (embedding-chunk rows, heaviest first): a tile of (128 / group) tokens of
//     one chunk times the `group` query heads of one KV head.  Rows attend causally to every
//     key of their request at positions <= their own: earlier chunks' keys from the paged
//     cache plus this chunk's keys, which the step appended before this launch.
//     bf16: each wave owns 32 query rows of one head; S^T = K Q^T and O^T += V^T P^T run on
//     v_mfma_f32_32x32x16_bf16 over 32-key blocks staged in LDS (V transposed on the way in),
//     with an online softmax in fp32 (exp2 domain).
//   * decode items: one (decode row, KV head, 256-key split).  All `group` query heads that
//     share the KV head are served from one read of each 4 KiB K / V page slice.  Scores go to
//     LDS, the softmax is taken over the split, then P V is accumulated.  Rows with more than
//     one split write (max, sum, unnormalised output) partials that attn_combine merges in
//     split order, so results do not depend on scheduling.
// Page ids read from the block table are range-checked; a bad id sets the sticky device error
// word and its keys are skipped (never dereferenced).
#include "common.hpp"
#include "plan.hpp"

namespace orthrus {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

struct PoolView {
    const char *k, *v;
    const int32_t *bt;
    int n_pages, max_blocks;
};

__device__ __forceinline__ PoolView pool_view(const AttnArgs &a, int p, size_t elem) {
    (void)elem;
    PoolView pv;
    pv.k = (const char *)a.k_cache[p];
    pv.v = (const char *)a.v_cache[p];
    pv.bt = a.block_table[p];
    pv.n_pages = a.n_pages[p];
    pv.max_blocks = a.max_blocks[p];
    return pv;
}

// ----------------------------------------------------------------------------- decode split
template <typename T, int HD, int G>
__device__ void decode_item(const AttnArgs &a, const int32_t *it, char *smem) {
    constexpr int DPL = HD / 4;    // dims per lane in the score pass (4 lanes per key)
    constexpr int VPL = HD / 16;   // dims per lane in the value pass (16 lanes per key)
    constexpr int MAXK = kSplitPages * 16;
    float *sc = (float *)smem;                         // [MAXK][G] scores, then weights
    float *red = sc + MAXK * G;                        // [4][2 * G] cross-wave reductions
    float *part = red + 8 * G;                         // [16 key groups][16 lanes][G][VPL]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = it[IT_INDEX], g = it[IT_KVHEAD];
    const int k0 = it[IT_KEY_BEGIN], k1 = it[IT_KEY_END], pslot = it[IT_PARTIAL];
    const int nk = k1 - k0;
    const int P = a.page;
    const int32_t *row = a.rows + kRowInts * j;
    const int seq = row[0], tok = row[2];
    const PoolView pv = pool_view(a, 1, sizeof(T));
    const int32_t *bt = pv.bt + (size_t)seq * pv.max_blocks + k0 / P;
    const int n_pg = (nk + P - 1) / P;
    const size_t page_elems = (size_t)a.nkv * P * HD;
    const float scale = kLog2e / sqrtf((float)HD);

    // ---- scores: lane = (key in page, quarter of the head dims)
    const int kin = lane >> 2, qtr = lane & 3;
    const T *qrow = (const T *)a.q + ((size_t)tok * a.nq + g * G) * HD + qtr * DPL;
    float q[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < DPL; ++e) q[h][e] = to_f32(qrow[h * HD + e]);
    for (int pg = wave; pg < n_pg; pg += 4) {
        const int page = bt[pg];
        const bool ok = page >= 0 && page < pv.n_pages;
        if (!ok && lane == 0) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
        const int key = pg * P + kin;  // relative to k0
        float s[G];
#pragma unroll
        for (int h = 0; h < G; ++h) s[h] = 0.f;
        if (ok && key < nk) {
            const T *kp = (const T *)pv.k + (size_t)page * page_elems + ((size_t)g * P + kin) * HD + qtr * DPL;
            if constexpr (sizeof(T) == 2) {
                const u32x4 *k4 = (const u32x4 *)kp;
#pragma unroll
                for (int c = 0; c < DPL / 8; ++c) {
                    const u32x4 kv = k4[c];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float klo = bf16_lo(kv[e]), khi = bf16_hi(kv[e]);
#pragma unroll
                        for (int h = 0; h < G; ++h)
                            s[h] = fmaf(q[h][c * 8 + 2 * e + 1], khi, fmaf(q[h][c * 8 + 2 * e], klo, s[h]));
                    }
                }
            } else {
                const f32x4 *k4 = (const f32x4 *)kp;
#pragma unroll
                for (int c = 0; c < DPL / 4; ++c) {
                    const f32x4 kv = k4[c];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int h = 0; h < G; ++h) s[h] = fmaf(q[h][c * 4 + e], kv[e], s[h]);
                }
            }
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
            s[h] += __shfl_xor(s[h], 1, 64);
            s[h] += __shfl_xor(s[h], 2, 64);
        }
        if (qtr == 0 && key < nk) {
#pragma unroll
            for (int h = 0; h < G; ++h) sc[key * G + h] = ok ? s[h] * scale : -INFINITY;
        }
    }
    __syncthreads();

    // ---- softmax statistics over the split (one key per thread)
    float v[G], m[G], l[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        v[h] = tid < nk ? sc[tid * G + h] : -INFINITY;
        const float wm = wave_max(v[h]);
        if (lane == 0) red[wave * 2 * G + h] = wm;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = fmaxf(fmaxf(red[h], red[2 * G + h]), fmaxf(red[4 * G + h], red[6 * G + h]));
        const float pv_ = (tid < nk && m[h] != -INFINITY) ? exp2f(v[h] - m[h]) : 0.f;
        if (tid < nk) sc[tid * G + h] = pv_;
        const float ws = wave_sum(pv_);
        if (lane == 0) red[wave * 2 * G + G + h] = ws;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) l[h] = red[G + h] + red[3 * G + h] + red[5 * G + h] + red[7 * G + h];

    // ---- P V: a page per step, wave w takes keys 4w..4w+3 of it, 16 lanes per key
    const int kq = lane >> 4, dl = lane & 15;
    float acc[G][VPL];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < VPL; ++e) acc[h][e] = 0.f;
    for (int pg = 0; pg < n_pg; ++pg) {
        const int page = bt[pg];
        const int kin2 = wave * 4 + kq;
        const int key = pg * P + kin2;
        if (page < 0 || page >= pv.n_pages || key >= nk) continue;
        const T *vp = (const T *)pv.v + (size_t)page * page_elems + ((size_t)g * P + kin2) * HD + dl * VPL;
        float w[G];
#pragma unroll
        for (int h = 0; h < G; ++h) w[h] = sc[key * G + h];
        float vv[VPL];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int c = 0; c < VPL / 2; ++c) {
                const uint32_t u = ((const uint32_t *)vp)[c];
                vv[2 * c] = bf16_lo(u);
                vv[2 * c + 1] = bf16_hi(u);
            }
        } else {
#pragma unroll
            for (int e = 0; e < VPL; ++e) vv[e] = to_f32(vp[e]);
        }
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int e = 0; e < VPL; ++e) acc[h][e] = fmaf(w[h], vv[e], acc[h][e]);
    }
    // cross key-group reduction in a fixed order
    float *mine = part + ((wave * 4 + kq) * 16 + dl) * G * VPL;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < VPL; ++e) mine[h * VPL + e] = acc[h][e];
    __syncthreads();
    for (int o = tid; o < G * HD; o += 256) {
        const int h = o / HD, d = o % HD;
        const int dlo = d / VPL, e = d % VPL;
        float sum = 0.f;
        for (int kg = 0; kg < 16; ++kg) sum += part[((kg * 16 + dlo) * G + h) * VPL + e];
        if (pslot < 0) {
            const float out = l[h] > 0.f ? sum / l[h] : 0.f;
            ((T *)a.o)[((size_t)tok * a.nq + g * G + h) * HD + d] = from_f32<T>(out);
        } else {
            float *pp = a.partials + ((size_t)pslot * G + h) * (HD + 2);
            if (d == 0) {
                pp[0] = m[h];
                pp[1] = l[h];
            }
            pp[2 + d] = sum;
        }
    }
}

// --------------------------------------------------------------- prefill, fp32 scalar path
template <typename T, int HD, int G>
__device__ void prefill_item_scalar(const AttnArgs &a, const int32_t *it) {
    const int tid = threadIdx.x;
    const int ci = it[IT_INDEX], g = it[IT_KVHEAD], qb = it[IT_A], qn = it[IT_B];
    if (tid >= qn * G) return;
    const int r = tid / G, h = g * G + tid % G;
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], tok = ch[4] + qb + r;
    const int qpos = off + qb + r;
    const PoolView pv = pool_view(a, 0, sizeof(T));
    const int P = a.page;
    const size_t page_elems = (size_t)a.nkv * P * HD;
    const T *qp = (const T *)a.q + ((size_t)tok * a.nq + h) * HD;
    float q[HD], acc[HD];
    const float scale = kLog2e / sqrtf((float)HD);
#pragma unroll
    for (int d = 0; d < HD; ++d) {
        q[d] = to_f32(qp[d]) * scale;
        acc[d] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    for (int kp = 0; kp <= qpos; ++kp) {
        const int page = pv.bt[(size_t)seq * pv.max_blocks + kp / P];
        if (page < 0 || page >= pv.n_pages) {
            flag_error(a.err, ORTHRUS_DEVERR_PAGE);
            continue;
        }
        const size_t base = (size_t)page * page_elems + ((size_t)g * P + kp % P) * HD;
        const T *kr = (const T *)pv.k + base;
        const T *vr = (const T *)pv.v + base;
        float s = 0.f;
#pragma unroll
        for (int d = 0; d < HD; ++d) s = fmaf(q[d], to_f32(kr[d]), s);
        const float mn = fmaxf(m, s);
        const float alpha = exp2f(m - mn), p = exp2f(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int d = 0; d < HD; ++d) acc[d] = fmaf(p, to_f32(vr[d]), acc[d] * alpha);
        m = mn;
    }
    T *op = (T *)a.o + ((size_t)tok * a.nq + h) * HD;
#pragma unroll
    for (int d = 0; d < HD; ++d) op[d] = from_f32<T>(l > 0.f ? acc[d] / l : 0.f);
}

// ------------------------------------------------------------------ prefill, bf16 MFMA path
template <int HD, int G>
__device__ void prefill_item_mfma(const AttnArgs &a, const int32_t *it, char *smem) {
    constexpr int KS = HD / 16;        // 16-wide k steps of S^T = K Q^T
    constexpr int DB = HD / 32;        // 32-row dim blocks of O^T
    constexpr int KROW = HD * 2 + 16;  // padded K row bytes in LDS
    constexpr int VROW = 32 * 2 + 8;   // padded V^T row bytes in LDS (32 keys)
    char *k_lds = smem;
    char *v_lds = smem + 32 * KROW;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ci = it[IT_INDEX], g = it[IT_KVHEAD], qb = it[IT_A], qn = it[IT_B], kend = it[IT_KEY_END];
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], tok0 = ch[4];
    const int h = g * G + (wave % G), sb = wave / G;
    const int col = lane & 31, half = lane >> 5;
    // this lane's query (clamped into the tile so padded rows stay finite)
    const int r = min(sb * 32 + col, qn - 1);
    const int tok = tok0 + qb + r;
    const int qpos = off + qb + r;
    const PoolView pv = pool_view(a, 0, 2);
    const int P = a.page;
    const size_t page_elems = (size_t)a.nkv * P * HD;

    bf16x8 qf[KS];
    const bf16 *qp = (const bf16 *)a.q + ((size_t)tok * a.nq + h) * HD;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = *(const bf16x8 *)(qp + kk * 16 + half * 8);

    f32x16 acc[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[d][e] = 0.f;
    float m = -INFINITY, l = 0.f;
    const float scale = kLog2e / sqrtf((float)HD);
    const int nkb = (kend + 31) / 32;

    for (int kb = 0; kb < nkb; ++kb) {
        // stage 32 keys: K rows as-is, V transposed to [dim][key]
        for (int c = tid; c < 32 * (HD / 8); c += 256) {
            const int key = c / (HD / 8), part = c % (HD / 8);
            const int kpos = kb * 32 + key;
            u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
            if (kpos < kend) {
                const int page = pv.bt[(size_t)seq * pv.max_blocks + kpos / P];
                if (page >= 0 && page < pv.n_pages) {
                    const size_t base = ((size_t)page * page_elems + ((size_t)g * P + kpos % P) * HD + part * 8) * 2;
                    kv = *(const u32x4 *)(pv.k + base);
                    vv = *(const u32x4 *)(pv.v + base);
                } else if (part == 0) {
                    flag_error(a.err, ORTHRUS_DEVERR_PAGE);
                }
            }
            *(u32x4 *)(k_lds + key * KROW + part * 16) = kv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                *(uint16_t *)(v_lds + (part * 8 + 2 * e) * VROW + key * 2) = (uint16_t)(vv[e] & 0xffffu);
                *(uint16_t *)(v_lds + (part * 8 + 2 * e + 1) * VROW + key * 2) = (uint16_t)(vv[e] >> 16);
            }
        }
        __syncthreads();

        // S^T[key][query] for this wave's 32 queries
        f32x16 s;
#pragma unroll
        for (int e = 0; e < 16; ++e) s[e] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            const bf16x8 kf = *(const bf16x8 *)(k_lds + col * KROW + (kk * 16 + half * 8) * 2);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s, 0, 0, 0);
        }
        // mask + online softmax (lane's query = col; keys of register e: 8*(e/4) + 4*half + e%4)
        float mloc = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int kpos = kb * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
            const bool vis = kpos <= qpos && kpos < kend;
            s[e] = vis ? s[e] * scale : -INFINITY;
            mloc = fmaxf(mloc, s[e]);
        }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
        const float mn = fmaxf(m, mloc);
        const float alpha = (m == -INFINITY) ? 0.f : exp2f(m - mn);
        float psum = 0.f;
        bf16x8 pf[2];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const float p = (mn == -INFINITY) ? 0.f : exp2f(s[e] - mn);
            psum += p;
            pf[e >> 3][e & 7] = from_f32<bf16>(p);
        }
        psum += __shfl_xor(psum, 32, 64);
        l = l * alpha + psum;
        m = mn;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[d][e] *= alpha;
        // O^T[dim][query] += V^T[dim][keys] P^T[keys][query], two 16-key steps
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                const char *vr = v_lds + (d * 32 + col) * VROW;
                const uint64_t lo = *(const uint64_t *)(vr + (k2 * 16 + half * 4) * 2);
                const uint64_t hi = *(const uint64_t *)(vr + (k2 * 16 + 8 + half * 4) * 2);
                u32x4 vu = {(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)};
                acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vu), pf[k2], acc[d], 0, 0, 0);
            }
        }
        __syncthreads();
    }
    if (sb * 32 + col >= qn) return;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    bf16 *op = (bf16 *)a.o + ((size_t)tok * a.nq + h) * HD;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const int dim = d * 32 + q4 * 8 + half * 4;
            const uint32_t w0 = pack_bf16x2(acc[d][q4 * 4 + 0] * inv, acc[d][q4 * 4 + 1] * inv);
            const uint32_t w1 = pack_bf16x2(acc[d][q4 * 4 + 2] * inv, acc[d][q4 * 4 + 3] * inv);
            *(uint64_t *)(op + dim) = (uint64_t)w0 | ((uint64_t)w1 << 32);
        }
}

template <typename T, int HD, int G>
constexpr size_t attn_smem() {
    constexpr size_t dec = (kSplitPages * 16 * G + 8 * G + 16 * 16 * G * (HD / 16)) * sizeof(float);
    constexpr size_t pre = sizeof(T) == 2 ? 32 * (HD * 2 + 16) + HD * (32 * 2 + 8) : 0;
    return dec > pre ? dec : pre;
}

template <typename T, int HD, int G>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[attn_smem<T, HD, G>()];
    const int32_t *it = a.items + kItemInts * blockIdx.x;
    if (it[IT_KIND] == 0) {
        if constexpr (sizeof(T) == 2) prefill_item_mfma<HD, G>(a, it, smem);
        else prefill_item_scalar<T, HD, G>(a, it);
    } else {
        decode_item<T, HD, G>(a, it, smem);
    }
}

template <typename T, int HD, int G>
__global__ __launch_bounds__(HD) void attn_combine_kernel(AttnArgs a) {
    const int j = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
    const int32_t *row = a.rows + kRowInts * j;
    const int nsplit = row[3], base = row[4], tok = row[2];
    if (nsplit <= 1) return;
    const int g = h / G, hl = h % G;
    float M = -INFINITY;
    for (int s = 0; s < nsplit; ++s)
        M = fmaxf(M, a.partials[((size_t)(base + g * nsplit + s) * G + hl) * (HD + 2)]);
    float L = 0.f, acc = 0.f;
    for (int s = 0; s < nsplit; ++s) {
        const float *pp = a.partials + ((size_t)(base + g * nsplit + s) * G + hl) * (HD + 2);
        const float w = (pp[0] == -INFINITY) ? 0.f : exp2f(pp[0] - M);
        L += pp[1] * w;
        acc += pp[2 + d] * w;
    }
    ((T *)a.o)[((size_t)tok * a.nq + h) * HD + d] = from_f32<T>(L > 0.f ? acc / L : 0.f);
}

template <typename T, int HD, int G>
hipError_t run_attn(const AttnArgs &a, hipStream_t s) {
    if (a.n_items <= 0) return hipSuccess;
    hipLaunchKernelGGL((attn_kernel<T, HD, G>), dim3(a.n_items), dim3(256), 0, s, a);
    return hipGetLastError();
}
template <typename T, int HD, int G>
hipError_t run_combine(const AttnArgs &a, int n_decode, hipStream_t s) {
    if (n_decode <= 0) return hipSuccess;
    hipLaunchKernelGGL((attn_combine_kernel<T, HD, G>), dim3(n_decode, a.nq), dim3(HD), 0, s, a);
    return hipGetLastError();
}

template <typename T>
hipError_t dispatch(const AttnArgs &a, int n_decode, bool combine, hipStream_t s) {
    const int G = a.nq / a.nkv;
#define ORTHRUS_ATTN_CASE(HDV, GV)                                                         \
    if (a.hd == HDV && G == GV)                                                            \
        return combine ? run_combine<T, HDV, GV>(a, n_decode, s) : run_attn<T, HDV, GV>(a, s);
    ORTHRUS_ATTN_CASE(128, 4)
    ORTHRUS_ATTN_CASE(128, 2)
    ORTHRUS_ATTN_CASE(128, 1)
    ORTHRUS_ATTN_CASE(64, 4)
    ORTHRUS_ATTN_CASE(64, 2)
    ORTHRUS_ATTN_CASE(64, 1)
#undef ORTHRUS_ATTN_CASE
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t s) {
    return dtype == 1 ? dispatch<bf16>(a, 0, false, s) : dispatch<float>(a, 0, false, s);
}

hipError_t launch_attn_combine(int dtype, const AttnArgs &a, int n_decode, hipStream_t s) {
    return dtype == 1 ? dispatch<bf16>(a, n_decode, true, s) : dispatch<float>(a, n_decode, true, s);
}

}  // namespace orthrus
