// Ragged attention over the mixed batch in one launch (Section 3.2: every batch item goes
// through the same attention layer, differing only in length).
//
// Cache layout (one page = 16 positions of one KV head): keys key-major [16][hd], values
// dim-major [hd][16].  Both MFMA operands of a 32x32x16 step then read 16 contiguous bytes per
// lane (a key row for S^T = K Q^T, a value row over 8 positions for O^T = V^T P^T), and the
// decode dot products pair adjacent dims (q.k) or adjacent positions (p.v) without shuffles.
//
// The host planner emits a work list; block b runs item b:
//   * prefill items (rows of embedding and generation prefill chunks, heaviest first; each
//     chunk reads the cache of its own model): (128 / group) tokens of one chunk
//     times the `group` query heads of one KV head; each wave owns 32 query rows of one head
//     and walks the keys of its request in 64-key blocks that the workgroup copies straight
//     into LDS (two buffers, one barrier per block; the block is shared by the group's waves),
//     with an online softmax in fp32 (exp2 domain) and causal masking on the diagonal blocks; a
//     wave past its causal bound skips the block's arithmetic.  A tile over a long cached
//     prefix comes as several items, one per run of keys (the walk is serial, so one long tile
//     would otherwise set the launch's length); those write partials like split decode rows,
//     merged by attn_combine.
//   * decode items: one (decode row, KV head, key-range split), walked in 128-key chunks (64
//     in the decode-only kernel).  Each wave owns two pages of a chunk (one), scores with
//     v_dot2_f32_bf16 for all `group` query heads at once, keeps an online softmax, and
//     accumulates P V from registers; the next chunk's K and V loads are in flight while a
//     chunk is computed.  Rows with several splits write (max, sum, unnormalised output)
//     partials merged by attn_combine in split order, so results do not depend on scheduling.
// Page ids read from the block table are range-checked; a bad id sets the sticky device error
// word and its keys are skipped (never dereferenced).
#include "common.hpp"
#include "plan.hpp"

namespace orthrus {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kPage = 16;
constexpr int kPrefillPageWindow = 512;  // page ids staged in LDS at a time (even)
constexpr int kDecodeChunkPages = 8;     // pages per step of a bf16 decode item (4 waves x 2)

struct PoolView {
    const char *k, *v;
    const int32_t *bt;
    int n_pages, max_blocks;
};

// cache of pool p (0: embedding model's, 1: generator's); selects, not an indexed load, so a
// run-time p keeps the kernel arguments in scalar registers
__device__ __forceinline__ PoolView pool_view(const AttnArgs &a, int p) {
    PoolView pv;
    pv.k = (const char *)(p ? a.k_cache[1] : a.k_cache[0]);
    pv.v = (const char *)(p ? a.v_cache[1] : a.v_cache[0]);
    pv.bt = p ? a.block_table[1] : a.block_table[0];
    pv.n_pages = p ? a.n_pages[1] : a.n_pages[0];
    pv.max_blocks = p ? a.max_blocks[1] : a.max_blocks[0];
    return pv;
}
// prefill chunks of the generator (prompt chunks) read its cache
__device__ __forceinline__ int chunk_pool(const int32_t *ch) { return (ch[3] & kChunkGen) ? 1 : 0; }

// Cross-lane partners without LDS permutes (each an exact copy of another lane's value):
//   quad_xor1 / quad_xor2: lane ^ 1 / lane ^ 2 (DPP quad permutations);
//   half_mirror: lane 7 - i within each 8 lanes, mirror: lane 15 - i within each 16 lanes (DPP);
//   with_partner16 / with_partner32: this lane's value and that of the same lane in the paired
//   16-lane row (lane ^ 16) or wave half (lane ^ 32), via v_permlane16_swap / v_permlane32_swap,
//   whose pair of results holds both values (in an order that depends on the lane).
// For a value equal across each quad (or each 8 or 16 lanes), a mirror partner is the xor
// partner's equal, so reductions over lanes give the same results as with xor shuffles.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float quad_xor1(float v) { return dpp_mov<0xB1>(v); }
__device__ __forceinline__ float quad_xor2(float v) { return dpp_mov<0x4E>(v); }
__device__ __forceinline__ float half_mirror(float v) { return dpp_mov<0x141>(v); }
__device__ __forceinline__ float mirror(float v) { return dpp_mov<0x140>(v); }
__device__ __forceinline__ float2 with_partner16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return float2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ float2 with_partner32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return float2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
// maximum and sum over the 16 quads of the wave of a value equal within each quad
__device__ __forceinline__ float quads_max(float v) {
    v = fmaxf(v, half_mirror(v));
    v = fmaxf(v, mirror(v));
    float2 p = with_partner16(v);
    v = fmaxf(p.x, p.y);
    p = with_partner32(v);
    return fmaxf(p.x, p.y);
}
__device__ __forceinline__ float quads_sum(float v) {
    v += half_mirror(v);
    v += mirror(v);
    float2 p = with_partner16(v);
    v = p.x + p.y;
    p = with_partner32(v);
    return p.x + p.y;
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c,
                                           false);
}

// ------------------------------------------------------------------ decode split, bf16 path
// A split is walked in chunks of CP pages (kDecodeChunkPages = 8 pages, 128 keys, in the combined
// kernel; 4 in the decode-only kernel); each wave owns CP / 4 pages of a chunk.  Loads are branch-free (invalid or absent pages read page 0 and are masked) and
// software-pipelined across chunks: the next chunk's K lines go out as soon as this chunk's
// scores are taken, its V lines as soon as this chunk's P V is done, and page ids two chunks
// ahead, so the memory pipe stays busy while the wave computes.  Each wave keeps an online
// softmax (max, sum, output) over its keys of all chunks; the four waves merge once at the end.
template <int HD, int G, int CP = kDecodeChunkPages>
__device__ void decode_item_bf16(const AttnArgs &a, const int32_t *it, char *smem) {
    constexpr int KL = HD / 32;     // 16-byte loads per lane per page, for K and for V
    constexpr int QD = HD / 4;      // head dims per lane in the score pass (4 lanes per key)
    constexpr int VD = HD / 64;     // head dims per lane in the value pass
    constexpr int PPW = CP / 4;                            // pages per wave per chunk
    constexpr int KPW = PPW * kPage;                       // keys per wave per chunk
    constexpr int CHUNK = CP * kPage;                      // keys per chunk
    uint32_t *pk_all = (uint32_t *)smem;                   // [4 waves][KPW / 2][G] bf16 weight pairs
    float *mw = (float *)(pk_all + 4 * (KPW / 2) * G);     // [4][G] wave maxima
    float *lw = mw + 4 * G;                                // [4][G] wave sums
    float *part = lw + 4 * G;                              // [4][G][HD] wave outputs
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    uint32_t *qs = (uint32_t *)(part + 4 * G * HD) + wave * (G * HD / 2);  // wave's copy of q
    const int j = it[IT_INDEX], g = it[IT_KVHEAD];
    const int k0 = it[IT_KEY_BEGIN], k1 = it[IT_KEY_END], pslot = it[IT_PARTIAL];
    const int nk = k1 - k0;
    const int n_pg = (nk + kPage - 1) / kPage;
    const int n_ch = (n_pg + CP - 1) / CP;
    const int32_t *row = a.rows + kRowInts * j;
    const int seq = row[0], tok = row[2];
    const PoolView pv = pool_view(a, 1);
    const int32_t *bt = pv.bt + (size_t)seq * pv.max_blocks + k0 / kPage;
    const size_t page_bytes = (size_t)a.nkv * kPage * HD * 2;
    const int kin = lane >> 2, qtr = lane & 3;

    // page ids of chunk c for this wave (pages c * CP + wave + 4 i), raw
    auto load_pages = [&](int c, int (&pg)[PPW]) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) pg[i] = bt[min(c * CP + wave + 4 * i, n_pg - 1)];
    };
    // range check: absent pages (past the split) and bad ids read page 0 and are masked later
    auto check_pages = [&](int c, int (&pg)[PPW], bool (&ok)[PPW]) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const bool present = c * CP + wave + 4 * i < n_pg;
            ok[i] = present && pg[i] >= 0 && pg[i] < pv.n_pages;
            if (present && !ok[i] && lane == 0) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
            pg[i] = ok[i] ? pg[i] : 0;
        }
    };
    u32x4 kr[PPW][KL], vr[PPW][KL];
    auto issue_k = [&](const int (&pg)[PPW]) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const char *kp = pv.k + pg[i] * page_bytes + (size_t)((g * kPage + kin) * HD + qtr * QD) * 2;
#pragma unroll
            for (int c = 0; c < KL; ++c) kr[i][c] = *(const u32x4 *)(kp + 16 * c);
        }
    };
    auto issue_v = [&](const int (&pg)[PPW]) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const char *vp = pv.v + pg[i] * page_bytes + (size_t)((g * HD + lane * VD) * kPage) * 2;
#pragma unroll
            for (int c = 0; c < KL; ++c) vr[i][c] = *(const u32x4 *)(vp + 16 * c);
        }
    };

    int pg_cur[PPW], pg_nxt[PPW];
    bool ok_cur[PPW], ok_nxt[PPW];
    load_pages(0, pg_cur);
    // query heads g*G .. g*G+G-1 (G*HD bf16, contiguous) into the wave's LDS copy, 16 bytes a lane;
    // the score pass reads one head's quarter at a time from there
    {
        const char *qrow = (const char *)a.q + ((size_t)tok * a.nq + g * G) * HD * 2;
#pragma unroll
        for (int c = 0; c < (G * HD * 2 + 1023) / 1024; ++c) {
            const int byte = (c * 64 + lane) * 16;
            if (byte < G * HD * 2) *(u32x4 *)((char *)qs + byte) = *(const u32x4 *)(qrow + byte);
        }
    }
    check_pages(0, pg_cur, ok_cur);
    issue_k(pg_cur);
    load_pages(1, pg_nxt);
    issue_v(pg_cur);

    const float scale = kLog2e / sqrtf((float)HD);
    float m[G], l[G], acc[G][VD];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int d = 0; d < VD; ++d) acc[h][d] = 0.f;
    }
    uint16_t *pk16 = (uint16_t *)(pk_all + wave * (KPW / 2) * G);
    const uint32_t *pkw = pk_all + wave * (KPW / 2) * G;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int c = 0; c < n_ch; ++c) {
        const int cbase = c * CHUNK;   // first key of the chunk inside the split
        // ---- scores of this wave's keys of the chunk (4 lanes per key)
        float s[PPW][G];
        float mloc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) mloc[h] = -INFINITY;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            u32x4 qh[QD / 8];
#pragma unroll
            for (int cc = 0; cc < QD / 8; ++cc) qh[cc] = *(const u32x4 *)(qs + h * (HD / 2) + qtr * (QD / 2) + 4 * cc);
#pragma unroll
            for (int i = 0; i < PPW; ++i) {
                const bool vis = ok_cur[i] && cbase + (wave + 4 * i) * kPage + kin < nk;
                float d2 = 0.f;
#pragma unroll
                for (int cc = 0; cc < KL; ++cc)
#pragma unroll
                    for (int e = 0; e < 4; ++e) d2 = dot2(qh[cc][e], kr[i][cc][e], d2);
                d2 += quad_xor1(d2);
                d2 += quad_xor2(d2);
                s[i][h] = vis ? d2 * scale : -INFINITY;
                mloc[h] = fmaxf(mloc[h], s[i][h]);
            }
            __builtin_amdgcn_sched_barrier(0);   // one head's q in registers at a time
        }
        // the next chunk's keys go out now (kr is free); its page ids were loaded a chunk ago.
        // The scheduling barrier keeps the loads below the dot products, so the next chunk's
        // keys reuse this chunk's registers instead of needing a second set.
        __builtin_amdgcn_sched_barrier(0);
        if (c + 1 < n_ch) {
            check_pages(c + 1, pg_nxt, ok_nxt);
            issue_k(pg_nxt);
        }
        // ---- online softmax over the wave's keys so far
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float mh = quads_max(mloc[h]);
            const float mn = fmaxf(m[h], mh);
            const float alpha = m[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[h] - mn);
            m[h] = mn;
            float ls = 0.f;
#pragma unroll
            for (int i = 0; i < PPW; ++i) {
                const float pr = mn == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s[i][h] - mn);
                ls += pr;
                // key i*16 + kin of this wave; adjacent keys share one 32-bit word
                const int key = i * kPage + kin;
                if (qtr == 0) pk16[((key >> 1) * G + h) * 2 + (key & 1)] = (uint16_t)f2bf_bits(pr);
            }
            l[h] = l[h] * alpha + quads_sum(ls);
#pragma unroll
            for (int d = 0; d < VD; ++d) acc[h][d] *= alpha;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        // ---- P V from registers: this lane owns head dims lane*VD .. lane*VD+VD-1 of its pages
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            // positions of page i inside the split (0 when the page is absent or invalid)
            const int valid = ok_cur[i] ? min(kPage, nk - cbase - (wave + 4 * i) * kPage) : 0;
#pragma unroll
            for (int d = 0; d < VD; ++d) {
#pragma unroll
                for (int jp = 0; jp < 8; ++jp) {
                    uint32_t vv = vr[i][(d * 8 + jp) >> 2][(d * 8 + jp) & 3];
                    // positions past the split hold other data (or NaN poison): zero them
                    vv = (2 * jp + 1 < valid) ? vv : ((2 * jp < valid) ? (vv & 0xffffu) : 0u);
                    const uint32_t *pw = pkw + (i * 8 + jp) * G;
#pragma unroll
                    for (int h = 0; h < G; ++h) acc[h][d] = dot2(pw[h], vv, acc[h][d]);
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (c + 1 < n_ch) {
            issue_v(pg_nxt);
#pragma unroll
            for (int i = 0; i < PPW; ++i) {
                pg_cur[i] = pg_nxt[i];
                ok_cur[i] = ok_nxt[i];
            }
            if (c + 2 < n_ch) load_pages(c + 2, pg_nxt);
        }
        // the next chunk's weights overwrite this wave's LDS slots only after these reads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (lane == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            mw[wave * G + h] = m[h];
            lw[wave * G + h] = l[h];
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < VD; ++d) part[(wave * G + h) * HD + lane * VD + d] = acc[h][d];
    __syncthreads();
    // ---- merge the four waves in a fixed order
    for (int o = tid; o < G * HD; o += 256) {
        const int h = o / HD, d = o % HD;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, mw[w * G + h]);
        float L = 0.f, sum = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float sc_w = mw[w * G + h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw[w * G + h] - M);
            L += lw[w * G + h] * sc_w;
            sum += part[(w * G + h) * HD + d] * sc_w;
        }
        if (pslot < 0) {
            const float out = L > 0.f ? sum / L : 0.f;
            ((bf16 *)a.o)[((size_t)tok * a.nq + g * G + h) * HD + d] = from_f32<bf16>(out);
        } else {
            float *pp = a.partials + ((size_t)pslot * G + h) * (HD + 2);
            if (d == 0) {
                pp[0] = M;
                pp[1] = L;
            }
            pp[2 + d] = sum;
        }
    }
}

// ------------------------------------------------------------------ decode split, fp32 path
template <int HD, int G>
__device__ void decode_item_f32(const AttnArgs &a, const int32_t *it, char *smem) {
    constexpr int MAXK = kSplitPages * kPage;
    float *sc = (float *)smem;  // [MAXK][G]
    float *red = sc + MAXK * G;
    float *part = red + 8 * G;  // [4][G][HD]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = it[IT_INDEX], g = it[IT_KVHEAD];
    const int k0 = it[IT_KEY_BEGIN], k1 = it[IT_KEY_END], pslot = it[IT_PARTIAL];
    const int nk = k1 - k0;
    const int32_t *row = a.rows + kRowInts * j;
    const int seq = row[0], tok = row[2];
    const PoolView pv = pool_view(a, 1);
    const int32_t *bt = pv.bt + (size_t)seq * pv.max_blocks + k0 / kPage;
    const size_t page_elems = (size_t)a.nkv * kPage * HD;
    const float scale = kLog2e / sqrtf((float)HD);
    const float *q = (const float *)a.q + ((size_t)tok * a.nq + g * G) * HD;
    // scores: one key per thread
    for (int key = tid; key < nk; key += 256) {
        const int page = bt[key / kPage];
        const bool ok = page >= 0 && page < pv.n_pages;
        if (!ok) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
        const float *kr = (const float *)pv.k + page * page_elems + ((size_t)g * kPage + key % kPage) * HD;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float s = 0.f;
            if (ok)
                for (int d = 0; d < HD; ++d) s = fmaf(q[h * HD + d], kr[d], s);
            sc[key * G + h] = ok ? s * scale : -INFINITY;
        }
    }
    __syncthreads();
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
        const float p = (tid < nk && m[h] != -INFINITY) ? exp2f(v[h] - m[h]) : 0.f;
        if (tid < nk) sc[tid * G + h] = p;
        const float ws = wave_sum(p);
        if (lane == 0) red[wave * 2 * G + G + h] = ws;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) l[h] = red[G + h] + red[3 * G + h] + red[5 * G + h] + red[7 * G + h];
    // P V: wave w sums keys w, w+4, ...; thread owns dims lane, lane+64
    for (int o = lane; o < HD; o += 64) {
        float acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = 0.f;
        for (int key = wave; key < nk; key += 4) {
            const int page = bt[key / kPage];
            if (page < 0 || page >= pv.n_pages) continue;
            const float vv = ((const float *)pv.v)[page * page_elems + ((size_t)g * HD + o) * kPage + key % kPage];
#pragma unroll
            for (int h = 0; h < G; ++h) acc[h] = fmaf(sc[key * G + h], vv, acc[h]);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) part[(wave * G + h) * HD + o] = acc[h];
    }
    __syncthreads();
    for (int o = tid; o < G * HD; o += 256) {
        const int h = o / HD, d = o % HD;
        const float sum = ((part[(0 * G + h) * HD + d] + part[(1 * G + h) * HD + d]) +
                           part[(2 * G + h) * HD + d]) + part[(3 * G + h) * HD + d];
        if (pslot < 0) {
            ((float *)a.o)[((size_t)tok * a.nq + g * G + h) * HD + d] = l[h] > 0.f ? sum / l[h] : 0.f;
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
template <int HD, int G>
__device__ void prefill_item_f32(const AttnArgs &a, const int32_t *it) {
    const int tid = threadIdx.x;
    const int ci = it[IT_INDEX], g = it[IT_KVHEAD], qb = it[IT_A], qn = it[IT_B];
    if (tid >= qn * G) return;
    const int r = tid / G, h = g * G + tid % G;
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], tok = ch[4] + qb + r;
    const int qpos = off + qb + r;
    const PoolView pv = pool_view(a, chunk_pool(ch));
    const size_t page_elems = (size_t)a.nkv * kPage * HD;
    const float *qp = (const float *)a.q + ((size_t)tok * a.nq + h) * HD;
    float q[HD], acc[HD];
    const float scale = kLog2e / sqrtf((float)HD);
#pragma unroll
    for (int d = 0; d < HD; ++d) {
        q[d] = qp[d] * scale;
        acc[d] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    for (int kp = 0; kp <= qpos; ++kp) {
        const int page = pv.bt[(size_t)seq * pv.max_blocks + kp / kPage];
        if (page < 0 || page >= pv.n_pages) {
            flag_error(a.err, ORTHRUS_DEVERR_PAGE);
            continue;
        }
        const float *kr = (const float *)pv.k + page * page_elems + ((size_t)g * kPage + kp % kPage) * HD;
        const float *vr = (const float *)pv.v + page * page_elems + (size_t)g * HD * kPage + kp % kPage;
        float s = 0.f;
#pragma unroll
        for (int d = 0; d < HD; ++d) s = fmaf(q[d], kr[d], s);
        const float mn = fmaxf(m, s);
        const float alpha = exp2f(m - mn), p = exp2f(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int d = 0; d < HD; ++d) acc[d] = fmaf(p, vr[d * kPage], acc[d] * alpha);
        m = mn;
    }
    float *op = (float *)a.o + ((size_t)tok * a.nq + h) * HD;
#pragma unroll
    for (int d = 0; d < HD; ++d) op[d] = l > 0.f ? acc[d] / l : 0.f;
}

// ------------------------------------------------------------------ prefill, bf16 MFMA path
// 64-key blocks (four pages) reach LDS by direct global->LDS copies (global_load_lds_dwordx4, no
// register staging): keys as [key][dim] rows of HD*2 bytes, 16-byte chunks XOR-swizzled by row
// so the 16 lanes reading one chunk of 16 keys hit distinct banks; values page by page as the
// cache holds them, [page][dim][16 positions], the two 16-byte halves of a dim swapped on every
// other group of 8 dims.  Two LDS buffers, alternating from the item's first block (a key piece
// may start on an odd block): the copies of block kb+1 go out after the barrier
// that opens block kb and land while block kb is computed; one barrier per 64 keys.  A block
// holding keys past the tile's end or a bad page gets those values (and a bad page's keys)
// zeroed in LDS before it is read (cache slots past a sequence's length may hold NaN).
template <int HD>
struct PrefillStage {
    static constexpr int KEYS = 64;                     // keys per block
    static constexpr int KRB = HD * 2;                  // bytes of one key row
    static constexpr int KCH = KRB / 16;                // 16-byte chunks per key row
    static constexpr int RP256 = 256 / KRB;             // key rows per 256 bytes
    static constexpr int KBYTES = KEYS * KRB;           // key block
    static constexpr int VPAGE = HD * kPage * 2;        // one page's values (one KV head)
    static constexpr int BYTES = KBYTES + 4 * VPAGE;    // one buffer
    static constexpr int K_INST = KBYTES / 1024, V_INST = 4 * VPAGE / 1024;   // 1 KiB copies
    static_assert(K_INST % 4 == 0 && V_INST % 4 == 0, "copies per wave");
    // physical 16-byte chunk of logical chunk c of key row r / of value chunk c of dim d
    static __device__ __forceinline__ int kchunk(int r, int c) { return c ^ ((r / RP256) % KCH); }
    static __device__ __forceinline__ int vchunk(int d, int c) { return c ^ ((d >> 3) & 1); }
};

template <int HD, int G>
__device__ void prefill_item_mfma(const AttnArgs &a, const int32_t *it, char *smem) {
    using St = PrefillStage<HD>;
    constexpr int KS = HD / 16, DB = HD / 32;
    // the wave index and everything derived from it (rows, heads, causal bounds) are wave-uniform;
    // taken from lane 0 they live in scalar registers and every branch on them is a scalar one
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ci = it[IT_INDEX], g = it[IT_KVHEAD], qb = it[IT_A], qn = it[IT_B];
    // keys [k0, kend) of the tile: all of them up to its causal bound, or one piece of a
    // key-split tile (pieces start on 64-key boundaries and only the last piece reaches the
    // diagonal), whose (max, sum, unnormalised output) go to partial slots
    const int k0 = it[IT_KEY_BEGIN], kend = it[IT_KEY_END], pslot = it[IT_PARTIAL];
    const int32_t *ch = a.chunks + kChunkInts * ci;
    const int seq = ch[0], off = ch[1], tok0 = ch[4];
    const int sb = wave / G;
    const int h = g * G + (wave % G);
    const int col = lane & 31, half = lane >> 5;
    const int rows = max(0, min(32, qn - sb * 32));
    const int r = sb * 32 + min(col, max(rows, 1) - 1);   // padded rows repeat a valid row
    const int tok = tok0 + qb + min(r, qn - 1);
    const int qpos = off + qb + min(r, qn - 1);
    const PoolView pv = pool_view(a, chunk_pool(ch));
    const size_t page_bytes = (size_t)a.nkv * kPage * HD * 2;
    const int32_t *bt = pv.bt + (size_t)seq * pv.max_blocks;
    const int kb0 = k0 / St::KEYS, nkb = (kend + St::KEYS - 1) / St::KEYS;
    const int last_block = (kend - 1) / kPage;      // last page index the tile reads

    // page ids of the tile's keys, staged in LDS a window at a time (validated there, -1 = bad)
    int *pg_lds = (int *)(smem + 2 * St::BYTES);
    auto load_window = [&](int w0) {
        bool bad = false;
        for (int i = tid; i < kPrefillPageWindow && w0 + i <= last_block; i += 256) {
            const int pg = bt[w0 + i];
            const bool ok = pg >= 0 && pg < pv.n_pages;
            bad |= !ok;
            pg_lds[i] = ok ? pg : -1;
        }
        if (bad) flag_error(a.err, ORTHRUS_DEVERR_PAGE);
    };
    int w0 = 4 * kb0;
    // page id of page p (0..3) of block blk (-1 = bad); pages past the tile's last one repeat it
    auto page_of = [&](int blk, int p) -> int {
        return __builtin_amdgcn_readfirstlane(pg_lds[min(4 * blk + p, last_block) - w0]);
    };
    // page ids of block b, switching the LDS window when b leaves it (blocks never straddle a
    // window: windows start at multiples of four pages); called at the same point by every thread
    auto block_pages = [&](int b, int (&pg)[4]) {
        if (4 * b - w0 >= kPrefillPageWindow) {
            __syncthreads();
            w0 += kPrefillPageWindow;
            load_window(w0);
            __syncthreads();
        }
#pragma unroll
        for (int p = 0; p < 4; ++p) pg[p] = page_of(b, p);
    };
    // this wave's copies of block b (pages pg) into buffer buf: key copies w, w + 4, ..., then
    // value copies; a bad page reads page 0 (zeroed in LDS afterwards)
    auto issue = [&](const int (&pg)[4], int buf) {
        char *kl = smem + buf * St::BYTES, *vl = kl + St::KBYTES;
#pragma unroll
        for (int j = wave; j < St::K_INST; j += 4) {
            const int row = j * (1024 / St::KRB) + lane / St::KCH;
            const int c = St::kchunk(row, lane % St::KCH);
            const char *src = pv.k + (size_t)max(pg[row / kPage], 0) * page_bytes +
                              ((size_t)(g * kPage + row % kPage) * HD + c * 8) * 2;
            __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(kl + j * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int j = wave; j < St::V_INST; j += 4) {
            constexpr int PER_PAGE = St::VPAGE / 1024;
            const int p = j / PER_PAGE, d = (j % PER_PAGE) * 32 + lane / 2;
            const int c = St::vchunk(d, lane % 2);
            const char *src = pv.v + (size_t)max(pg[p], 0) * page_bytes + ((size_t)(g * HD + d) * kPage + c * 8) * 2;
            __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(vl + j * 1024), 16, 0, 0);
        }
    };
    // zero, in buffer buf of block b, the values of keys at or past kend and the keys and values
    // of bad pages (a uniform condition decides whether any thread needs to)
    auto needs_fixup = [&](int b, const int (&pg)[4]) {
        return (b + 1) * St::KEYS > kend || pg[0] < 0 || pg[1] < 0 || pg[2] < 0 || pg[3] < 0;
    };
    auto fixup = [&](int b, const int (&pg)[4], int buf) {
        char *kl = smem + buf * St::BYTES, *vl = kl + St::KBYTES;
        for (int i = tid; i < 4 * HD; i += 256) {           // value rows: (page, dim)
            const int p = i / HD, d = i % HD;
            const int first = b * St::KEYS + p * kPage;     // key of slot 0 of this page
            const int keep = pg[p] < 0 ? 0 : max(0, min(kPage, kend - first));
            for (int sl = keep; sl < kPage; ++sl)
                *(uint16_t *)(vl + p * St::VPAGE + d * 32 + St::vchunk(d, sl / 8) * 16 + (sl % 8) * 2) = 0;
        }
        for (int i = tid; i < St::KEYS * St::KCH; i += 256) {   // key chunks of bad pages
            const int row = i / St::KCH, c = i % St::KCH;
            if (pg[row / kPage] < 0) *(u32x4 *)(kl + row * St::KRB + St::kchunk(row, c) * 16) = u32x4{0u, 0u, 0u, 0u};
        }
    };

    bf16x8 qf[KS];
    const bf16 *qp = (const bf16 *)a.q + ((size_t)tok * a.nq + h) * HD;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = *(const bf16x8 *)(qp + kk * 16 + half * 8);

    f32x16 acc[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[d][e] = 0.f;
    // running maximum m (log2 domain, scores times `scale`) and sum l of this lane's query.  m
    // is raised only when a block's maximum exceeds it by more than 2^8 (any lane of the wave),
    // so the rescale of the accumulators is rare; probabilities stay below 2^8 in between and
    // the final division by l is unaffected.
    float m = -INFINITY, l = 0.f;
    const float scale = kLog2e / sqrtf((float)HD);
    const int wave_first = off + qb + sb * 32;    // first query position of this wave

    auto compute = [&](int kb) {
        if (rows <= 0 || kb * St::KEYS > wave_first + rows - 1) return;   // past this wave's queries
        const char *kl = smem + ((kb - kb0) & 1) * St::BYTES, *vl = kl + St::KBYTES;
        // S^T = K Q^T for the two 32-key halves: two independent MFMA chains; lane's query = col.
        // Row r of half j's operand is key 32 j + (r with bits 2 and 3 swapped), so register e
        // of half j holds key 32 j + 16 (e / 8) + 8 half + 4 (e / 4 % 2) + e % 4: the eight
        // probabilities a lane packs for one page are then its slots 8 half .. 8 half + 7, one
        // 16-byte chunk of each value row
        f32x16 s[2];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) s[j][e] = 0.f;
        const int kcol = col ^ ((((col >> 2) ^ (col >> 3)) & 1) * 12);
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int row = 32 * j + kcol;
                const bf16x8 kf = *(const bf16x8 *)(kl + row * St::KRB + St::kchunk(row, 2 * kk + half) * 16);
                s[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[j], 0, 0, 0);
            }
        if ((kb + 1) * St::KEYS > wave_first) {   // block reaches this wave's first query: mask
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int kpos = kb * St::KEYS + 32 * j + (e >> 3) * 16 + half * 8 + ((e >> 2) & 1) * 4 + (e & 3);
                    if (kpos > qpos) s[j][e] = -INFINITY;
                }
        }
        float mloc = s[0][0];
#pragma unroll
        for (int e = 1; e < 16; ++e) mloc = fmaxf(mloc, s[0][e]);
#pragma unroll
        for (int e = 0; e < 16; ++e) mloc = fmaxf(mloc, s[1][e]);
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * scale;
        if (__ballot(mloc > m + 8.f) != 0) {
            const float mn = fmaxf(m, mloc);
            const float alpha = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - mn);
            l *= alpha;
#pragma unroll
            for (int d = 0; d < DB; ++d)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[d][e] *= alpha;
            m = mn;
        }
        const float neg_m = (m == -INFINITY) ? 0.f : -m;
        float psum = 0.f;
        bf16x8 pf[2][2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            float p[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                p[e] = __builtin_amdgcn_exp2f(fmaf(s[j][e], scale, neg_m));
                psum += p[e];
            }
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                u32x4 w;
#pragma unroll
                for (int q = 0; q < 4; ++q) w[q] = pack_bf16x2(p[k2 * 8 + 2 * q], p[k2 * 8 + 2 * q + 1]);
                pf[j][k2] = __builtin_bit_cast(bf16x8, w);
            }
        }
        psum += __shfl_xor(psum, 32, 64);
        l += psum;
        // O^T[dim][query] += V^T[dim][keys] P^T[keys][query]; for half j and k2, lane half `half`
        // holds slots 8 half .. 8 half + 7 of page 2 j + k2 of the block
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                for (int d = 0; d < DB; ++d) {
                    const int dim = d * 32 + col;
                    const bf16x8 vf =
                        *(const bf16x8 *)(vl + (2 * j + k2) * St::VPAGE + dim * 32 + St::vchunk(dim, half) * 16);
                    acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[j][k2], acc[d], 0, 0, 0);
                }
    };

    load_window(w0);
    __syncthreads();
    int pg_cur[4];
    block_pages(kb0, pg_cur);
    issue(pg_cur, 0);
    for (int kb = kb0; kb < nkb; ++kb) {
        // this wave's copies of block kb have landed; the barrier: everyone's have, and everyone
        // is done with block kb - 1, whose buffer the next copies refill
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        const bool fix = needs_fixup(kb, pg_cur);
        int pg_nxt[4];
        if (kb + 1 < nkb) {
            block_pages(kb + 1, pg_nxt);
            issue(pg_nxt, (kb + 1 - kb0) & 1);
        }
        if (fix) {
            fixup(kb, pg_cur, (kb - kb0) & 1);
            __syncthreads();
        }
        compute(kb);
        if (kb + 1 < nkb) {
#pragma unroll
            for (int p = 0; p < 4; ++p) pg_cur[p] = pg_nxt[p];
        }
    }
    if (col >= rows) return;
    if (pslot >= 0) {
        // piece of a split tile: row r of the tile is slot pslot + r, holding the group's heads
        float *pp = a.partials + ((size_t)(pslot + sb * 32 + col) * G + (wave % G)) * (HD + 2);
        if (half == 0) {
            pp[0] = m;
            pp[1] = l;
        }
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                float2 *dst = (float2 *)(pp + 2 + d * 32 + q4 * 8 + half * 4);
                dst[0] = float2{acc[d][q4 * 4 + 0], acc[d][q4 * 4 + 1]};
                dst[1] = float2{acc[d][q4 * 4 + 2], acc[d][q4 * 4 + 3]};
            }
        return;
    }
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

// LDS of a bf16 decode item walked in chunks of CP pages
template <int HD, int G, int CP>
constexpr size_t decode_smem() {
    return (4 * (CP * kPage / 4 / 2) * G + 8 * G + 4 * G * HD + 4 * G * HD / 2) * 4;
}

template <bool BF16, int HD, int G>
constexpr size_t attn_smem() {
    constexpr int MAXK = kSplitPages * kPage;
    constexpr size_t dec = BF16 ? decode_smem<HD, G, kDecodeChunkPages>() : (MAXK * G + 8 * G + 4 * G * HD) * 4;
    constexpr size_t pre = BF16 ? 2 * PrefillStage<HD>::BYTES + 4 * kPrefillPageWindow : 0;
    return dec > pre ? dec : pre;
}

template <bool BF16, int HD, int G>
__global__ __launch_bounds__(256, BF16 ? 2 : 1) void attn_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[attn_smem<BF16, HD, G>()];
    const int32_t *it = a.items + kItemInts * blockIdx.x;
    if (it[IT_KIND] == 0) {
        if constexpr (BF16) prefill_item_mfma<HD, G>(a, it, smem);
        else prefill_item_f32<HD, G>(a, it);
    } else {
        if constexpr (BF16) decode_item_bf16<HD, G>(a, it, smem);
        else decode_item_f32<HD, G>(a, it, smem);
    }
}

// Decode items only (bf16; a launch whose work list holds no prefill tile, e.g. the generator's
// rows of a two-model step): chunks of kDecodeOnlyChunkPages pages, one page per wave.  Without the
// prefill path's registers and LDS the workgroup needs 134 VGPRs and 13 KB (7B shape, group 4)
// instead of 212 and 38 KB, so three fit per CU instead of two (two-model step with decode rows
// only: 10.30 -> 10.14 ms).
constexpr int kDecodeOnlyChunkPages = 4;
template <int HD, int G>
__global__ __launch_bounds__(256, 3) void attn_decode_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[decode_smem<HD, G, kDecodeOnlyChunkPages>()];
    decode_item_bf16<HD, G, kDecodeOnlyChunkPages>(a, a.items + kItemInts * blockIdx.x, smem);
}

// Merge key-range partials in split order: M = max m_s, L = sum l_s 2^(m_s - M),
// o = sum acc_s 2^(m_s - M) / L.  Blocks [0, n_dec_blocks): one (split decode row, KV head)
// each, for its `group` query heads (rows with one split wrote their output directly); then
// kCombineRows rows of one key-split prefill tile per block.  Up to kCombineSplits splits are
// loaded in one round before any arithmetic (a block is a single memory round trip), longer
// decode rows loop.
constexpr int kCombineRows = 4;
constexpr int kCombineSplits = 8;
static_assert(kMaxPrefillSplits <= kCombineSplits, "prefill pieces load in one round");

template <typename T>
__device__ __forceinline__ void merge_splits(const AttnArgs &a, const float *pp, size_t stride, int nsplit,
                                             int d, size_t out) {
    float m[kCombineSplits], l[kCombineSplits], v[kCombineSplits];
#pragma unroll
    for (int s = 0; s < kCombineSplits; ++s) {
        if (s < nsplit) {
            const float *q = pp + (size_t)s * stride;
            m[s] = q[0];
            l[s] = q[1];
            v[s] = q[2 + d];
        }
    }
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < kCombineSplits; ++s)
        if (s < nsplit) M = fmaxf(M, m[s]);
    for (int s = kCombineSplits; s < nsplit; ++s) M = fmaxf(M, pp[(size_t)s * stride]);
    float L = 0.f, acc = 0.f;
#pragma unroll
    for (int s = 0; s < kCombineSplits; ++s) {
        if (s < nsplit) {
            const float w = (m[s] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[s] - M);
            L += l[s] * w;
            acc += v[s] * w;
        }
    }
    for (int s = kCombineSplits; s < nsplit; ++s) {
        const float *q = pp + (size_t)s * stride;
        const float w = (q[0] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(q[0] - M);
        L += q[1] * w;
        acc += q[2 + d] * w;
    }
    ((T *)a.o)[out] = from_f32<T>(L > 0.f ? acc / L : 0.f);
}

template <typename T, int HD, int G>
__global__ __launch_bounds__(G * HD) void attn_combine_kernel(AttnArgs a, int n_dec_blocks) {
    const int h = threadIdx.x / HD, d = threadIdx.x % HD;
    if ((int)blockIdx.x < n_dec_blocks) {
        const int j = a.split_rows[blockIdx.x / a.nkv], g = blockIdx.x % a.nkv;
        const int32_t *row = a.rows + kRowInts * j;
        const int nsplit = row[3];
        if (nsplit <= 1) return;
        const float *pp = a.partials + ((size_t)(row[4] + g * nsplit) * G + h) * (HD + 2);
        merge_splits<T>(a, pp, (size_t)G * (HD + 2), nsplit, d, ((size_t)row[2] * a.nq + g * G + h) * HD + d);
        return;
    }
    constexpr int QR = kPrefillRows / G, BPM = QR / kCombineRows;   // blocks per merge entry
    const int b = blockIdx.x - n_dec_blocks;
    const int32_t *mg = a.combine + kCombineInts * (b / BPM);
    const int r0 = (b % BPM) * kCombineRows;
#pragma unroll
    for (int i = 0; i < kCombineRows; ++i) {
        const int r = r0 + i;
        if (r < mg[1]) {
            const float *pp = a.partials + ((size_t)(mg[4] + r) * G + h) * (HD + 2);
            merge_splits<T>(a, pp, (size_t)QR * G * (HD + 2), mg[3], d,
                            ((size_t)(mg[0] + r) * a.nq + mg[2] * G + h) * HD + d);
        }
    }
}

template <bool BF16, int HD, int G>
hipError_t run(const AttnArgs &a, int n_decode, bool combine, hipStream_t s) {
    if (combine) {
        const int n_dec = n_decode * a.nkv, blocks = n_dec + a.n_combine * (kPrefillRows / G / kCombineRows);
        if (blocks <= 0) return hipSuccess;
        if (BF16) hipLaunchKernelGGL((attn_combine_kernel<bf16, HD, G>), dim3(blocks), dim3(G * HD), 0, s, a, n_dec);
        else hipLaunchKernelGGL((attn_combine_kernel<float, HD, G>), dim3(blocks), dim3(G * HD), 0, s, a, n_dec);
        return hipGetLastError();
    }
    if (a.n_items <= 0) return hipSuccess;
    if (BF16 && a.n_prefill == 0)
        hipLaunchKernelGGL((attn_decode_kernel<HD, G>), dim3(a.n_items), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((attn_kernel<BF16, HD, G>), dim3(a.n_items), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <bool BF16>
hipError_t dispatch(const AttnArgs &a, int n_decode, bool combine, hipStream_t s) {
    const int G = a.nq / a.nkv;
#define ORTHRUS_ATTN_CASE(HDV, GV) \
    if (a.hd == HDV && G == GV) return run<BF16, HDV, GV>(a, n_decode, combine, s);
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
    return dtype == 1 ? dispatch<true>(a, 0, false, s) : dispatch<false>(a, 0, false, s);
}

hipError_t launch_attn_combine(int dtype, const AttnArgs &a, int n_decode, hipStream_t s) {
    return dtype == 1 ? dispatch<true>(a, n_decode, true, s) : dispatch<false>(a, n_decode, true, s);
}

}  // namespace orthrus
