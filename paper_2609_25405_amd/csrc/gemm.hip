// Dense projections of the step: C[M][N] = A[M][K] * W[N][K]^T over the concatenated token
// batch (QKV, attention output, gate/up, down, LM head), with fused epilogues.
//
// bf16 path: CDNA4 MFMA v_mfma_f32_32x32x16_bf16, WM x WN wave64s per workgroup, K staged 64
// elements at a time through two LDS buffers filled by direct global->LDS copies
// (global_load_lds_dwordx4, no register staging), so each K stage costs one barrier.  LDS rows
// are 128 B; 16-byte chunks are XOR-swizzled by row so the per-lane 16-byte operand reads of
// one MFMA hit distinct banks (the copies pick their source chunk to land in swizzled order).
// Tiles are mapped to blocks so that consecutive tiles of one weight column block land on
// the same XCD (blocks are dealt round-robin to the 8 XCDs), which keeps re-reads of a
// weight tile inside one L2.
// fp32 path: plain LDS-tiled FMA kernel (64x64 tile, 4x4 per thread) for exact checks.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "orthrus.h"

namespace orthrus {

namespace {

constexpr int BK = 64;

__device__ __forceinline__ float silu(float g) { return g / (1.f + __expf(-g)); }

// 16-byte global -> LDS copy: lane i of the wave writes lds + 16 * i (lds is wave-uniform).
// AUX is the cache policy: 0 default, kNonTemporal for data the launch reads exactly once.
constexpr int kNonTemporal = 2;
template <int AUX = 0>
__device__ __forceinline__ void copy16_to_lds(const void *src, char *lds) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds, 16, 0, AUX);
}

// s_waitcnt immediate that waits until at most n vector-memory operations are outstanding
// (gfx9 encoding: vmcnt[3:0] in bits 3:0 and vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt at
// their maxima so they impose no wait)
template <int N>
constexpr int vmcnt_imm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    return (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);
}

// workgroup barrier for the LDS ring: the LDS reads issued before it have completed and no
// memory access moves across it; unlike __syncthreads it does not drain the outstanding
// global->LDS copies of later stages (their completion is awaited explicitly with vmcnt)
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// STREAM_B: the launch has one row tile, so each weight byte is read exactly once; its copies
// are non-temporal (LM head 64 x 32000 x 4096 in the step: 66 -> 56 us)
template <int BM, int BN, int WM, int WN, int EPI, int BKS, int STAGES, int BSTAGES, bool STREAM_B>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_bf16_kernel(GemmArgs a) {
    constexpr int NW = WM * WN;               // waves per workgroup
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 32, FN = TN / 32;
    constexpr int ROWB = BKS * 2;             // bytes of one LDS row (BKS bf16 of K)
    constexpr int CHUNKS = ROWB / 16;         // 16-byte chunks per row
    constexpr int RPI = 1024 / ROWB;          // rows moved by one wave copy instruction (1 KiB)
    constexpr int RP256 = 256 / ROWB;         // rows per 256 bytes (one pass of the 64 LDS banks)
    // global -> LDS copies of one K stage
    constexpr int A_INST = BM / (RPI * NW), B_INST = BN / (RPI * NW);
    constexpr int INST = A_INST + B_INST;     // copy instructions per wave per stage
    constexpr int KSTEPS = BKS / 16;
    // separate rings for A (STAGES buffers of BM rows) and B (BSTAGES buffers of BN rows): the
    // weight operand may prefetch deeper than the activations within the same LDS budget
    constexpr int RING_BYTES = STAGES * BM * ROWB + BSTAGES * BN * ROWB;
    // the shallower ring's copies are issued first in every iteration; vector-memory operations
    // complete in order, so iteration kt may leave these many copies of this wave in flight when
    // it waits for its stage kt (the deeper ring's copies issued after the shallower's stage kt)
    constexpr int SD = STAGES < BSTAGES ? STAGES : BSTAGES, SDD = STAGES < BSTAGES ? BSTAGES : STAGES;
    constexpr int DEEP_INST = STAGES < BSTAGES ? B_INST : A_INST;
    constexpr int IN_FLIGHT = (SD - 2) * INST + (SDD > SD ? DEEP_INST : 0);
    static_assert(A_INST * RPI * NW == BM && B_INST * RPI * NW == BN, "copy split");
    static_assert(FM >= 1 && FN >= 1 && (EPI != EPI_SWIGLU || FN % 2 == 0), "tile shape");
    static_assert(SD >= 2 && IN_FLIGHT < 64, "pipeline depth");
    // the QKV epilogue stages the fp32 tile (rows padded to 136 floats) and per-row metadata
    constexpr int CROW = 136;
    constexpr int EPI_BYTES = EPI == EPI_QKV_ROPE ? BM * CROW * 4 + BM * 16 : 0;
    __shared__ __attribute__((aligned(1024))) char smem[RING_BYTES > EPI_BYTES ? RING_BYTES : EPI_BYTES];
    char *const smem_b = smem + STAGES * BM * ROWB;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int mt = (a.M + BM - 1) / BM;
    constexpr int COLS_ = EPI == EPI_SWIGLU ? BN / 2 : BN;
    const int tiles = mt * ((a.N + COLS_ - 1) / COLS_);
    const int splits = gridDim.x / tiles;          // split-K factor (1 = whole K per tile)
    const int split = blockIdx.x / tiles;
    const int b = blockIdx.x % tiles;
    const int t = (tiles % 8 == 0) ? (b % 8) * (tiles / 8) + b / 8 : b;
    const int n_tile = t / mt, m_tile = t % mt;
    const int m0 = m_tile * BM;
    constexpr int COLS = EPI == EPI_SWIGLU ? BN / 2 : BN;  // output columns per tile
    const int n0 = n_tile * COLS;

    // LDS row r holds 16-byte chunk c at physical position c ^ key(r), key(r) = (r / RP256) %
    // CHUNKS, so the 16 lanes of one pass of a fragment read (16 consecutive rows, same chunk)
    // hit 16 distinct 16-byte bank groups.  Lane `lane` of copy instruction i of this wave
    // writes LDS bytes base + 16 * lane, i.e. row r0 + lane / CHUNKS at physical chunk
    // lane % CHUNKS (r0 = RPI * (NW i + wave)); it fetches the logical chunk stored there.
    auto key_of = [](int row) { return (row / RP256) % CHUNKS; };
    const size_t lda_b = (size_t)a.lda * 2, ldb_b = (size_t)a.K * 2;
    const char *a_src[A_INST];
    const char *b_src[B_INST];
#pragma unroll
    for (int i = 0; i < A_INST; ++i) {
        const int row = RPI * (NW * i + wave) + lane / CHUNKS;
        const int chunk = (lane % CHUNKS) ^ key_of(row);
        a_src[i] = (const char *)a.A + (size_t)min(m0 + row, a.M - 1) * lda_b + chunk * 16;
    }
#pragma unroll
    for (int i = 0; i < B_INST; ++i) {
        const int r = RPI * (NW * i + wave) + lane / CHUNKS;
        const int chunk = (lane % CHUNKS) ^ key_of(BM + r);
        int grow;
        const char *src = (const char *)a.B0;
        if (EPI == EPI_SWIGLU) {
            const int slice = r / TN, j = r % TN;
            const int half = j / (TN / 2), k = j % (TN / 2);
            if (half) src = (const char *)a.B1;
            grow = n0 + slice * (TN / 2) + k;
        } else {
            grow = n0 + r;
        }
        const int gn = min(grow, a.N - 1);
        b_src[i] = a.b_blocked ? src + ((size_t)(gn / 64) * (a.K / 64) * 64 + gn % 64) * ROWB + chunk * 16
                               : src + (size_t)gn * ldb_b + chunk * 16;
    }
    const size_t b_stage = a.b_blocked ? 64 * ROWB : ROWB;   // bytes between k-stages of a B row
    // this wave's copies of K stage kt of A (into A buffer buf) and of B (into B buffer buf)
    auto copy_a = [&](int kt, int buf) {
        const size_t kb = (size_t)kt * ROWB;
#pragma unroll
        for (int j = 0; j < A_INST; ++j)
            copy16_to_lds(a_src[j] + kb, smem + buf * BM * ROWB + (NW * j + wave) * 1024);
    };
    auto copy_b = [&](int kt, int buf) {
        const size_t kb = (size_t)kt * b_stage;
#pragma unroll
        for (int j = 0; j < B_INST; ++j)
            copy16_to_lds<STREAM_B ? kNonTemporal : 0>(b_src[j] + kb, smem_b + buf * BN * ROWB + (NW * j + wave) * 1024);
    };
    // iteration i's copies: A stage i + STAGES - 1 and B stage i + BSTAGES - 1 (the shallower
    // ring first).  Past the last stage they repeat it into the buffer just freed, which nobody
    // reads, so every iteration issues the same count and the wait bound stays exact.
    auto issue = [&](int i, int kt0, int nk) {
        const int sa = i + STAGES - 1, sb = i + BSTAGES - 1;
        if (STAGES <= BSTAGES) {
            if (sa >= 0) copy_a(kt0 + min(sa, nk - 1), sa % STAGES);
            if (sb >= 0) copy_b(kt0 + min(sb, nk - 1), sb % BSTAGES);
        } else {
            if (sb >= 0) copy_b(kt0 + min(sb, nk - 1), sb % BSTAGES);
            if (sa >= 0) copy_a(kt0 + min(sa, nk - 1), sa % STAGES);
        }
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment rows of this lane; the swizzle key is the same for every 32-row fragment of the
    // lane (32 rows span a whole number of 256-byte passes), so offsets differ by constants
    // (B rows keep the swizzle key of row BM + r, as the copies above write them)
    const int arow = wm * TM + (lane & 31), brow = wn * TN + (lane & 31);
    const int akey = key_of(arow), bkey = key_of(BM + brow);
    bf16x8 fa[2][FM], fb[2][FN];
    auto lds_frag = [&](const char *sa, const char *sb, int kk, int buf) {
        const int chk = kk * 2 + (lane >> 5);
#pragma unroll
        for (int mi = 0; mi < FM; ++mi)
            fa[buf][mi] = *(const bf16x8 *)(sa + (arow + mi * 32) * ROWB + ((chk ^ akey) << 4));
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
            fb[buf][ni] = *(const bf16x8 *)(sb + (brow + ni * 32) * ROWB + ((chk ^ bkey) << 4));
    };

    // Rings of LDS stages: the copies of A stage kt + STAGES - 1 and B stage kt + BSTAGES - 1
    // are issued while stage kt is computed.  Iteration kt: wait for this wave's copies of
    // stage kt (later ones stay in flight), barrier (everyone's copies landed; everyone
    // finished reading the buffers about to be refilled), issue, then the MFMAs of stage kt
    // with the next k-step's fragments read under the current k-step's.  (Spreading the copies
    // between the MFMAs, or L2 prefetches further ahead, measured slower on MI355X.)
    constexpr int NMF = FM * FN, NFR = FM + FN;
    // this split's stages: [kt0, kt0 + nk), the K stages dealt as evenly as the count allows
    const int nk_all = a.K / BKS;
    const int kt0 = split * nk_all / splits;
    const int nk = (split + 1) * nk_all / splits - kt0;
    for (int i = -(SDD - 1); i < 0; ++i) issue(i, kt0, nk);
    // A wave whose rows all lie past M (in the last row tile, when M leaves it partly empty)
    // issues its share of the copies and takes every barrier but reads no fragments and issues
    // no MFMA: its accumulators stay zero and its rows are never stored (1088 rows on 256-row
    // tiles: 1.18x -> 1.06x executed / algorithmic flops).
    auto k_loop = [&](auto live) {
        for (int kt = 0; kt < nk; ++kt) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm<IN_FLIGHT>());
            ring_barrier();
            issue(kt, kt0, nk);
            if constexpr (decltype(live)::value) {
                // the compute phase at raised wave priority: where both waves of a SIMD have an
                // instruction ready, the one feeding the MFMA pipe issues first (1024-row gate/up
                // alone 211.9 -> 204.0 us, down 107.6 -> 103.8 us; raising the copy phase
                // instead, or both at different levels, measured equal or slower)
                __builtin_amdgcn_s_setprio(1);
                const char *sa = smem + (kt % STAGES) * BM * ROWB, *sb = smem_b + (kt % BSTAGES) * BN * ROWB;
                lds_frag(sa, sb, 0, 0);
#pragma unroll
                for (int kk = 0; kk < KSTEPS; ++kk) {
                    if (kk + 1 < KSTEPS) lds_frag(sa, sb, kk + 1, (kk + 1) & 1);
#pragma unroll
                    for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                        for (int ni = 0; ni < FN; ++ni)
                            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk & 1][mi], fb[kk & 1][ni],
                                                                                  acc[mi][ni], 0, 0, 0);
                }
                // schedule: DS_READ=0x100, MFMA=0x008
                __builtin_amdgcn_sched_group_barrier(0x100, NFR, 0);
#pragma unroll
                for (int kk = 0; kk < KSTEPS; ++kk) {
#pragma unroll
                    for (int i = 0; i < NMF; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        if (kk + 1 < KSTEPS && i < NFR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                }
                __builtin_amdgcn_s_setprio(0);
            }
        }
    };
    // the wave's row range is the same for all its lanes; taking lane 0's answer makes the
    // branch scalar, so each wave runs exactly one of the two loops (equal barrier counts)
    if (__builtin_amdgcn_readfirstlane(m0 + wm * TM < a.M ? 1 : 0)) k_loop(std::true_type{});
    else k_loop(std::false_type{});
    // the repeated copies of the last iterations still write LDS: drain them before the
    // epilogues reuse the stage buffers
    __builtin_amdgcn_s_waitcnt(0);

    // LoRA update: acc += U B^T for the launch's rows below lora.rows (split 0 of a split-K
    // launch), 16 columns of U per MFMA step (U as its bf16 rounding plus remainder, two MFMAs),
    // operands straight from global memory in the same fragment layout as the main loop (rows
    // of U and of B are contiguous in the rank)
    if (a.lora.n > 0 && split == 0 && m0 < a.lora.rows) {
        const LoraGemm &L = a.lora;
        const int ldu = L.n * L.r;
        const bf16x8 zero = {};
        for (int c0 = 0; c0 < ldu; c0 += 16) {
            const int j = c0 / L.r, kk = c0 % L.r + 8 * (lane >> 5);
            bf16x8 ua[FM], ul[FM], ub[FN];
#pragma unroll
            for (int mi = 0; mi < FM; ++mi) {
                const int row = m0 + wm * TM + mi * 32 + (lane & 31);
                const size_t off = (size_t)row * ldu + c0 + 8 * (lane >> 5);
                ua[mi] = row < L.rows ? *(const bf16x8 *)((const bf16 *)L.u + off) : zero;
                ul[mi] = row < L.rows ? *(const bf16x8 *)((const bf16 *)L.u_lo + off) : zero;
            }
#pragma unroll
            for (int ni = 0; ni < FN; ++ni) {
                int col;
                const bf16 *src;
                if constexpr (EPI == EPI_SWIGLU) {
                    col = n0 + wn * (TN / 2) + (ni % (FN / 2)) * 32 + (lane & 31);
                    src = (const bf16 *)(ni < FN / 2 ? L.b0[j] : L.b1[j]);
                } else {
                    col = n0 + wn * TN + ni * 32 + (lane & 31);
                    src = (const bf16 *)L.b0[j];
                }
                ub[ni] = *(const bf16x8 *)(src + (size_t)min(col, a.N - 1) * L.r + kk);
            }
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) {
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ua[mi], ub[ni], acc[mi][ni], 0, 0, 0);
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ul[mi], ub[ni], acc[mi][ni], 0, 0, 0);
                }
        }
    }

    if constexpr (EPI == EPI_QKV_ROPE) {
        // Rotation of q and k at each token's position (pairs (i, i + hd/2)), q stored for
        // attention, rotated k and raw v appended to the paged cache.  The fp32 tile goes
        // through LDS so every store is a 16-byte piece: 8 dims of a q or k row, or (values,
        // dim-major pages) 8 consecutive slots of one dim when 8 rows fill them.
        static_assert(BN == 128, "tiles of whole heads");
        const QkvRope &q = a.rope;
        float *ct = (float *)smem;                       // [BM][CROW] fp32 tile
        int4 *meta = (int4 *)(smem + BM * CROW * 4);     // per row {token, slot, page or -1, pool}
        __syncthreads();                                 // every wave is done with the stage buffers
#pragma unroll
        for (int mi = 0; mi < FM; ++mi)
#pragma unroll
            for (int ni = 0; ni < FN; ++ni)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = wm * TM + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                    ct[row * CROW + wn * TN + ni * 32 + (lane & 31)] = acc[mi][ni][r];
                }
        for (int rr = tid; rr < BM; rr += 64 * NW) {
            const int lr = m0 + rr;
            int4 md{-1, 0, -1, 0};
            if (lr < a.M) {
                const int t = q.row0 + lr;
                const int pos = q.pos[t], sq = q.seq[t], pl = t < q.Te ? 0 : 1;
                const int page = q.block_table[pl][(size_t)sq * q.max_blocks[pl] + pos / q.page];
                const bool ok = page >= 0 && page < q.n_pages[pl];
                // flagged once per row: by the tile holding the first key head
                if (!ok && n0 == q.nq * q.hd) flag_error(q.err, ORTHRUS_DEVERR_PAGE);
                md = int4{t, pos % q.page, ok ? page : -1, pl};
            }
            meta[rr] = md;
        }
        __syncthreads();
        const int hd = q.hd, half = hd / 2, G8 = half / 8;
        for (int h2 = 0; h2 < 128 / hd; ++h2) {
            const int head = (n0 + h2 * hd) / hd;
            if (head < q.nq + q.nkv) {
                // q or k: items (row, group of 8 pairs)
                const bool is_q = head < q.nq;
                const int kvh = head - q.nq;
                for (int it = tid; it < BM * G8; it += 64 * NW) {
                    const int row = it / G8, g = it % G8;
                    const int4 md = meta[row];
                    if (md.x < 0 || (!is_q && md.z < 0)) continue;
                    const float *lo = ct + row * CROW + h2 * hd + g * 8, *hi = lo + half;
                    const float4 *csp = (const float4 *)(q.cs + (size_t)md.x * half + g * 8);
                    u32x4 w1, w2;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float4 cs = csp[e];   // (cos, sin) of pairs 2e and 2e + 1
                        const float a0 = lo[2 * e], a1 = lo[2 * e + 1], b0 = hi[2 * e], b1 = hi[2 * e + 1];
                        w1[e] = pack_bf16x2(a0 * cs.x - b0 * cs.y, a1 * cs.z - b1 * cs.w);
                        w2[e] = pack_bf16x2(b0 * cs.x + a0 * cs.y, b1 * cs.z + a1 * cs.w);
                    }
                    bf16 *dst = is_q ? (bf16 *)q.q_out + ((size_t)md.x * q.nq + head) * hd
                                     : (bf16 *)q.k_cache[md.w] + (((size_t)md.z * q.nkv + kvh) * q.page + md.y) * hd;
                    *(u32x4 *)(dst + g * 8) = w1;
                    *(u32x4 *)(dst + half + g * 8) = w2;
                }
            } else {
                // v: items (dim, group of 8 rows); a dim of one page holds `page` slots contiguously.
                // Adjacent lanes take the two 8-row halves of one dim's 16 rows, so a page-aligned
                // run of 16 rows leaves as whole 32-byte runs of consecutive dims (7B-layer mixed
                // step: 80.3 -> 78.8 us against lanes along the dims)
                static_assert(BM % 16 == 0, "16-row groups");
                const int kvh = head - q.nq - q.nkv;
                for (int it = tid; it < hd * (BM / 8); it += 64 * NW) {
                    const int d = (it >> 1) % hd, r0 = ((it >> 1) / hd) * 16 + (it & 1) * 8;
                    const int4 m0d = meta[r0];
                    bool run = m0d.x >= 0 && m0d.z >= 0 && (m0d.y & 7) == 0;
#pragma unroll
                    for (int k = 1; k < 8; ++k) {
                        const int4 mk = meta[r0 + k];
                        run = run && mk.z == m0d.z && mk.w == m0d.w && mk.y == m0d.y + k;
                    }
                    const float *col = ct + r0 * CROW + h2 * hd + d;
                    if (run) {
                        u32x4 w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(col[(2 * e) * CROW], col[(2 * e + 1) * CROW]);
                        bf16 *vc = (bf16 *)q.v_cache[m0d.w] + (((size_t)m0d.z * q.nkv + kvh) * hd + d) * q.page + m0d.y;
                        *(u32x4 *)vc = w;
                    } else {
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const int4 mk = meta[r0 + k];
                            if (mk.x < 0 || mk.z < 0) continue;
                            bf16 *vc = (bf16 *)q.v_cache[mk.w] + (((size_t)mk.z * q.nkv + kvh) * hd + d) * q.page + mk.y;
                            *vc = (bf16)col[k * CROW];
                        }
                    }
                }
            }
        }
        return;
    }

    if constexpr (EPI == EPI_SWIGLU) {
        // The MFMA layout leaves each lane one column of 16 rows per fragment, i.e. 2-byte
        // stores per output.  Instead the BM x BN/2 bf16 output tile is staged through the
        // idle stage buffers and written back as whole 16-byte pieces of its rows.
        constexpr int OC = BN / 2;                 // output columns of the tile
        constexpr int OROW = OC * 2 + 16;          // padded LDS row: rows 4 apart differ by 16 banks
        static_assert(BM * OROW <= RING_BYTES, "output tile fits the stage buffers");
        __syncthreads();                           // every wave is done with the stage buffers
#pragma unroll
        for (int mi = 0; mi < FM; ++mi)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = wm * TM + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
#pragma unroll
                for (int ni = 0; ni < FN / 2; ++ni) {
                    const int col = wn * (TN / 2) + ni * 32 + (lane & 31);
                    *(bf16 *)(smem + row * OROW + col * 2) = (bf16)(silu(acc[mi][ni][r]) * acc[mi][ni + FN / 2][r]);
                }
            }
        __syncthreads();
        constexpr int PPR = OC / 8;                // 16-byte pieces per row
        for (int c = tid; c < BM * PPR; c += 64 * NW) {
            const int row = c / PPR, part = c % PPR;
            const int grow = m0 + row, gcol = n0 + part * 8;
            if (grow < a.M && gcol < a.N)
                *(u32x4 *)((bf16 *)a.out + (size_t)grow * a.ldo + gcol) = *(const u32x4 *)(smem + row * OROW + part * 16);
        }
        return;
    }

    // epilogue: lane holds column (lane & 31) of each 32x32 tile, rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
    for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm * TM + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            if (row >= a.M) continue;
            if (EPI == EPI_SWIGLU) {
                bf16 *o = (bf16 *)a.out + (size_t)row * a.ldo;
#pragma unroll
                for (int ni = 0; ni < FN / 2; ++ni) {
                    const int col = n0 + wn * (TN / 2) + ni * 32 + (lane & 31);
                    if (col < a.N) o[col] = from_f32<bf16>(silu(acc[mi][ni][r]) * acc[mi][ni + FN / 2][r]);
                }
            } else if (splits > 1) {
                // split-K: this split's share goes to its own fp32 slab; the row's consumer adds
                // the slabs to the residual stream in split order
                float *o = a.partial + (size_t)split * a.split_stride + (size_t)row * a.ldo;
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) {
                    const int col = n0 + wn * TN + ni * 32 + (lane & 31);
                    if (col < a.N) o[col] = acc[mi][ni][r];
                }
            } else {
                float *o = (float *)a.out + (size_t)row * a.ldo;
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) {
                    const int col = n0 + wn * TN + ni * 32 + (lane & 31);
                    if (col >= a.N) continue;
                    if (EPI == EPI_ADD_F32) o[col] += acc[mi][ni][r];
                    else o[col] = acc[mi][ni][r];
                }
            }
        }
    }
}

// ------------------------------------------------------------------ fp32 reference-grade path
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
    constexpr int T = 64, KT = 16;
    __shared__ float As[KT][T + 4];
    __shared__ float Bs[KT][T + 4];
    __shared__ float Us[KT][T + 4];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
    const float *A = (const float *)a.A, *B0 = (const float *)a.B0, *B1 = (const float *)a.B1;
    float acc[4][4] = {}, accu[4][4] = {};
    for (int k0 = 0; k0 < a.K; k0 += KT) {
        for (int i = tid; i < T * KT; i += 256) {
            const int r = i / KT, k = i % KT;
            const int gm = min(m0 + r, a.M - 1), gn = min(n0 + r, a.N - 1);
            As[k][r] = A[(size_t)gm * a.lda + k0 + k];
            Bs[k][r] = B0[(size_t)gn * a.K + k0 + k];
            if (EPI == EPI_SWIGLU) Us[k][r] = B1[(size_t)gn * a.K + k0 + k];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < KT; ++k) {
            float av[4], bv[4], uv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                av[i] = As[k][ty * 4 + i];
                bv[i] = Bs[k][tx * 4 + i];
                uv[i] = EPI == EPI_SWIGLU ? Us[k][tx * 4 + i] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
                    if (EPI == EPI_SWIGLU) accu[i][j] = fmaf(av[i], uv[j], accu[i][j]);
                }
        }
        __syncthreads();
    }
    // LoRA update U B^T for the rows below lora.rows
    if (a.lora.n > 0) {
        const LoraGemm &L = a.lora;
        const int ldu = L.n * L.r;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = m0 + ty * 4 + i;
            if (row >= a.M || row >= L.rows) continue;
            const float *u = (const float *)L.u + (size_t)row * ldu;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = min(n0 + tx * 4 + j, a.N - 1);
                float d0 = 0.f, d1 = 0.f;
                for (int c = 0; c < ldu; ++c) {
                    const int ad = c / L.r, kk = c % L.r;
                    d0 = fmaf(u[c], ((const float *)L.b0[ad])[(size_t)col * L.r + kk], d0);
                    if (EPI == EPI_SWIGLU) d1 = fmaf(u[c], ((const float *)L.b1[ad])[(size_t)col * L.r + kk], d1);
                }
                acc[i][j] += d0;
                if (EPI == EPI_SWIGLU) accu[i][j] += d1;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = m0 + ty * 4 + i;
        if (row >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + tx * 4 + j;
            if (col >= a.N) continue;
            if (EPI == EPI_SWIGLU) {
                ((float *)a.out)[(size_t)row * a.ldo + col] = silu(acc[i][j]) * accu[i][j];
            } else if (EPI == EPI_ADD_F32) {
                ((float *)a.out)[(size_t)row * a.ldo + col] += acc[i][j];
            } else {
                ((float *)a.out)[(size_t)row * a.ldo + col] = acc[i][j];
            }
        }
    }
}

template <int BM, int BN, int WM, int WN, int EPI, int BKS = 64, int STAGES = 2, int BSTAGES = STAGES,
          bool STREAM_B = false>
hipError_t run_bf16(const GemmArgs &a, hipStream_t s) {
    const int mt = (a.M + BM - 1) / BM;
    const int cols = EPI == EPI_SWIGLU ? BN / 2 : BN;
    const int nt = (a.N + cols - 1) / cols;
    const int splits =
        (EPI == EPI_ADD_F32 && a.partial && a.splits > 1 && a.K % BKS == 0 && a.K / BKS >= a.splits) ? a.splits : 1;
    if (STREAM_B && mt != 1) return hipErrorInvalidValue;
    if (a.b_blocked && (BKS != 64 || EPI == EPI_SWIGLU || a.K % 64)) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, EPI, BKS, STAGES, BSTAGES, STREAM_B>), dim3(mt * nt * splits),
                       dim3(64 * WM * WN), 0, s, a);
    return hipGetLastError();
}

// Tile choice per shape, from measurements of the step's projections on MI355X (M = 1088
// tokens of a 7B-class layer).  Copy latency, not LDS or MFMA issue, bounds these GEMMs, so
// the choice trades tile reuse against filling the CUs:
//  - M <= 64 (decode-only batches, the LM head): weight streaming; 64x64 tiles (more
//    workgroups) with a 4-deep copy ring keep enough bytes in flight per CU (LM head
//    64 x 32000 x 4096: 70 -> 43 us with warm caches; decode-batch QKV 35 -> 25 us); gate/up
//    on 64x128 tiles (224 workgroups instead of 112: 58.6 -> 43.9 us with cold weights);
//  - gate/up above 896 rows: 192x256 or 256x256 tiles over 8 waves, whichever needs fewer
//    rounds of workgroups times tile rows;
//  - gate/up of 129..256 rows: one 256x128 row tile, the weights streamed once (non-temporal)
//    through 3-deep rings (M = 256 with cold weights: 110 -> 71 us against 128x128 tiles);
//  - residual-add projections of M > 896 rows: 256x256 tiles over 8 waves with the split-K
//    count gemm_add_splits picks (o 58 -> 46 us, down 177 -> 135 us against 128x128 tiles at
//    M = 1088; down at M = 1568 264 -> 195 us, at M = 2048 275 -> 211 us against 192x256
//    tiles split 2, whose 288 or 352 workgroups spill into a second round);
//  - otherwise 128x128 (64 KiB of LDS, two workgroups per CU hide each other's waits).
//  - medium M (64 < M <= 896: decode-heavy and small mixed batches, where the weights stream):
//    more, smaller workgroups and deeper split-K for the residual-add projections (down at
//    M = 384: 124 -> 57 us; o: 42 -> 23 us), 64x128 tiles for QKV up to M = 512, and for
//    gate/up up to M = 896 the 128- or 192-row tile that pads M least (M = 512: 162 -> 129 us);
//  - 64 < M <= 128 (decode batches of up to 128 rows): one row tile of 128 rows and a 4-deep
//    ring (128 KiB of LDS), weights streamed: gate/up 66.5 -> 47.3 us, LM head 74.6 -> 66.5 us,
//    down split 4 ways on 128x64 tiles 38.8 -> 32.7 us (M = 96, cold weights);
//  - split-K residual-add projections of 128 < M <= 256: 128x128 tiles with 4-deep rings (one
//    workgroup per CU; down at M = 192 57.1 -> 45.7 us, o at M = 256 27.1 -> 21.8 us); above 256
//    rows two 64 KiB workgroups per CU win again (down at M = 384: 71 against 86 us).  Run
//    concurrently with another stream (GemmArgs::wide), the same projections take 256x256
//    tiles: 4x fewer workgroup-microseconds per flop at a longer launch, which the other
//    stream's launches fill (the two-model 32-layer step, QKV, o and down of the generator's
//    256 decode rows so tiled: 23.4 -> 22.5 ms and 23.9 -> 23.2 ms on two GPUs; the
//    generator's gate/up on such tiles as well measured slower);
//  - gate/up of 256 < M <= 896, measured on the 7B shape with cold weights: 192x256 when
//    128x128 tiles need more than the 512 slots of one round and 192x256 tiles fit in one
//    (M = 640: 172 against 195 us), else the tile that pads M least (M = 384 98 against 130 us,
//    M = 512 147 against 174 us, M = 896 240 against 256 us).
template <int EPI>
hipError_t dispatch_bf16(const GemmArgs &a, hipStream_t s) {
    if constexpr (EPI == EPI_QKV_ROPE) {
        if (a.M <= 64) return run_bf16<64, 128, 2, 2, EPI, 64, 4, 4, true>(a, s);
        if (a.M <= 512) return run_bf16<64, 128, 1, 4, EPI, 64, 3>(a, s);
        return run_bf16<128, 128, 2, 2, EPI>(a, s);
    } else if constexpr (EPI == EPI_SWIGLU) {
        if (a.M <= 64) return run_bf16<64, 128, 2, 2, EPI, 64, 4, 4, true>(a, s);
        if (a.M <= 128) return run_bf16<128, 128, 2, 2, EPI, 64, 4, 4, true>(a, s);
        if (a.M <= 256) return run_bf16<256, 128, 4, 2, EPI, 64, 3, 3, true>(a, s);
        if (a.M > 896) {
            // the row tile whose rounds of workgroups over 256 CUs cost least, a round costing
            // its tile's rows (M = 1024: 256x256 tiles, two rounds, 211 against 242 us)
            const long t192 = (long)((a.M + 191) / 192) * ((a.N + 127) / 128);
            const long t256 = (long)((a.M + 255) / 256) * ((a.N + 127) / 128);
            if ((t256 + 255) / 256 * 256 < (t192 + 255) / 256 * 192) return run_bf16<256, 256, 2, 4, EPI>(a, s);
            return run_bf16<192, 256, 2, 4, EPI>(a, s);
        }
        const int pad128 = (a.M + 127) / 128 * 128 - a.M, pad192 = (a.M + 191) / 192 * 192 - a.M;
        const int w128 = (a.M + 127) / 128 * ((a.N + 127) / 128), w192 = (a.M + 191) / 192 * ((a.N + 255) / 256);
        if ((w128 > 512 && w192 <= 256) || pad192 <= pad128) return run_bf16<192, 256, 2, 4, EPI>(a, s);
        return run_bf16<128, 128, 2, 2, EPI>(a, s);
    } else {
        // the blocked LM head of 33..64 rows: 64x128 tiles (16 KB runs per stage) 49.5 -> 46.9 us
        if (EPI == EPI_STORE_F32 && a.b_blocked && a.M > 32 && a.M <= 64)
            return run_bf16<64, 128, 2, 2, EPI, 64, 4, 4, true>(a, s);
        if (a.M <= 64) return run_bf16<64, 64, 2, 2, EPI, 64, 4, 4, true>(a, s);
        const bool split = EPI == EPI_ADD_F32 && a.partial && a.splits > 1;
        if (split && a.M <= 128) return run_bf16<128, 64, 2, 2, EPI, 64, 4, 4, true>(a, s);
        if (EPI != EPI_ADD_F32 && a.M <= 128) return run_bf16<128, 128, 2, 2, EPI, 64, 4, 4, true>(a, s);
        // stored rows of 129..256 (the LM head of up to 256 decode rows): one 256-row tile, the
        // weights streamed once
        if (EPI == EPI_STORE_F32 && a.M <= 256) return run_bf16<256, 128, 4, 2, EPI, 64, 3, 3, true>(a, s);
        if (split && a.wide && a.M > 128 && a.M <= 256) return run_bf16<256, 256, 2, 4, EPI>(a, s);
        if (split && a.M <= 256) return run_bf16<128, 128, 2, 2, EPI, 64, 4, 4, false>(a, s);
        if (split && a.M <= 896) return run_bf16<128, 128, 2, 2, EPI>(a, s);
        if (EPI == EPI_ADD_F32 && a.partial && a.M > 896) return run_bf16<256, 256, 2, 4, EPI>(a, s);
        if (EPI == EPI_ADD_F32) return run_bf16<128, 128, 4, 2, EPI>(a, s);
        // fp32 rows of a large QKV projection (rotated by a row kernel): one round of big tiles
        if (a.M > 1280) return a.M <= 1728 ? run_bf16<192, 256, 2, 4, EPI>(a, s) : run_bf16<256, 256, 2, 4, EPI>(a, s);
        return run_bf16<128, 128, 2, 2, EPI>(a, s);
    }
}

}  // namespace

// Split-K factor for a residual-add projection on the bf16 path, matched to the tiles
// dispatch_bf16 uses with it.  Each split takes a run of whole 64-deep stages (the stages dealt
// as evenly as the count allows), at least 512 deep.  1 = no split.
//  - M <= 64 (64x64 tiles): the factor whose workgroups fill the last round over 256 CUs best,
//    the smaller one on a tie;
//  - 64 < M <= 896, from measurements of the 7B projections: 4 up to M = 640 (64x64 or 128x128
//    tiles; weight streaming wants many workgroups), then 2;
//  - M > 896 (256x256 tiles, one workgroup per CU): the factor with the least (rounds of
//    workgroups over 256 CUs) x (stages per split), the smaller one on a tie.  The copies of a
//    round's stages bound these launches, so a second round that is only partly full costs as
//    much as the first (M = 1568: split 2 fills one round with 224 workgroups).
int gemm_add_splits(int M, int N, int K, int max_splits) {
    const int stages = K / BK;
    auto valid = [&](int s) { return s <= max_splits && K % BK == 0 && K / s >= 512; };
    if (M > 896) {
        const long tiles = (long)((M + 255) / 256) * ((N + 255) / 256);
        int best = 1;
        long best_cost = -1;
        for (int s = 1; s <= max_splits; ++s) {
            if (s > 1 && !valid(s)) continue;
            const long cost = (tiles * s + 255) / 256 * ((stages + s - 1) / s);
            if (best_cost < 0 || cost < best_cost) { best = s; best_cost = cost; }
        }
        return best;
    }
    if (M > 64) {
        int s = M <= 640 ? 4 : 2;
        while (s > 1 && !valid(s)) s /= 2;
        return s;
    }
    const long tiles = (long)((M + 63) / 64) * ((N + 63) / 64);
    auto fill = [](long w) { const long rounds = (w + 255) / 256; return (double)w / (double)(rounds * 256); };
    int best = 1;
    double best_fill = fill(tiles);
    for (int s = 2; s <= max_splits; ++s) {
        if (!valid(s)) continue;
        const double f = fill(tiles * s);
        if (f > best_fill + 1e-9) { best = s; best_fill = f; }
    }
    return best;
}

// dst [ceil(rows/64)][cols/64][64][64] <- src [rows][cols] (bf16), one 16-byte piece per thread
// step; rows past `rows` in the last row block are zero
__global__ __launch_bounds__(256) void block_weights_kernel(const uint4 *src, uint4 *dst, int rows, int cols) {
    const int cpr = cols / 8;                              // 16-byte pieces per source row
    const size_t total = (size_t)((rows + 63) / 64) * 64 * cpr;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (size_t)gridDim.x * 256) {
        const int c = (int)(i % 8);                        // piece within the block row
        const size_t q = i / 8;
        const int r = (int)(q % 64);                       // row within the block
        const size_t bq = q / 64;                          // block index: rb * (cols / 64) + cb
        const int cb = (int)(bq % (cols / 64));
        const int row = (int)(bq / (cols / 64)) * 64 + r;
        dst[i] = row < rows ? src[(size_t)row * cpr + cb * 8 + c] : uint4{0, 0, 0, 0};
    }
}

hipError_t launch_block_weights(const void *src, void *dst, int rows, int cols, hipStream_t s) {
    const size_t total = (size_t)((rows + 63) / 64) * 64 * (cols / 8);
    const int blocks = (int)std::min<size_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(block_weights_kernel, dim3(blocks), dim3(256), 0, s, (const uint4 *)src, (uint4 *)dst,
                       rows, cols);
    return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int epi, const GemmArgs &a, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    if (a.b_blocked && dtype != 1) return hipErrorInvalidValue;
    if (dtype == 1) {
        switch (epi) {
            case EPI_STORE_F32: return dispatch_bf16<EPI_STORE_F32>(a, s);
            case EPI_ADD_F32: return dispatch_bf16<EPI_ADD_F32>(a, s);
            case EPI_QKV_ROPE:
                if (a.rope.hd != 64 && a.rope.hd != 128) return hipErrorInvalidValue;
                return dispatch_bf16<EPI_QKV_ROPE>(a, s);
            default: return dispatch_bf16<EPI_SWIGLU>(a, s);
        }
    }
    if (epi == EPI_QKV_ROPE) return hipErrorInvalidValue;   // fp32 path: GEMM, then rope_append
    dim3 grid((a.N + 63) / 64, (a.M + 63) / 64);
    switch (epi) {
        case EPI_STORE_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, dim3(256), 0, s, a); break;
        case EPI_ADD_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_ADD_F32>, grid, dim3(256), 0, s, a); break;
        default: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace orthrus
