// Dense projections of the step: C[M][N] = A[M][K] * W[N][K]^T over the concatenated token
// batch (QKV, attention output, gate/up, down, LM head), with fused epilogues.
//
// bf16 path: CDNA4 MFMA v_mfma_f32_32x32x16_bf16, 256 threads (4 wave64s in a WM x WN grid),
// K staged 64 elements at a time through two LDS buffers with a register prefetch of the
// next stage, so each K step costs one barrier.  LDS rows are 128 B; 16-byte chunks are
// XOR-swizzled by row so the per-lane 16-byte operand reads of one MFMA spread over banks.
// Tiles are mapped to blocks so that consecutive tiles of one weight column block land on
// the same XCD (blocks are dealt round-robin to the 8 XCDs), which keeps re-reads of a
// weight tile inside one L2.
// fp32 path: plain LDS-tiled FMA kernel (64x64 tile, 4x4 per thread) for exact checks.
#include "common.hpp"

namespace orthrus {

namespace {

constexpr int BK = 64;

__device__ __forceinline__ int swz(int row, int chunk) {
    return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
}

__device__ __forceinline__ float silu(float g) { return g / (1.f + __expf(-g)); }

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmArgs a) {
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 32, FN = TN / 32;
    constexpr int A_LOADS = BM * 8 / 256, B_LOADS = BN * 8 / 256;
    constexpr int STAGE = (BM + BN) * BK * 2;
    static_assert(WM * WN == 4, "four waves");
    static_assert(FM >= 1 && FN >= 1 && (EPI != EPI_SWIGLU || FN % 2 == 0), "tile shape");
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int mt = (a.M + BM - 1) / BM;
    const int total = gridDim.x;
    const int b = blockIdx.x;
    const int t = (total % 8 == 0) ? (b % 8) * (total / 8) + b / 8 : b;
    const int n_tile = t / mt, m_tile = t % mt;
    const int m0 = m_tile * BM;
    constexpr int COLS = EPI == EPI_SWIGLU ? BN / 2 : BN;  // output columns per tile
    const int n0 = n_tile * COLS;

    const char *Abase = (const char *)a.A;
    const size_t lda_b = (size_t)a.lda * 2, ldb_b = (size_t)a.K * 2;
    uint32_t a_off[A_LOADS], b_off[B_LOADS];
    const char *b_src[B_LOADS];
    int a_lds[A_LOADS], b_lds[B_LOADS];
    const int ch = tid & 7;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        const int row = (tid >> 3) + 32 * i;
        const int grow = min(m0 + row, a.M - 1);
        a_off[i] = (uint32_t)(grow * lda_b + ch * 16);
        a_lds[i] = swz(row, ch);
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int r = (tid >> 3) + 32 * i;
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
        grow = min(grow, a.N - 1);
        b_src[i] = src;
        b_off[i] = (uint32_t)(grow * ldb_b + ch * 16);
        b_lds[i] = swz(BM + r, ch);
    }

    u32x4 ra[A_LOADS], rb[B_LOADS];
    auto gload = [&](int kt) {
        const uint32_t kb = (uint32_t)kt * (BK * 2);
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) ra[i] = *(const u32x4 *)(Abase + a_off[i] + kb);
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) rb[i] = *(const u32x4 *)(b_src[i] + b_off[i] + kb);
    };
    auto lstore_to = [&](char *s) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) *(u32x4 *)(s + a_lds[i]) = ra[i];
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) *(u32x4 *)(s + b_lds[i]) = rb[i];
    };
    auto lstore = [&](int buf) { lstore_to(smem + buf * STAGE); };
    int next_k = 0;
    auto gload_next = [&]() { gload(next_k); };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment rows of this lane; the swizzle key (row >> 1) & 7 is the same for every
    // 32-row fragment of the lane, so the LDS offsets differ only by constants
    const int arow = wm * TM + (lane & 31), brow = BM + wn * TN + (lane & 31);
    const int akey = (arow >> 1) & 7, bkey = (brow >> 1) & 7;
    bf16x8 fa[2][FM], fb[2][FN];
    auto lds_frag = [&](const char *s, int kk, int buf) {
        const int chk = kk * 2 + (lane >> 5);
#pragma unroll
        for (int mi = 0; mi < FM; ++mi)
            fa[buf][mi] = *(const bf16x8 *)(s + (arow + mi * 32) * 128 + ((chk ^ akey) << 4));
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
            fb[buf][ni] = *(const bf16x8 *)(s + (brow + ni * 32) * 128 + ((chk ^ bkey) << 4));
    };

    // One K stage per iteration, software-pipelined by hand (the scheduler is told the order):
    //   LDS fragments of k-step 0, then per k-step its MFMAs interleaved with the LDS reads of the
    //   next k-step's fragments; the next stage's global loads ride along k-step 0 and its LDS
    //   stores (other buffer, not read this iteration) along k-step 3.  One barrier per stage.
    constexpr int NMF = FM * FN, NFR = FM + FN, NLD = A_LOADS + B_LOADS;
    auto stage = [&](const char *s, char *s_next, bool more) {
        lds_frag(s, 0, 0);
        if (more) gload_next();
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            if (kk + 1 < BK / 16) lds_frag(s, kk + 1, (kk + 1) & 1);
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int ni = 0; ni < FN; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk & 1][mi], fb[kk & 1][ni],
                                                                          acc[mi][ni], 0, 0, 0);
            if (kk == BK / 16 - 1 && more) lstore_to(s_next);
        }
        // schedule: DS_READ=0x100, DS_WRITE=0x200, VMEM_READ=0x020, MFMA=0x008
        __builtin_amdgcn_sched_group_barrier(0x100, NFR, 0);
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
#pragma unroll
            for (int i = 0; i < NMF; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (kk == 0 && more) {
                    if (i < NLD) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                }
                if (kk + 1 < BK / 16 && i < NFR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                if (kk == BK / 16 - 1 && more && i < NLD) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
            }
        }
    };

    const int nk = a.K / BK;
    gload(0);
    lstore(0);
    __syncthreads();
    int kt = 0;
    for (; kt + 1 < nk; ++kt) {
        next_k = kt + 1;
        stage(smem + (kt & 1) * STAGE, smem + ((kt + 1) & 1) * STAGE, true);
        __syncthreads();
    }
    stage(smem + (kt & 1) * STAGE, nullptr, false);

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

template <int BM, int BN, int WM, int WN, int EPI>
hipError_t run_bf16(const GemmArgs &a, hipStream_t s) {
    const int mt = (a.M + BM - 1) / BM;
    const int cols = EPI == EPI_SWIGLU ? BN / 2 : BN;
    const int nt = (a.N + cols - 1) / cols;
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, EPI>), dim3(mt * nt), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int EPI>
hipError_t dispatch_bf16(const GemmArgs &a, hipStream_t s) {
    if (a.M <= 64) return run_bf16<64, 256, 1, 4, EPI>(a, s);
    const long long big = (long long)((a.M + 255) / 256) * ((a.N + (EPI == EPI_SWIGLU ? 127 : 255)) /
                                                             (EPI == EPI_SWIGLU ? 128 : 256));
    if (big >= 512) return run_bf16<256, 256, 2, 2, EPI>(a, s);
    return run_bf16<128, 128, 2, 2, EPI>(a, s);
}

}  // namespace

hipError_t launch_gemm(int dtype, int epi, const GemmArgs &a, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    if (dtype == 1) {
        switch (epi) {
            case EPI_STORE_F32: return dispatch_bf16<EPI_STORE_F32>(a, s);
            case EPI_ADD_F32: return dispatch_bf16<EPI_ADD_F32>(a, s);
            default: return dispatch_bf16<EPI_SWIGLU>(a, s);
        }
    }
    dim3 grid((a.N + 63) / 64, (a.M + 63) / 64);
    switch (epi) {
        case EPI_STORE_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, dim3(256), 0, s, a); break;
        case EPI_ADD_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_ADD_F32>, grid, dim3(256), 0, s, a); break;
        default: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace orthrus
