// LoRA shrink x A^T of the embedding rows (the first half of the low-rank update; the second,
// U B^T, runs inside the projection GEMM's epilogue).  The shared-backbone deployment of the
// paper adapts the generator into the embedding model this way (Section 2, parameter sharing).
//
// bf16 path: one workgroup per 32 rows x 64 columns of U, eight waves splitting K eight ways,
// each accumulating a 32x64 fp32 block on v_mfma_f32_32x32x16_bf16 with operands loaded straight
// from global memory (x rows and A rows are both K-contiguous, the MFMA operand layout); the
// eight partial blocks are summed in LDS in a fixed order (deterministic), scaled, masked to the
// row's adapter and stored as two bf16 arrays, the rounding of each value and its remainder, so
// the expand can use U to about 16 significant bits (a single bf16 U doubles the adapter
// path's rounding error at 7B shapes).  fp32 path: one thread per output, plain dot products.
#include "common.hpp"

namespace orthrus {

namespace {

__global__ __launch_bounds__(512) void lora_shrink_bf16(LoraShrink p) {
    __shared__ float red[8][32][65];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m0 = blockIdx.x * 32, c0 = blockIdx.y * 64;
    const int ldu = p.n * p.r;
    const int kw = p.K / 8;                        // this wave's slice of K (a multiple of 16)
    const int k_begin = wave * kw + 8 * (lane >> 5);
    const int row = min(m0 + (lane & 31), p.rows - 1);
    const bf16 *xr = (const bf16 *)p.x + (size_t)row * p.ldx + k_begin;
    const bf16 *br[2];
    bool bok[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
        const int col = c0 + f * 32 + (lane & 31);
        bok[f] = col < ldu;
        const int j = bok[f] ? col / p.r : 0, kk = bok[f] ? col % p.r : 0;
        br[f] = (const bf16 *)p.a[j] + (size_t)kk * p.K + k_begin;
    }
    f32x16 acc[2];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[f][e] = 0.f;
    const bf16x8 zero = {};
    for (int k = 0; k < kw; k += 16) {
        const bf16x8 xa = *(const bf16x8 *)(xr + k);
#pragma unroll
        for (int f = 0; f < 2; ++f) {
            const bf16x8 bb = bok[f] ? *(const bf16x8 *)(br[f] + k) : zero;
            acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa, bb, acc[f], 0, 0, 0);
        }
    }
    // D layout: column lane % 32, row 8 (e / 4) + 4 (lane / 32) + e % 4
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int e = 0; e < 16; ++e)
            red[wave][(e >> 2) * 8 + (lane >> 5) * 4 + (e & 3)][f * 32 + (lane & 31)] = acc[f][e];
    __syncthreads();
    for (int o = threadIdx.x; o < 32 * 64; o += 512) {
        const int rr = o >> 6, cc = o & 63, grow = m0 + rr, gcol = c0 + cc;
        if (grow >= p.rows || gcol >= ldu) continue;
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < 8; ++w) sum += red[w][rr][cc];
        const int j = gcol / p.r;
        const float v = p.row_adapter[grow] == j ? sum * p.scale[j] : 0.f;
        const bf16 hi = (bf16)v;
        ((bf16 *)p.u)[(size_t)grow * ldu + gcol] = hi;
        ((bf16 *)p.u_lo)[(size_t)grow * ldu + gcol] = (bf16)(v - to_f32<bf16>(hi));
    }
}

__global__ __launch_bounds__(256) void lora_shrink_f32(LoraShrink p) {
    const int row = blockIdx.x, ldu = p.n * p.r;
    const float *x = (const float *)p.x + (size_t)row * p.ldx;
    const int ra = p.row_adapter[row];
    for (int c = threadIdx.x; c < ldu; c += 256) {
        const int j = c / p.r, kk = c % p.r;
        float v = 0.f;
        if (ra == j) {
            const float *a = (const float *)p.a[j] + (size_t)kk * p.K;
            for (int i = 0; i < p.K; ++i) v = fmaf(x[i], a[i], v);
            v *= p.scale[j];
        }
        ((float *)p.u)[(size_t)row * ldu + c] = v;
    }
}

}  // namespace

hipError_t launch_lora_shrink(int dtype, const LoraShrink &p, hipStream_t s) {
    if (p.rows <= 0 || p.n <= 0) return hipSuccess;
    if (dtype == 1) {
        if (p.K % 128 || p.r % 16) return hipErrorInvalidValue;
        dim3 grid((p.rows + 31) / 32, (p.n * p.r + 63) / 64);
        hipLaunchKernelGGL(lora_shrink_bf16, grid, dim3(512), 0, s, p);
    } else {
        hipLaunchKernelGGL(lora_shrink_f32, dim3(p.rows), dim3(256), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace orthrus
