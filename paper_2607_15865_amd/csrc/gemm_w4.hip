// W4A16 GEMM for the prefill stages: Y[M][N] = X[M][K] * W[K][N] on the
// 32x32x16 fp16 MFMA with fp32 accumulation.
//
// X is an activation already rounded to bf16 and held as fp16 (exact), so the
// MFMA sees exactly the W4BF16 operand values.  W is used exactly: the B
// fragment of every k16 step is (code - zero) as fp16 integers and the group
// scale is applied in fp32.  The scale is carried as a running ratio: the
// accumulator u holds sum_g s_g T_g / s_cur, and at the start of group g it is
// multiplied by s_{g-1} / s_g, so one VALU multiply per output per group and
// no second accumulator set are needed; the epilogue multiplies by s_last.
//
// Block: 256 threads = 4 waves in a 2 x 2 grid, block tile 128 x 128, wave
// tile 64 x 64 (2 x 2 MFMA tiles).  The X tile (128 x 64 per k-block) is
// staged in LDS (double buffered); each wave reads its weight tiles (1 KB,
// one 16-byte load per lane) straight from global memory.
#include "common.h"
#include "launch.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDA = BK + 8;      // fp16 elements per LDS row (16-byte pad)

template <int EPI>
__global__ void __launch_bounds__(256) gemm_w4_kernel(const f16* __restrict__ X, int M, int ldx,
                                                      DevLinear W, EpiArgs ep) {
    __shared__ __attribute__((aligned(16))) f16 As[2][BM * LDA];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM;
    const int n0 = blockIdx.x * BN;
    const int h = lane >> 5, c = lane & 31;
    const int KB = W.K_pad / BK;
    const int Gm1 = (1 << W.lgG) - 1;      // group size in k, minus one

    // weight tiles of this wave: n-tiles nt0, nt0 + 1
    const int nt0 = (n0 + wn * 64) / 32;
    const u32x4* wt0 = reinterpret_cast<const u32x4*>(W.qw) + ((size_t)nt0 * KB) * 64 + lane;
    const u32x4* wt1 = wt0 + (size_t)KB * 64;
    const int col0 = nt0 * 32 + c, col1 = col0 + 32;

    // global -> LDS mapping of the X tile: 128 rows x 64 halves = 1024 x 16 B
    auto load_x = [&](int kb, u32x4 (&r)[4]) {
#pragma unroll
        for (int i = 0; i < 4; i++) {
            int idx = tid + i * 256;
            int row = idx >> 3, seg = idx & 7;
            int m = m0 + row;
            if (m < M)
                r[i] = *reinterpret_cast<const u32x4*>(X + (size_t)m * ldx + kb * BK + seg * 8);
            else
                r[i] = u32x4{0, 0, 0, 0};
        }
    };
    auto store_x = [&](int buf, const u32x4 (&r)[4]) {
#pragma unroll
        for (int i = 0; i < 4; i++) {
            int idx = tid + i * 256;
            int row = idx >> 3, seg = idx & 7;
            *reinterpret_cast<u32x4*>(&As[buf][row * LDA + seg * 8]) = r[i];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) acc[i][j] = f32x16{};

    const DqConst dq = dq_const();
    u32x4 xr[4];
    load_x(0, xr);
    store_x(0, xr);
    u32x4 b0 = wt0[0], b1 = wt1[0];
    ZeroOff zo0 = zero_off(W.zeros ? (float)W.zeros[col0] : 8.0f);
    ZeroOff zo1 = zero_off(W.zeros ? (float)W.zeros[col1] : 8.0f);

    for (int kb = 0; kb < KB; kb++) {
        __syncthreads();
        const int buf = kb & 1;
        u32x4 nb0 = b0, nb1 = b1;
        if (kb + 1 < KB) {
            load_x(kb + 1, xr);
            nb0 = wt0[(size_t)(kb + 1) * 64];
            nb1 = wt1[(size_t)(kb + 1) * 64];
        }
#pragma unroll
        for (int s = 0; s < 4; s++) {
            const int k = kb * BK + s * 16;
            if ((k & Gm1) == 0 && k > 0) {
                const int g = k >> W.lgG;
                const float r0 = W.ratios[(size_t)g * W.N_dev + col0];
                const float r1 = W.ratios[(size_t)g * W.N_dev + col1];
#pragma unroll
                for (int i = 0; i < 2; i++)
#pragma unroll
                    for (int e = 0; e < 16; e++) { acc[i][0][e] *= r0; acc[i][1][e] *= r1; }
                if (W.zeros) {
                    zo0 = zero_off((float)W.zeros[(size_t)g * W.N_dev + col0]);
                    zo1 = zero_off((float)W.zeros[(size_t)g * W.N_dev + col1]);
                }
            }
            f16x8 bf0 = dequant8(b0[s], zo0, dq);
            f16x8 bf1 = dequant8(b1[s], zo1, dq);
#pragma unroll
            for (int i = 0; i < 2; i++) {
                const f16* ap = &As[buf][(wm * 64 + i * 32 + c) * LDA + s * 16 + h * 8];
                f16x8 af = *reinterpret_cast<const f16x8*>(ap);
                acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af, bf0, acc[i][0], 0, 0, 0);
                acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af, bf1, acc[i][1], 0, 0, 0);
            }
        }
        if (kb + 1 < KB) store_x(buf ^ 1, xr);
        b0 = nb0; b1 = nb1;
    }

    const float sl0 = W.slast[col0], sl1 = W.slast[col1];
    // rows of register e: 8*(e/4) + 4*h + (e%4)
#pragma unroll
    for (int i = 0; i < 2; i++) {
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = m0 + wm * 64 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
            if (m >= M) continue;
            const float v0 = acc[i][0][e] * sl0;
            const float v1 = acc[i][1][e] * sl1;
            if (EPI == EPI_RESID) {
                const size_t o = (size_t)m * W.N;
                ep.out_f32[o + col0] = ep.resid[o + col0] + v0;
                ep.out_f32[o + col1] = ep.resid[o + col1] + v1;
            } else if (EPI == EPI_SWIGLU) {
                // tile pair (2j, 2j+1) = gate block j, up block j
                const int f = (nt0 / 2) * 32 + c;
                ep.act_out[(size_t)m * ep.F_pad + f] = act_f16(silu(v0) * v1);
            } else {
                epi_qkv_pair(ep, m, nt0 * 32, c, v0, v1, ep.slot_base + (m - 0), 0);
            }
        }
    }
}

}  // namespace

int launch_gemm_w4(int epi, const f16* X, int M, int ldx, const DevLinear& W, const EpiArgs& ep,
                   hipStream_t stream) {
    dim3 grid(W.N_dev / BN, (M + BM - 1) / BM);
    dim3 block(256);
    switch (epi) {
        case EPI_QKV: hipLaunchKernelGGL(gemm_w4_kernel<EPI_QKV>, grid, block, 0, stream, X, M, ldx, W, ep); break;
        case EPI_RESID: hipLaunchKernelGGL(gemm_w4_kernel<EPI_RESID>, grid, block, 0, stream, X, M, ldx, W, ep); break;
        case EPI_SWIGLU: hipLaunchKernelGGL(gemm_w4_kernel<EPI_SWIGLU>, grid, block, 0, stream, X, M, ldx, W, ep); break;
        default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
