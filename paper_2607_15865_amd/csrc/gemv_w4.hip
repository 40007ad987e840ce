// W4A16 GEMV for the decode stage (B <= 8 rows): y[b][n] = sum_k x[b][k] W[k][n].
//
// HBM-streaming: every weight tile (32 columns x 64 k, 1 KB) is read once with
// one 16-byte load per lane.  Codes are turned into exact fp16 (code - zero)
// pairs in registers and dotted with the fp16-held bf16 activations by
// v_dot2_f32_f16 into a per-group fp32 sum, which is multiplied by the group
// scale.  The two lanes that share a column (k halves) meet with one shuffle,
// the waves that split K meet in LDS.
//
// Block: 512 threads = 8 waves on a pair of tiles (64 device columns: a RoPE
// pair of q/k blocks or a gate/up pair), 4 waves per tile splitting the
// block's k range.  Grid: (N_dev / 64, ksplit); with ksplit > 1 the residual
// epilogue adds into an output that an earlier kernel initialised.
//
// Optional prologue: RMSNorm of the fp32 rows (every block reduces the whole
// row; the rows are small and L2-resident), rounded to bf16.
#include "common.h"
#include "launch.h"

namespace {

constexpr int NW = 8;            // waves per block
constexpr int NSUB = NW / 2;     // waves per tile
constexpr int MAXB = 8;

__device__ __forceinline__ float scale_at(const DevLinear& W, int n, int g) {
    return (float)__builtin_bit_cast(f16, W.scales[(size_t)n * W.KG + g]);
}

template <int EPI, bool NORM>
__global__ void __launch_bounds__(NW * 64) gemv_w4_kernel(GemvArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const DevLinear& W = a.W;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pair = blockIdx.x;
    const int KB = W.K_pad / 64;
    const int kb_lo = (int)((long long)blockIdx.y * KB / a.ksplit);
    const int kb_hi = (int)((long long)(blockIdx.y + 1) * KB / a.ksplit);
    const int klo = kb_lo * 64, klen = (kb_hi - kb_lo) * 64;
    const int B = a.B;
    f16* xs = reinterpret_cast<f16*>(smem);                        // [B][klen]
    float* red = reinterpret_cast<float*>(smem + (size_t)MAXB * klen * 2);  // [NSUB][2][MAXB][32]
    float* rinv = red + NSUB * 2 * MAXB * 32;                        // [MAXB]
    float* tot = rinv + MAXB;                                        // [MAXB][64]

    // side copy (e.g. residual initialisation of the next accumulation)
    if (a.copy_n > 0) {
        const int nthreads = gridDim.x * gridDim.y * blockDim.x;
        for (int i = (blockIdx.y * gridDim.x + blockIdx.x) * blockDim.x + tid; i < a.copy_n; i += nthreads)
            a.copy_dst[i] = a.copy_src[i];
    }

    // ---- prologue: activation slice into LDS
    if (NORM) {
        const int K = W.K;
        for (int b = wave; b < B; b += NW) {
            const float* xr = a.x_f32 + (size_t)b * K;
            float ss = 0.f;
            for (int k = lane * 4; k < K; k += 256) {
                float4 v = *reinterpret_cast<const float4*>(xr + k);
                ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
            }
            ss = wave_sum(ss);
            if (lane == 0) rinv[b] = 1.0f / sqrtf(ss / (float)K + a.eps);
        }
        __syncthreads();
        for (int i = tid; i < B * klen; i += NW * 64) {
            const int b = i / klen, k = i - b * klen;
            const float g = bf16_bits_to_f32(a.gamma[klo + k]);
            xs[i] = act_f16(a.x_f32[(size_t)b * K + klo + k] * rinv[b] * g);
        }
    } else {
        const int nv = klen / 8;
        for (int i = tid; i < B * nv; i += NW * 64) {
            const int b = i / nv, v = i - b * nv;
            *reinterpret_cast<u32x4*>(xs + (size_t)b * klen + v * 8) =
                *reinterpret_cast<const u32x4*>(a.x_f16 + (size_t)b * a.ldx + klo + v * 8);
        }
    }
    __syncthreads();

    // ---- main loop
    const int t = wave & 1, sub = wave >> 1;
    const int h = lane >> 5, c = lane & 31;
    const int nt = pair * 2 + t;
    const int col = nt * 32 + c;
    const u32x4* tiles = reinterpret_cast<const u32x4*>(W.qw) + (size_t)nt * KB * 64 + lane;

    float acc[MAXB], gacc[MAXB];
#pragma unroll
    for (int b = 0; b < MAXB; b++) { acc[b] = 0.f; gacc[b] = 0.f; }
    int cur_g = -1;
    float sc = 0.f;
    f16x2 zo = zero_offset_pair(nullptr, 0);

    constexpr int DEPTH = 4;
    for (int kb0 = kb_lo + sub; kb0 < kb_hi; kb0 += NSUB * DEPTH) {
        u32x4 wv[DEPTH];
#pragma unroll
        for (int u = 0; u < DEPTH; u++) {
            const int kb = kb0 + u * NSUB;
            wv[u] = (kb < kb_hi) ? tiles[(size_t)kb * 64] : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < DEPTH; u++) {
            const int kb = kb0 + u * NSUB;
            if (kb >= kb_hi) break;
#pragma unroll
            for (int s = 0; s < 4; s++) {
                const int k = kb * 64 + s * 16 + h * 8;
                const int g = (kb * 64 + s * 16) >> W.lgG;
                if (g != cur_g) {
#pragma unroll
                    for (int b = 0; b < MAXB; b++) { acc[b] += sc * gacc[b]; gacc[b] = 0.f; }
                    cur_g = g;
                    sc = scale_at(W, col, g);
                    if (W.zeros) zo = zero_offset_pair(W.zeros, (size_t)col * W.KG + g);
                }
                const uint32_t wd = wv[u][s];
                const f16x2 d0 = dequant_pair(wd, 0, zo), d1 = dequant_pair(wd, 1, zo);
                const f16x2 d2 = dequant_pair(wd, 2, zo), d3 = dequant_pair(wd, 3, zo);
#pragma unroll
                for (int b = 0; b < MAXB; b++) {
                    if (b < B) {
                        const f16x8 xv = *reinterpret_cast<const f16x8*>(xs + (size_t)b * klen + (k - klo));
                        float v = gacc[b];
                        v = __builtin_amdgcn_fdot2(f16x2{xv[0], xv[1]}, d0, v, false);
                        v = __builtin_amdgcn_fdot2(f16x2{xv[2], xv[3]}, d1, v, false);
                        v = __builtin_amdgcn_fdot2(f16x2{xv[4], xv[5]}, d2, v, false);
                        v = __builtin_amdgcn_fdot2(f16x2{xv[6], xv[7]}, d3, v, false);
                        gacc[b] = v;
                    }
                }
            }
        }
    }
#pragma unroll
    for (int b = 0; b < MAXB; b++) acc[b] += sc * gacc[b];

    // ---- reduction: k halves (lanes l, l^32), then the waves of a tile
#pragma unroll
    for (int b = 0; b < MAXB; b++) acc[b] += __shfl_xor(acc[b], 32, 64);
    if (h == 0) {
#pragma unroll
        for (int b = 0; b < MAXB; b++)
            if (b < B) red[((sub * 2 + t) * MAXB + b) * 32 + c] = acc[b];
    }
    __syncthreads();
    for (int i = tid; i < B * 64; i += NW * 64) {
        const int b = i / 64, cc = i % 64;
        const int tt = cc / 32, c2 = cc % 32;
        float v = 0.f;
        for (int s2 = 0; s2 < NSUB; s2++) v += red[((s2 * 2 + tt) * MAXB + b) * 32 + c2];
        tot[b * 64 + cc] = v;
    }
    __syncthreads();

    // ---- epilogue
    if (EPI == EPI_RESID) {
        for (int i = tid; i < B * 64; i += NW * 64) {
            const int b = i / 64, cc = i % 64;
            const int n = pair * 64 + cc;
            float* o = a.ep.out_f32 + (size_t)b * W.N + n;
            if (a.ksplit == 1 && a.ep.resid)
                *o = a.ep.resid[(size_t)b * W.N + n] + tot[i];
            else
                atomicAdd(o, tot[i]);
        }
    } else if (EPI == EPI_SWIGLU) {
        for (int i = tid; i < B * 32; i += NW * 64) {
            const int b = i / 32, cc = i % 32;
            const float gv = tot[b * 64 + cc], uv = tot[b * 64 + 32 + cc];
            a.ep.act_out[(size_t)b * a.ep.F_pad + pair * 32 + cc] = act_f16(silu(gv) * uv);
        }
    } else {
        for (int i = tid; i < B * 32; i += NW * 64) {
            const int b = i / 32, cc = i % 32;
            const int slot = a.ep.slot_dev[b];
            epi_qkv_pair(a.ep, b, pair * 64, cc, tot[b * 64 + cc], tot[b * 64 + 32 + cc], slot, b);
        }
    }
}

template <int EPI, bool NORM>
int launch_t(const GemvArgs& a, hipStream_t stream) {
    const int KB = a.W.K_pad / 64;
    const int kmax = (KB + a.ksplit - 1) / a.ksplit * 64;
    const size_t smem = (size_t)MAXB * kmax * 2 + (NSUB * 2 * MAXB * 32 + MAXB + MAXB * 64) * sizeof(float);
    if (smem > 160 * 1024) return -1;
    if (smem > 64 * 1024 &&
        hipFuncSetAttribute((const void*)gemv_w4_kernel<EPI, NORM>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)smem) != hipSuccess)
        return -1;
    dim3 grid(a.W.N_dev / 64, a.ksplit);
    hipLaunchKernelGGL((gemv_w4_kernel<EPI, NORM>), grid, dim3(NW * 64), smem, stream, a);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_gemv_w4(int epi, bool norm, const GemvArgs& a, hipStream_t stream) {
    if (epi == EPI_QKV && norm) return launch_t<EPI_QKV, true>(a, stream);
    if (epi == EPI_SWIGLU && norm) return launch_t<EPI_SWIGLU, true>(a, stream);
    if (epi == EPI_RESID && !norm) return launch_t<EPI_RESID, false>(a, stream);
    return -1;
}
