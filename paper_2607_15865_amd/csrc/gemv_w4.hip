// W4A16 GEMV for the decode stage, one kernel per linear (B <= 8 rows):
// y[b][n] = sum_k x[b][k] W[k][n].  The INT8 and F16 weight formats go
// through the same kernel with their own fragment unpack (gemv_core.h).
//
// Block: 512 threads = 8 waves on a pair of column tiles (64 device columns:
// a RoPE pair of q/k blocks, a gate/up pair, or two residual tiles) and the
// block's k range; the waves split the k range evenly and each streams its
// share through the register ring of the GEMV core (gemv_core.h).  The wave
// partials meet in LDS in a fixed order.  Grid: (N_dev / 64, ksplit); with
// ksplit > 1 the residual epilogue adds into an output that an earlier
// kernel initialised.
//
// Optional prologue: RMSNorm of the fp32 rows (every block reduces the whole
// row; the rows are small and L2-resident), rounded to bf16.  The first
// weight tiles are requested before the prologue runs.  (For 4 rows or more
// the caller normalises the rows once beforehand instead and passes them as
// fp16: the per-block reduction then costs more than the extra launch.)
#include "common.h"
#include "gemv_core.h"
#include "launch.h"

namespace {

constexpr int NW = 8;            // waves per block
constexpr int MAXB = 8;
constexpr int RING = 8;          // 1 KB tiles in flight per wave (the 8- and 16-bit formats' larger
                                 // tiles: the same bytes in flight)

// WF: weight format (WeightFormat); the 8-bit format always has zero points (ZP)
template <int EPI, bool NORM, bool ZP, bool G32, int WF>
__global__ void __launch_bounds__(NW * 64) gemv_w4_kernel(GemvArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const DevLinear& W = a.W;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int pair = blockIdx.x;
    const int KB = W.K_pad / 64;
    const int kb_lo = (int)((long long)blockIdx.y * KB / a.ksplit);
    const int kb_hi = (int)((long long)(blockIdx.y + 1) * KB / a.ksplit);
    const int klo = kb_lo * 64, klen = (kb_hi - kb_lo) * 64;
    const int ldx = klen + 8;
    const int B = a.B;
    const int nkb = kb_hi - kb_lo;
    // the activation rows, and after the main loop the wave partials over them
    const int reg0 = max(B * ldx * 2, NW * 2 * B * 32 * 4);
    f16* xs = reinterpret_cast<f16*>(smem);                                   // [B][ldx]
    float* red = reinterpret_cast<float*>(smem);                              // [NW][2][B][32]
    f16* zero = reinterpret_cast<f16*>(smem + reg0);                          // [64]
    float* c64 = reinterpret_cast<float*>(zero + 64);                         // [nkb][GEMV_ROWS]
    // [2 nkb][GEMV_ROWS], present only with zero points or groups of 32
    float2* uv32 = reinterpret_cast<float2*>(c64 + nkb * GEMV_ROWS);
    float* rinv = reinterpret_cast<float*>(uv32 + ((ZP || G32) ? 2 * nkb * GEMV_ROWS : 0));  // [MAXB]
    float* tot = rinv + MAXB;                                                 // [MAXB][64]

    // this wave's k-tiles of both column tiles
    const Run run{pair * 2, pair * 2 + 2, kb_lo + wave * nkb / NW, kb_lo + (wave + 1) * nkb / NW};
    constexpr int RD = RING >> WF;
    TileRing<RD, G32, WF> R;
    RunCursor q;
    if (run.ka < run.kz) ring_prefetch<RD, ZP, G32>(W, run, R, q);

    // side copy (e.g. residual initialisation of the next accumulation)
    if (a.copy_n > 0) {
        const int nthreads = gridDim.x * gridDim.y * blockDim.x;
        for (int i = (blockIdx.y * gridDim.x + blockIdx.x) * blockDim.x + tid; i < a.copy_n; i += nthreads)
            a.copy_dst[i] = a.copy_src[i];
    }

    // ---- prologue: activation slice into LDS
    if (NORM) {
        // wave b reduces row b; 16-byte loads, unrolled so that 8 are in
        // flight at once (a loop that waits for each load pays one L2 round
        // trip per step)
        const int K = W.K;
        for (int b = wave; b < B; b += NW) {
            const float* xr = a.x_f32 + (size_t)b * K;
            float ss = 0.f;
#pragma unroll 8
            for (int k = lane * 4; k < K; k += 256) {
                const float4 v = *reinterpret_cast<const float4*>(xr + k);
                ss += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
            }
            ss = wave_sum(ss);
            if (lane == 0) rinv[b] = 1.0f / sqrtf(ss / (float)K + a.eps);
        }
        __syncthreads();
        // the block's k slice, 4 elements per thread and pass
        const int k4n = klen / 4;
        bool bad = false;
#pragma unroll 4
        for (int i = tid; i < B * k4n; i += NW * 64) {
            const int b = i / k4n, k = 4 * (i - b * k4n);
            const float4 v = *reinterpret_cast<const float4*>(a.x_f32 + (size_t)b * K + klo + k);
            const uint2 g = *reinterpret_cast<const uint2*>(a.gamma + klo + k);
            const float rb = rinv[b];
            f16 o[4] = {act_f16(v.x * rb * __uint_as_float(g.x << 16), bad),
                        act_f16(v.y * rb * __uint_as_float(g.x & 0xFFFF0000u), bad),
                        act_f16(v.z * rb * __uint_as_float(g.y << 16), bad),
                        act_f16(v.w * rb * __uint_as_float(g.y & 0xFFFF0000u), bad)};
            *reinterpret_cast<uint2*>(xs + b * ldx + k) = *reinterpret_cast<const uint2*>(o);
        }
        flag_range(a.ep.err, bad);
    } else {
        const int nv = klen / 8;
#pragma unroll 4
        for (int i = tid; i < B * nv; i += NW * 64) {
            const int b = i / nv, v = i - b * nv;
            *reinterpret_cast<u32x4*>(xs + b * ldx + v * 8) =
                *reinterpret_cast<const u32x4*>(a.x_f16 + (size_t)b * a.ldx + klo + v * 8);
        }
    }
    if (tid < 8) reinterpret_cast<u32x4*>(zero)[tid] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    gemv_prep(xs - klo, ldx, c64 - kb_lo * GEMV_ROWS, (ZP || G32) ? uv32 - 2 * kb_lo * GEMV_ROWS : nullptr, B, klo,
              klen, tid, NW * 64);
    __syncthreads();

    // ---- main loop: partial sums of this wave's two tiles, kept in registers
    const int h = lane >> 5, c = lane & 31;
    const GemvAct xa{xs - klo, ldx, c64 - kb_lo * GEMV_ROWS, uv32 - 2 * kb_lo * GEMV_ROWS, zero};
    float p0[4] = {0.f, 0.f, 0.f, 0.f}, p1[4] = {0.f, 0.f, 0.f, 0.f};
    if (run.ka < run.kz) {
        gemv_run<RD, ZP, G32>(W, run, xa, B, R, q, [&](int t, const float (&out)[4]) {
            if (t == pair * 2) {
#pragma unroll
                for (int r = 0; r < 4; r++) p0[r] = out[r];
            } else {
#pragma unroll
                for (int r = 0; r < 4; r++) p1[r] = out[r];
            }
        });
    }
    __syncthreads();   // every wave is done with the activation rows
#pragma unroll
    for (int r = 0; r < 4; r++) {
        const int b = 4 * h + r;
        if (b < B) {
            red[((wave * 2 + 0) * B + b) * 32 + c] = p0[r];
            red[((wave * 2 + 1) * B + b) * 32 + c] = p1[r];
        }
    }
    __syncthreads();
    for (int i = tid; i < B * 64; i += NW * 64) {
        const int b = i / 64, cc = i % 64;
        const int tt = cc / 32, c2 = cc % 32;
        float v = 0.f;
        for (int w = 0; w < NW; w++) v += red[((w * 2 + tt) * B + b) * 32 + c2];
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
        bool bad = false;
        for (int i = tid; i < B * 32; i += NW * 64) {
            const int b = i / 32, cc = i % 32;
            const float gv = tot[b * 64 + cc], uv = tot[b * 64 + 32 + cc];
            a.ep.act_out[(size_t)b * a.ep.F_pad + pair * 32 + cc] = act_f16(silu(gv) * uv, bad);
        }
        flag_range(a.ep.err, bad);
    } else {
        for (int i = tid; i < B * 32; i += NW * 64) {
            const int b = i / 32, cc = i % 32;
            const int slot = a.ep.slot_dev ? a.ep.slot_dev[b] : a.ep.slot_base + b;
            epi_qkv_pair(a.ep, b, pair * 64, cc, tot[b * 64 + cc], tot[b * 64 + 32 + cc], slot, b);
        }
    }
}

template <int EPI, bool NORM, bool ZP, bool G32, int WF>
int launch_t(const GemvArgs& a, hipStream_t stream) {
    const int KB = a.W.K_pad / 64;
    const int kmax = (KB + a.ksplit - 1) / a.ksplit * 64;
    const size_t smem = std::max((size_t)a.B * (kmax + 8) * 2, (size_t)NW * 2 * a.B * 32 * 4) + 128 +
                        (size_t)(kmax / 64) * GEMV_ROWS * ((ZP || G32) ? 20 : 4) + (MAXB + MAXB * 64) * sizeof(float);
    if (smem > 160 * 1024) return -1;
    static LdsLimit lim;
    if (ensure_lds_limit(lim, (const void*)gemv_w4_kernel<EPI, NORM, ZP, G32, WF>, smem)) return -1;
    dim3 grid(a.W.N_dev / 64, a.ksplit);
    hipLaunchKernelGGL((gemv_w4_kernel<EPI, NORM, ZP, G32, WF>), grid, dim3(NW * 64), smem, stream, a);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <bool ZP, bool G32, int WF = WF_INT4>
int launch_zp(int epi, bool norm, const GemvArgs& a, hipStream_t stream) {
    if (epi == EPI_QKV)
        return norm ? launch_t<EPI_QKV, true, ZP, G32, WF>(a, stream) : launch_t<EPI_QKV, false, ZP, G32, WF>(a, stream);
    if (epi == EPI_SWIGLU)
        return norm ? launch_t<EPI_SWIGLU, true, ZP, G32, WF>(a, stream)
                    : launch_t<EPI_SWIGLU, false, ZP, G32, WF>(a, stream);
    if (epi == EPI_RESID && !norm) return launch_t<EPI_RESID, false, ZP, G32, WF>(a, stream);
    return -1;
}

}  // namespace

int launch_gemv_w4(int epi, bool norm, const GemvArgs& a, hipStream_t stream) {
    if (a.B < 1 || a.B > MAXB) return -1;
    if (a.W.wf == WF_INT8) return a.W.sz ? launch_zp<true, false, WF_INT8>(epi, norm, a, stream) : -1;
    if (a.W.wf == WF_F16) return launch_zp<false, false, WF_F16>(epi, norm, a, stream);
    const bool g32 = a.W.lgG == 5;
    if (a.W.sz) return g32 ? launch_zp<true, true>(epi, norm, a, stream) : launch_zp<true, false>(epi, norm, a, stream);
    return g32 ? launch_zp<false, true>(epi, norm, a, stream) : launch_zp<false, false>(epi, norm, a, stream);
}
