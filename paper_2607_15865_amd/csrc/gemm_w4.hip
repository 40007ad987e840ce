// W4A16 GEMM for the prefill stages: Y[M][N] = X[M][K] * W[K][N] on the
// 32x32x16 fp16 MFMA with fp32 accumulation.
//
// X is an activation already rounded to bf16 and held as fp16 (exact), so the
// MFMA sees exactly the W4BF16 operand values.  W is used exactly: the B
// fragment of every k16 step is (code - zero) as fp16 integers (dequant8) and
// the group scale is applied in fp32.  The scale is carried as a running
// ratio: the accumulator u holds sum_g s_g T_g / s_cur, and at the start of
// group g it is multiplied by s_{g-1} / s_g, so one VALU multiply per output
// per group and no second accumulator set are needed; the epilogue multiplies
// by the scale of the last group of the k range.
//
// Block: 256 threads = 4 waves side by side along N.  Block tile BM x 256
// with BM = 32 * TM; wave tile BM x 64 (TM x 2 MFMA tiles), so a wave's two
// 32-column weight tiles are a RoPE pair or a gate/up pair and every
// dequantised weight fragment feeds TM MFMAs.  The X tile (BM x 64 per k
// tile) is staged in LDS (double buffered); each wave streams its own weight
// tiles (1 KB, one 16-byte load per lane) through a ring PF k-tiles deep.
//
// Split K: with S > 1 the k tiles are cut into S ranges, one block each.
// Every block stores its fp32 partial tile, and the last block of a tile to
// arrive (a per-tile counter) adds the S partials in range order and runs
// the epilogue, so the result does not depend on the arrival order.
//
// Block order: the blocks of one column block (its row blocks and k ranges)
// are placed on the same XCD (consecutive block ids go round robin over the
// 8 XCDs), so each weight column block is read from HBM into one L2.
#include "common.h"
#include "launch.h"

namespace {

constexpr int BN = 256, BK = 64;
constexpr int LDA = BK + 8;      // fp16 elements per LDS row (16-byte pad)
constexpr int PF = 4;            // weight k-tiles in flight per wave
constexpr int NXCD = 8;

struct GemmShape {
    int M, nrb, ncb, S, KB;
    float* part;                 // [S][M][N_dev] (S > 1)
    unsigned* cnt;               // [nrb * ncb] (S > 1), zero between calls
};

// GEN: zero points or groups of 32 (a group may start at either k half of a
// tile); otherwise groups of 64 or more without zero points.
template <int EPI, int TM, bool GEN>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) gemm_w4_kernel(const f16* __restrict__ X, int ldx, DevLinear W, EpiArgs ep,
                                                      GemmShape gs) {
    constexpr int BM = 32 * TM;
    __shared__ __attribute__((aligned(16))) f16 As[2][BM * LDA];
    __shared__ unsigned last_flag;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = lane >> 5, c = lane & 31;
    const int M = gs.M;

    // block -> (column block, row block, k range); the blocks of a column
    // block share an XCD when the column blocks divide evenly over the XCDs
    int cb, rb, sp;
    {
        const int lid = blockIdx.x;
        if (gs.ncb % NXCD == 0) {
            const int xcd = lid % NXCD, j = lid / NXCD;
            rb = j % gs.nrb;
            const int j2 = j / gs.nrb;
            sp = j2 % gs.S;
            cb = (j2 / gs.S) * NXCD + xcd;
        } else {
            rb = lid % gs.nrb;
            const int j2 = lid / gs.nrb;
            sp = j2 % gs.S;
            cb = j2 / gs.S;
        }
    }
    const int m0 = rb * BM;
    const int nt0 = cb * 8 + wave * 2;                  // first of this wave's two column tiles
    const bool wave_on = nt0 * 32 < W.N_dev;            // columns past N_dev: idle wave
    const int KB = gs.KB;
    const int kb_lo = sp * KB / gs.S, kb_hi = (sp + 1) * KB / gs.S;
    const int Gm1 = (1 << W.lgG) - 1;
    const int col0 = (wave_on ? nt0 : 0) * 32 + c, col1 = col0 + 32;
    const DqConst dq = dq_const();

    // ---- X tile: BM rows x 64 halves = BM * 8 segments of 16 bytes
    constexpr int XSEG = BM * 8 / 256;                  // per thread: 1, 2 or 4
    auto load_x = [&](int kb, u32x4 (&r)[XSEG]) {
#pragma unroll
        for (int i = 0; i < XSEG; i++) {
            const int idx = tid + i * 256, row = idx >> 3, seg = idx & 7;
            const int m = m0 + row;
            r[i] = m < M ? *reinterpret_cast<const u32x4*>(X + (size_t)m * ldx + kb * BK + seg * 8)
                         : u32x4{0, 0, 0, 0};
        }
    };
    auto store_x = [&](int buf, const u32x4 (&r)[XSEG]) {
#pragma unroll
        for (int i = 0; i < XSEG; i++) {
            const int idx = tid + i * 256, row = idx >> 3, seg = idx & 7;
            *reinterpret_cast<u32x4*>(&As[buf][row * LDA + seg * 8]) = r[i];
        }
    };

    // ---- weight ring: k-tile kb_lo + j in slot j % PF; the ratios (and zero
    // points) of the groups that start in the tile's two k halves travel with
    // it.  Loads past the range re-read the first tile (a cache hit), so every
    // slot is refilled unconditionally.
    const u32x4* wt0 = reinterpret_cast<const u32x4*>(W.qw) + (size_t)(wave_on ? nt0 : 0) * (W.K_pad / 64) * 64 + lane;
    const u32x4* wt1 = wt0 + (size_t)(W.K_pad / 64) * 64;
    constexpr int NH = GEN ? 2 : 1;                     // k halves with their own group parameters
    u32x4 rb0[PF], rb1[PF];
    float rr0[PF][NH], rr1[PF][NH];
    uint32_t rz[PF][NH];
    auto load_w = [&](int kb, int u) {
        const int kk = kb < kb_hi ? kb : kb_lo;
        rb0[u] = wt0[(size_t)kk * 64];
        rb1[u] = wt1[(size_t)kk * 64];
#pragma unroll
        for (int hh = 0; hh < NH; hh++) {
            const int g = (kk * 64 + 32 * hh) >> W.lgG;
            rr0[u][hh] = W.ratios[(size_t)g * W.N_dev + col0];
            rr1[u][hh] = W.ratios[(size_t)g * W.N_dev + col1];
            if (GEN && W.zeros)
                rz[u][hh] = (uint32_t)W.zeros[(size_t)g * W.N_dev + col0] |
                            ((uint32_t)W.zeros[(size_t)g * W.N_dev + col1] << 8);
            else
                rz[u][hh] = 0x0808u;
        }
    };

    f32x16 acc[TM][2];
#pragma unroll
    for (int i = 0; i < TM; i++) { acc[i][0] = f32x16{}; acc[i][1] = f32x16{}; }

    u32x4 xr[XSEG];
    load_x(kb_lo, xr);
#pragma unroll
    for (int u = 0; u < PF; u++) load_w(kb_lo + u, u);
    store_x(0, xr);
    ZeroOff zo0 = zero_off((float)(rz[0][0] & 0xFF)), zo1 = zero_off((float)(rz[0][0] >> 8));

    for (int kb0 = kb_lo; kb0 < kb_hi; kb0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; u++) {
            const int kb = kb0 + u;
            if (kb < kb_hi) {                              // block-uniform
                __syncthreads();
                const int buf = (kb - kb_lo) & 1;
                if (kb + 1 < kb_hi) load_x(kb + 1, xr);
                const u32x4 b0 = rb0[u], b1 = rb1[u];
                float r0[NH], r1[NH];
                uint32_t z[NH];
#pragma unroll
                for (int hh = 0; hh < NH; hh++) { r0[hh] = rr0[u][hh]; r1[hh] = rr1[u][hh]; z[hh] = rz[u][hh]; }
                load_w(kb + PF, u);                        // refill the slot
                if (wave_on) {
#pragma unroll
                    for (int s = 0; s < 4; s++) {
                        const int k = kb * BK + s * 16;
                        if ((s == 0 || (GEN && s == 2)) && (k & Gm1) == 0) {
                            const int hh = GEN ? (s >> 1) : 0;
                            if (k > kb_lo * BK) {          // a new group inside the range
                                const float q0 = r0[hh], q1 = r1[hh];
#pragma unroll
                                for (int i = 0; i < TM; i++)
#pragma unroll
                                    for (int e = 0; e < 16; e++) { acc[i][0][e] *= q0; acc[i][1][e] *= q1; }
                            }
                            if (GEN && W.zeros) {
                                zo0 = zero_off((float)(z[hh] & 0xFF));
                                zo1 = zero_off((float)(z[hh] >> 8));
                            }
                        }
                        const f16x8 bf0 = dequant8(b0[s], zo0, dq), bf1 = dequant8(b1[s], zo1, dq);
#pragma unroll
                        for (int i = 0; i < TM; i++) {
                            const f16x8 af = *reinterpret_cast<const f16x8*>(&As[buf][(i * 32 + c) * LDA + s * 16 + h * 8]);
                            acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af, bf0, acc[i][0], 0, 0, 0);
                            acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af, bf1, acc[i][1], 0, 0, 0);
                        }
                    }
                }
                if (kb + 1 < kb_hi) store_x(buf ^ 1, xr);
            }
        }
    }

    // ---- scale of the range's last group
    const int glast = ((kb_hi * BK) - 1) >> W.lgG;
    const float sl0 = (float)__builtin_bit_cast(f16, W.scales[(size_t)glast * W.N_dev + col0]);
    const float sl1 = (float)__builtin_bit_cast(f16, W.scales[(size_t)glast * W.N_dev + col1]);

    auto epilogue = [&](int m, float v0, float v1) {
        if (EPI == EPI_RESID) {
            const size_t o = (size_t)m * W.N;
            ep.out_f32[o + col0] = ep.resid[o + col0] + v0;
            ep.out_f32[o + col1] = ep.resid[o + col1] + v1;
        } else if (EPI == EPI_SWIGLU) {
            const int f = (nt0 / 2) * 32 + c;          // tile pair (2j, 2j+1) = gate block j, up block j
            ep.act_out[(size_t)m * ep.F_pad + f] = act_f16(silu(v0) * v1);
        } else {
            epi_qkv_pair(ep, m, nt0 * 32, c, v0, v1, ep.slot_base + m, 0);
        }
    };

    if (gs.S == 1) {
        if (!wave_on) return;
        // rows of register e: 8*(e/4) + 4*h + (e%4)
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
                if (m < M) epilogue(m, acc[i][0][e] * sl0, acc[i][1][e] * sl1);
            }
        return;
    }

    // ---- split K: store the partial tile; the last block of the tile adds
    // the S partials in range order and runs the epilogue
    float* part = gs.part + (size_t)sp * M * W.N_dev;
    if (wave_on) {
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
                if (m < M) {
                    part[(size_t)m * W.N_dev + col0] = acc[i][0][e] * sl0;
                    part[(size_t)m * W.N_dev + col1] = acc[i][1][e] * sl1;
                }
            }
    }
    __threadfence();                 // the partial is visible at device scope before the count
    __syncthreads();
    if (tid == 0) {
        unsigned* cnt = gs.cnt + rb * gs.ncb + cb;
        const unsigned old = atomicAdd(cnt, 1u);
        last_flag = (old + 1 == (unsigned)gs.S);
        if (last_flag) atomicExch(cnt, 0u);   // ready for the next call
    }
    __syncthreads();
    if (!last_flag) return;
    __threadfence();                 // acquire the other blocks' partials
    if (!wave_on) return;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
            if (m >= M) continue;
            float v0 = 0.f, v1 = 0.f;
            for (int s = 0; s < gs.S; s++) {
                const float* ps = gs.part + ((size_t)s * M + m) * W.N_dev;
                v0 += s == sp ? acc[i][0][e] * sl0 : ps[col0];
                v1 += s == sp ? acc[i][1][e] * sl1 : ps[col1];
            }
            epilogue(m, v0, v1);
        }
}

template <int EPI, int TM>
int launch_tm(const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmShape& gs, hipStream_t stream) {
    const int blocks = gs.nrb * gs.ncb * gs.S;
    if (W.zeros || W.lgG < 6)
        hipLaunchKernelGGL((gemm_w4_kernel<EPI, TM, true>), dim3(blocks), dim3(256), 0, stream, X, ldx, W, ep, gs);
    else
        hipLaunchKernelGGL((gemm_w4_kernel<EPI, TM, false>), dim3(blocks), dim3(256), 0, stream, X, ldx, W, ep, gs);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <int EPI>
int launch_epi(int TM, const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmShape& gs,
               hipStream_t stream) {
    if (TM == 4) return launch_tm<EPI, 4>(X, ldx, W, ep, gs, stream);
    if (TM == 2) return launch_tm<EPI, 2>(X, ldx, W, ep, gs, stream);
    return launch_tm<EPI, 1>(X, ldx, W, ep, gs, stream);
}

}  // namespace

GemmPlan gemm_w4_plan(int M, const DevLinear& W, int num_cus) {
    GemmPlan p;
    const int ncb = (W.N_dev + BN - 1) / BN, KB = W.K_pad / 64;
    p.TM = 4;
    // smaller row tiles, then k splits, until the grid covers the CUs
    while (p.TM > 1 && ((M + 32 * p.TM - 1) / (32 * p.TM)) * ncb < num_cus) p.TM /= 2;
    const int nrb = (M + 32 * p.TM - 1) / (32 * p.TM);
    p.S = 1;
    while (nrb * ncb * p.S < num_cus && KB / (p.S * 2) >= 8 && p.S < 8) p.S *= 2;
    p.nrb = nrb;
    p.ncb = ncb;
    p.part_bytes = p.S > 1 ? (size_t)p.S * M * W.N_dev * 4 : 0;
    p.tiles = nrb * ncb;
    return p;
}

int launch_gemm_w4(int epi, const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmPlan& p,
                   int M, float* part, unsigned* cnt, hipStream_t stream) {
    if (p.S > 1 && (!part || !cnt)) return -1;
    GemmShape gs{M, p.nrb, p.ncb, p.S, W.K_pad / 64, part, cnt};
    switch (epi) {
        case EPI_QKV: return launch_epi<EPI_QKV>(p.TM, X, ldx, W, ep, gs, stream);
        case EPI_RESID: return launch_epi<EPI_RESID>(p.TM, X, ldx, W, ep, gs, stream);
        case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(p.TM, X, ldx, W, ep, gs, stream);
        default: return -1;
    }
}
