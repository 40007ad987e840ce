// Grouped-query causal attention (top.FAttention, Sec. 2.2) for the three
// stages.
//
// Prefill / prefill_kv: flash attention on the 32x32x16 bf16 MFMA.  A wave
// owns 32 queries of one head; the waves of a block share the kv head (and
// the K/V tiles staged in LDS).  Scores are formed transposed, S^T = K Q^T,
// with the 32 key rows of a tile fed in a permuted order (bits 2 and 3 of the
// row index swapped) so that register e of the score tile holds key
// 16*(e/8) + 8*(lane/32) + e%8 of query lane%32: exactly the operand layout
// of P^T in O^T = V^T P^T.  Every lane therefore owns one query: the online
// softmax (running max and sum) lives in registers.  P is fed to the MFMA as
// a bf16 pair hi + lo (P - hi), which keeps P V at near-fp32 accuracy; V is
// stored transposed in LDS.  The causal mask is computed from indices, only
// on the tiles that straddle the diagonal; tiles past it are skipped (the
// role the paper's small reusable mask plays, Sec. 4.6.1).
//
// Decode: one query per sequence.  Split-KV: a block reads one chunk of one
// kv head's cache once for all the query heads of its group (VALU dot
// products, v_dot2 on bf16 pairs), writes a partial (max, sum, unnormalised
// output), and a combine kernel merges the chunks with the log-sum-exp rule.
#include "common.h"
#include "launch.h"

namespace {

__device__ __forceinline__ int key_perm(int r) {  // swap bits 2 and 3
    return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int D>
__global__ void __launch_bounds__(256) attn_prefill_kernel(AttnPrefillArgs a, int HB, int QB) {
    constexpr int LDK = D + 8;   // bf16 per K row in LDS
    constexpr int LDV = 32 + 8;  // bf16 per V^T row in LDS
    __shared__ __attribute__((aligned(16))) __bf16 Ks[32 * LDK];
    __shared__ __attribute__((aligned(16))) __bf16 Vt[D * LDV];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, c = lane & 31;
    const int r = a.nq / a.nkv;
    const int ngrp = (r + HB - 1) / HB;
    const int g = blockIdx.y / ngrp, hg = blockIdx.y % ngrp;
    const int hw = wave % HB, qt = wave / HB;
    const int hidx = hg * HB + hw;
    const bool active = (wave < HB * QB) && (hidx < r);
    const int head = g * r + hidx;
    const int q0 = (blockIdx.x * QB + qt) * 32;
    const int qb_end = min(a.T, (blockIdx.x + 1) * QB * 32);
    const int nkeys = a.L + qb_end;              // keys the block may need
    const int ntile = (nkeys + 31) / 32;
    const uint16_t* kc = a.k_cache + (size_t)g * a.cache_stride_h;
    const uint16_t* vc = a.v_cache + (size_t)g * a.cache_stride_h;

    // Q^T fragments (B operand): query q0 + c, dims 16s + 8h .. +8
    bf16x8 qf[D / 16];
    const int qrow = q0 + c;
#pragma unroll
    for (int s = 0; s < D / 16; s++) {
        if (active && qrow < a.T)
            qf[s] = *reinterpret_cast<const bf16x8*>(a.q + ((size_t)qrow * a.nq + head) * D + s * 16 + h * 8);
        else
            qf[s] = bf16x8{};
    }
    f32x16 o[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; i++) o[i] = f32x16{};
    float m = -INFINITY, l = 0.f;
    const int qslot = a.L + qrow;
    const int wave_last_slot = a.L + min(q0 + 31, a.T - 1);

    for (int kt = 0; kt < ntile; kt++) {
        __syncthreads();
        // K tile rows and V^T columns: 32 keys x D dims, 16 bytes per load
        for (int i = tid; i < 32 * (D / 8); i += 256) {
            const int key = i / (D / 8), seg = i % (D / 8);
            const int slot = kt * 32 + key;
            u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
            if (slot < nkeys) {
                kv = *reinterpret_cast<const u32x4*>(kc + (size_t)slot * D + seg * 8);
                vv = *reinterpret_cast<const u32x4*>(vc + (size_t)slot * D + seg * 8);
            }
            *reinterpret_cast<u32x4*>(&Ks[key * LDK + seg * 8]) = kv;
            const __bf16* ve = reinterpret_cast<const __bf16*>(&vv);
#pragma unroll
            for (int j = 0; j < 8; j++) Vt[(seg * 8 + j) * LDV + key] = ve[j];
        }
        __syncthreads();
        if (!active || q0 >= a.T || kt * 32 > wave_last_slot) continue;

        // S^T = K Q^T (rows: permuted keys, columns: queries)
        f32x16 s_acc = f32x16{};
        const int krow = key_perm(c);
#pragma unroll
        for (int s = 0; s < D / 16; s++) {
            const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[krow * LDK + s * 16 + h * 8]);
            s_acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], s_acc, 0, 0, 0);
        }
        float p[16];
        float mt = -INFINITY;
        const bool diag = (kt * 32 + 31 > a.L + q0);
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int kslot = kt * 32 + 16 * (e / 8) + 8 * h + (e % 8);
            float v = s_acc[e] * a.scale_log2;
            if (diag && kslot > qslot) v = -INFINITY;
            p[e] = v;
            mt = fmaxf(mt, v);
        }
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float m_new = fmaxf(m, mt);
        const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m - m_new);
        float ls = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            p[e] = (p[e] == -INFINITY) ? 0.f : exp2f(p[e] - m_new);
            ls += p[e];
        }
        l = l * alpha + ls;
        m = m_new;
#pragma unroll
        for (int i = 0; i < D / 32; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) o[i][e] *= alpha;

        bf16x8 phi[2], plo[2];
#pragma unroll
        for (int s = 0; s < 2; s++)
#pragma unroll
            for (int j = 0; j < 8; j++) {
                const float pv = p[8 * s + j];
                const __bf16 hi = (__bf16)pv;
                phi[s][j] = hi;
                plo[s][j] = (__bf16)(pv - (float)hi);
            }
#pragma unroll
        for (int i = 0; i < D / 32; i++) {
#pragma unroll
            for (int s = 0; s < 2; s++) {
                const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vt[(i * 32 + c) * LDV + s * 16 + h * 8]);
                o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, phi[s], o[i], 0, 0, 0);
                o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, plo[s], o[i], 0, 0, 0);
            }
        }
    }
    if (!active || qrow >= a.T) return;
    const float lt = l + __shfl_xor(l, 32, 64);
    const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
    f16* out = a.out + ((size_t)qrow * a.nq + head) * D;
#pragma unroll
    for (int i = 0; i < D / 32; i++)
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int dim = i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
            out[dim] = act_f16(o[i][e] * inv);
        }
}

// ---------------------------------------------------------------- decode

constexpr int MAXR = 8;      // query heads per kv head
constexpr int DEC_MAXCH = 512;

template <int D>
__global__ void __launch_bounds__(256) attn_decode_split_kernel(AttnDecodeArgs a) {
    constexpr int LPK = D / 8;        // lanes per key
    constexpr int KPW = 64 / LPK;     // keys per wave load
    __shared__ float sc[MAXR][DEC_MAXCH];
    __shared__ float ored[4][MAXR][D];
    __shared__ float stat[MAXR][2];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x / a.nkv, g = blockIdx.x % a.nkv;
    const int chunk = blockIdx.y;
    const int ctx = a.ctx_lens[b];
    const int start = chunk * a.chunk;
    const int end = min(start + a.chunk, ctx + 1);
    if (start >= end) return;
    const int r = a.nq / a.nkv;
    const int kl = lane / LPK, dseg = lane % LPK;
    const uint16_t* kc = a.k_cache + (size_t)b * a.stride_b + (size_t)g * a.stride_h;
    const uint16_t* vc = a.v_cache + (size_t)b * a.stride_b + (size_t)g * a.stride_h;

    // q of the group's heads: dims 8*dseg .. +8, as bf16 pairs
    uint32_t qv[MAXR][4];
#pragma unroll
    for (int i = 0; i < MAXR; i++) {
        u32x4 t = {0, 0, 0, 0};
        if (i < r) t = *reinterpret_cast<const u32x4*>(a.q + ((size_t)b * a.nq + g * r + i) * D + dseg * 8);
        qv[i][0] = t[0]; qv[i][1] = t[1]; qv[i][2] = t[2]; qv[i][3] = t[3];
    }
    const float* mrow = a.mask ? a.mask + (size_t)b * a.max_seq : nullptr;
    const float LOG2E = 1.4426950408889634f;

    // scores
    for (int k0 = start + wave * KPW; k0 < end; k0 += 4 * KPW) {
        const int key = k0 + kl;
        const bool valid = key < end;
        u32x4 kk = {0, 0, 0, 0};
        if (valid) kk = *reinterpret_cast<const u32x4*>(kc + (size_t)key * D + dseg * 8);
        const uint32_t kw[4] = {kk[0], kk[1], kk[2], kk[3]};
#pragma unroll
        for (int i = 0; i < MAXR; i++) {
            if (i >= r) break;
            float v = 0.f;
#pragma unroll
            for (int p = 0; p < 4; p++)
                v = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(qv[i][p]), as_bf16x2(kw[p]), v, false);
#pragma unroll
            for (int o = 1; o < LPK; o <<= 1) v += __shfl_xor(v, o, 64);
            if (dseg == 0 && valid) {
                float s = v * a.scale_log2;
                if (mrow) s += mrow[key] * LOG2E;
                sc[i][key - start] = s;
            }
        }
    }
    __syncthreads();
    // softmax statistics of the chunk (one wave per head)
    const int n = end - start;
    for (int i = wave; i < r; i += 4) {
        float mx = -INFINITY;
        for (int j = lane; j < n; j += 64) mx = fmaxf(mx, sc[i][j]);
        mx = wave_max(mx);
        float sum = 0.f;
        for (int j = lane; j < n; j += 64) {
            const float pv = (mx == -INFINITY) ? 0.f : exp2f(sc[i][j] - mx);
            sc[i][j] = pv;
            sum += pv;
        }
        sum = wave_sum(sum);
        if (lane == 0) { stat[i][0] = mx; stat[i][1] = sum; }
    }
    __syncthreads();
    // P V
    float ov[MAXR][8];
#pragma unroll
    for (int i = 0; i < MAXR; i++)
#pragma unroll
        for (int j = 0; j < 8; j++) ov[i][j] = 0.f;
    for (int k0 = start + wave * KPW; k0 < end; k0 += 4 * KPW) {
        const int key = k0 + kl;
        if (key >= end) continue;
        const u32x4 vv = *reinterpret_cast<const u32x4*>(vc + (size_t)key * D + dseg * 8);
        const uint32_t vw[4] = {vv[0], vv[1], vv[2], vv[3]};
        float vf[8];
#pragma unroll
        for (int p = 0; p < 4; p++) {
            vf[2 * p] = __uint_as_float(vw[p] << 16);
            vf[2 * p + 1] = __uint_as_float(vw[p] & 0xFFFF0000u);
        }
#pragma unroll
        for (int i = 0; i < MAXR; i++) {
            if (i >= r) break;
            const float pv = sc[i][key - start];
#pragma unroll
            for (int j = 0; j < 8; j++) ov[i][j] += pv * vf[j];
        }
    }
    // reduce over the keys of the wave (lanes with equal dseg), then waves
#pragma unroll
    for (int i = 0; i < MAXR; i++) {
        if (i >= r) break;
#pragma unroll
        for (int j = 0; j < 8; j++) {
            float v = ov[i][j];
#pragma unroll
            for (int o = LPK; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
            ov[i][j] = v;
        }
        if (kl == 0)
#pragma unroll
            for (int j = 0; j < 8; j++) ored[wave][i][dseg * 8 + j] = ov[i][j];
    }
    __syncthreads();
    for (int idx = tid; idx < r * D; idx += 256) {
        const int i = idx / D, dim = idx % D;
        const float v = ored[0][i][dim] + ored[1][i][dim] + ored[2][i][dim] + ored[3][i][dim];
        float* pp = a.part + (((size_t)b * a.nq + g * r + i) * a.nchunks + chunk) * (D + 2);
        pp[dim] = v;
        if (dim == 0) { pp[D] = stat[i][0]; pp[D + 1] = stat[i][1]; }
    }
}

template <int D>
__global__ void __launch_bounds__(D) attn_decode_combine_kernel(AttnDecodeArgs a) {
    const int b = blockIdx.x / a.nq, head = blockIdx.x % a.nq;
    const int dim = threadIdx.x;
    const int ctx = a.ctx_lens[b];
    const int nch = (ctx + 1 + a.chunk - 1) / a.chunk;
    const float* pp = a.part + ((size_t)b * a.nq + head) * a.nchunks * (D + 2);
    float M = -INFINITY;
    for (int ch = 0; ch < nch; ch++) M = fmaxf(M, pp[ch * (D + 2) + D]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
        for (int ch = 0; ch < nch; ch++) {
            const float mc = pp[ch * (D + 2) + D];
            if (mc == -INFINITY) continue;
            const float w = exp2f(mc - M);
            L += w * pp[ch * (D + 2) + D + 1];
            O += w * pp[ch * (D + 2) + dim];
        }
    }
    const float v = (L > 0.f) ? O / L : 0.f;
    a.out[((size_t)b * a.nq + head) * D + dim] = act_f16(v);
}

}  // namespace

int launch_attn_prefill(const AttnPrefillArgs& a, hipStream_t stream) {
    const int r = a.nq / a.nkv;
    int HB = r < 4 ? r : 4;
    int QB = (4 % HB == 0) ? 4 / HB : 1;
    const int ngrp = (r + HB - 1) / HB;
    dim3 grid((a.T + 32 * QB - 1) / (32 * QB), a.nkv * ngrp);
    if (a.d == 128)
        hipLaunchKernelGGL(attn_prefill_kernel<128>, grid, dim3(256), 0, stream, a, HB, QB);
    else if (a.d == 64)
        hipLaunchKernelGGL(attn_prefill_kernel<64>, grid, dim3(256), 0, stream, a, HB, QB);
    else
        return -1;
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_attn_decode(const AttnDecodeArgs& a, hipStream_t stream) {
    if (a.chunk > DEC_MAXCH || a.nq / a.nkv > MAXR) return -1;
    dim3 g1(a.B * a.nkv, a.nchunks), g2(a.B * a.nq);
    if (a.d == 128) {
        hipLaunchKernelGGL(attn_decode_split_kernel<128>, g1, dim3(256), 0, stream, a);
        hipLaunchKernelGGL(attn_decode_combine_kernel<128>, g2, dim3(128), 0, stream, a);
    } else if (a.d == 64) {
        hipLaunchKernelGGL(attn_decode_split_kernel<64>, g1, dim3(256), 0, stream, a);
        hipLaunchKernelGGL(attn_decode_combine_kernel<64>, g2, dim3(64), 0, stream, a);
    } else {
        return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
