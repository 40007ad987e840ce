// Grouped-query causal attention (top.FAttention, Sec. 2.2) for the three
// stages.
//
// Prefill / prefill_kv: flash attention on the 32x32x16 bf16 MFMA.  A block
// works on one kv head, one tile of 32 queries and one chunk of the keys
// those queries see; its waves are the query heads of the kv head's group
// (one head per wave), so every K/V tile staged in LDS serves all of them.
// Chunks split long key ranges across blocks (a causal prefill's late query
// tiles, a prefill_kv over a long history), so the grid has enough blocks;
// work items are ordered longest first.
//
// Keys are staged 64 at a time (two 32-key tiles), K and V both straight
// from memory to LDS (direct-to-LDS loads), double buffered: one memory round
// trip per 64 keys, one barrier.  K rows are 16-byte-chunk XOR-swizzled by
// row (conflict-free fragment reads); V stays in its natural [key][dim]
// layout and the V^T fragments of O^T = V^T P^T are gathered with 16-bit LDS
// reads.  Scores are formed transposed, S^T = K Q^T, with the 32 key rows
// of a tile fed in a permuted order (bits 2 and 3 of the row index swapped)
// so that register e of the score tile holds key 16*(e/8) + 8*(lane/32) +
// e%8 of query lane%32: exactly the operand layout of P^T.  Every lane
// therefore owns one query: the online softmax (running max and sum) lives
// in registers and is updated once per 64 keys.  P is fed to the MFMA as a
// bf16 pair hi + lo (P - hi), which keeps P V at near-fp32 accuracy.  The
// causal mask is computed from indices, only on tiles that straddle the
// diagonal; tiles past it are never visited (the role the paper's small
// reusable mask plays, Sec. 4.6.1).
//
// A query tile whose keys fit one chunk writes its output directly.
// Otherwise every chunk writes its partial state (running max, sum and
// unnormalised output, in the accumulator layout: coalesced) and a second
// kernel merges the chunks of each query tile in chunk order with the
// log-sum-exp rule, so results do not depend on timing.
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

constexpr int PF_MAXHB = 8;                  // query heads per block
constexpr int PF_KST = 64;                   // keys per LDS stage

// Query tile and key chunk of work item `item` (longest first): query tile
// qt has nkeys(qt) = L + min(T, 32 (qt + 1)) keys, cut into chunks of
// chunk_keys.  `first` is the item of the tile's chunk 0.
__device__ __forceinline__ void prefill_item(const AttnPrefillArgs& a, int item, int& qt, int& chunk, int& nch,
                                             int& first) {
    const int nqt = (a.T + 31) / 32;
    int base = 0;
    for (qt = nqt - 1; qt > 0; qt--) {
        const int nk = a.L + min(a.T, 32 * (qt + 1));
        const int n = (nk + a.chunk_keys - 1) / a.chunk_keys;
        if (item < base + n) break;
        base += n;
    }
    const int nk = a.L + min(a.T, 32 * (qt + 1));
    nch = (nk + a.chunk_keys - 1) / a.chunk_keys;
    chunk = item - base;
    first = base;
}

template <int D>
__device__ __forceinline__ size_t part_index(const AttnPrefillArgs& a, int row, int item, int wave, int lane) {
    constexpr int NREG = 2 + 16 * (D / 32);
    return ((size_t)(row * a.items + item) * PF_MAXHB + wave) * NREG * 64 + lane;
}

template <int D>
__global__ void __launch_bounds__(64 * PF_MAXHB) attn_prefill_kernel(AttnPrefillArgs a) {
    constexpr int NCH = D / 8;               // 16-byte chunks per K / V row
    constexpr int STB = PF_KST * D * 2;      // bytes of one K or V stage
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    unsigned char* const Ks = smem;              // [2][64 keys][D], chunks swizzled
    unsigned char* const Vs = smem + 2 * STB;    // [2][64 keys][D]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int HB = blockDim.x / 64;
    const int h = lane >> 5, c = lane & 31;
    const int r = a.nq / a.nkv;
    const int g = blockIdx.y / a.ngrp, hg = blockIdx.y % a.ngrp;
    const int hidx = hg * HB + wave;
    const bool active = hidx < r;
    const int head = g * r + (active ? hidx : 0);
    int qt, chunk, nch, first;
    prefill_item(a, blockIdx.x, qt, chunk, nch, first);
    const int q0 = qt * 32;
    const int nkeys = a.L + min(a.T, q0 + 32);
    const int k0 = chunk * a.chunk_keys, k1 = min(nkeys, k0 + a.chunk_keys);
    const int nst = (k1 - k0 + PF_KST - 1) / PF_KST;
    const uint16_t* kc = a.k_cache + (size_t)g * a.cache_stride_h;
    const uint16_t* vc = a.v_cache + (size_t)g * a.cache_stride_h;

    // ---- stage of 64 keys: 2 x 64 loads of 1 KB (K, V); load i fills rows
    // KROWS i .. + KROWS - 1; lane l writes chunk l % NCH of its row (for K
    // holding logical chunk (l % NCH) ^ (row % NCH))
    constexpr int KROWS = 1024 / (2 * D);
    constexpr int NLOAD = PF_KST / KROWS;
    auto load_stage = [&](int st, int buf) __attribute__((always_inline)) {
        for (int i = wave; i < NLOAD; i += HB) {
            const int row = i * KROWS + lane / NCH;
            int slot = k0 + st * PF_KST + row;
            slot = slot < k1 ? slot : k1 - 1;
            const int pc = lane % NCH, lc = pc ^ (row % NCH);
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(kc + (size_t)slot * D + lc * 8),
                                             (__attribute__((address_space(3))) void*)(Ks + buf * STB + i * 1024),
                                             16, 0, 0);
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(vc + (size_t)slot * D + pc * 8),
                                             (__attribute__((address_space(3))) void*)(Vs + buf * STB + i * 1024),
                                             16, 0, 0);
        }
    };

    // Q^T fragments (B operand): query q0 + c, dims 16s + 8h .. +8
    bf16x8 qf[D / 16];
    const int qrow = q0 + c;
    const int qload = qrow < a.T ? qrow : a.T - 1;
    load_stage(0, 0);
#pragma unroll
    for (int s = 0; s < D / 16; s++)
        qf[s] = *reinterpret_cast<const bf16x8*>(a.q + ((size_t)qload * a.nq + head) * D + s * 16 + h * 8);

    f32x16 o[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; i++) o[i] = f32x16{};
    float m = -INFINITY, l = 0.f;
    const int qslot = a.L + qrow;
    const int krow = key_perm(c);
    __syncthreads();
    for (int st = 0; st < nst; st++) {
        const int buf = st & 1;
        if (st + 1 < nst) load_stage(st + 1, buf ^ 1);
        if (active) {
            const unsigned char* K = Ks + buf * STB;
            const __bf16* V = reinterpret_cast<const __bf16*>(Vs + buf * STB);
            // S^T of the two 32-key tiles, two independent MFMA chains
            f32x16 sa = f32x16{}, sb = f32x16{};
#pragma unroll
            for (int s = 0; s < D / 16; s++) {
                const int lc = (2 * s + h) ^ (krow % NCH);
                const bf16x8 ka = *reinterpret_cast<const bf16x8*>(K + krow * (2 * D) + lc * 16);
                const bf16x8 kb = *reinterpret_cast<const bf16x8*>(K + (32 + krow) * (2 * D) + lc * 16);
                sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[s], sa, 0, 0, 0);
                sb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qf[s], sb, 0, 0, 0);
            }
            const int kbase = k0 + st * PF_KST;
            const bool diag = kbase + PF_KST - 1 > a.L + q0;
            float p[32];
            float mt = -INFINITY;
#pragma unroll
            for (int e = 0; e < 32; e++) {
                const int kslot = kbase + 32 * (e / 16) + 16 * ((e % 16) / 8) + 8 * h + (e % 8);
                float v = (e < 16 ? sa[e] : sb[e - 16]) * a.scale_log2;
                if (diag && kslot > qslot) v = -INFINITY;
                p[e] = v;
                mt = fmaxf(mt, v);
            }
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float m_new = fmaxf(m, mt);
            const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m - m_new);
            float ls = 0.f;
#pragma unroll
            for (int e = 0; e < 32; e++) {
                p[e] = (p[e] == -INFINITY) ? 0.f : exp2f(p[e] - m_new);
                ls += p[e];
            }
            l = l * alpha + ls;
            m = m_new;
#pragma unroll
            for (int i = 0; i < D / 32; i++)
#pragma unroll
                for (int e = 0; e < 16; e++) o[i][e] *= alpha;
            // O^T += V^T P^T over the 4 key groups of 16 (tile, step)
#pragma unroll
            for (int ks = 0; ks < 4; ks++) {
                bf16x8 phi, plo;
#pragma unroll
                for (int j = 0; j < 8; j++) {
                    const float pv = p[8 * ks + j];
                    const __bf16 hi = (__bf16)pv;
                    phi[j] = hi;
                    plo[j] = (__bf16)(pv - (float)hi);
                }
                const int key0 = 16 * ks + 8 * h;       // this lane's 8 keys of the group
#pragma unroll
                for (int i = 0; i < D / 32; i++) {
                    bf16x8 vf;
#pragma unroll
                    for (int j = 0; j < 8; j++) vf[j] = V[(key0 + j) * D + i * 32 + c];
                    o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, phi, o[i], 0, 0, 0);
                    o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, plo, o[i], 0, 0, 0);
                }
            }
        }
        __syncthreads();
    }
    if (!active) return;

    if (nch == 1) {
        // output: dim of register e of o[i] is i * 32 + 8 (e / 4) + 4 h + e % 4
        if (qrow >= a.T) return;
        const float lt = l + __shfl_xor(l, 32, 64);
        const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
        f16* out = a.out + ((size_t)qrow * a.nq + head) * D;
#pragma unroll
        for (int i = 0; i < D / 32; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) out[i * 32 + 8 * (e / 4) + 4 * h + (e % 4)] = act_f16(o[i][e] * inv);
        return;
    }
    // partial state of this chunk: [row][item][wave][m, l, O registers][64 lanes]
    float* pp = a.part + part_index<D>(a, blockIdx.y, blockIdx.x, wave, lane);
    pp[0] = m;
    pp[64] = l;
#pragma unroll
    for (int i = 0; i < D / 32; i++)
#pragma unroll
        for (int e = 0; e < 16; e++) pp[(size_t)(2 + i * 16 + e) * 64] = o[i][e];
}

// Merge of the chunk states of the query tiles with more than one chunk:
// block (query tile, block row, 32-dim slice): thread (wave, lane) merges the
// lane's 16 output registers of the slice over the tile's chunks, in order.
template <int D>
__global__ void __launch_bounds__(64 * PF_MAXHB) attn_prefill_merge_kernel(AttnPrefillArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int HB = blockDim.x / 64;
    const int h = lane >> 5, c = lane & 31;
    const int qt = blockIdx.x, row = blockIdx.y, i = blockIdx.z;
    const int r = a.nq / a.nkv;
    const int g = row / a.ngrp, hidx = (row % a.ngrp) * HB + wave;
    const int nqt = (a.T + 31) / 32;
    // first item of tile qt (items run from the last tile down)
    int first = 0;
    for (int t = nqt - 1; t > qt; t--) first += (a.L + min(a.T, 32 * (t + 1)) + a.chunk_keys - 1) / a.chunk_keys;
    const int nch = (a.L + min(a.T, 32 * (qt + 1)) + a.chunk_keys - 1) / a.chunk_keys;
    if (nch == 1 || hidx >= r) return;
    // chunks in groups of CB: the states of a group are requested together,
    // then merged into the running maximum M, sum L and output acc
    constexpr int CB = 4;
    float M = -INFINITY, L = 0.f, acc[16] = {};
    for (int ch0 = 0; ch0 < nch; ch0 += CB) {
        float mc[CB], lc[CB], v[CB][16];
#pragma unroll
        for (int j = 0; j < CB; j++) {
            const int ch = ch0 + j < nch ? ch0 + j : nch - 1;
            const float* pp = a.part + part_index<D>(a, row, first + ch, wave, lane);
            mc[j] = pp[0];
            lc[j] = pp[64];
#pragma unroll
            for (int e = 0; e < 16; e++) v[j][e] = pp[(size_t)(2 + i * 16 + e) * 64];
        }
        float Mn = M;
#pragma unroll
        for (int j = 0; j < CB; j++)
            if (ch0 + j < nch) Mn = fmaxf(Mn, mc[j]);
        if (Mn == -INFINITY) continue;
        const float sc = (M == -INFINITY) ? 0.f : exp2f(M - Mn);
        L *= sc;
#pragma unroll
        for (int e = 0; e < 16; e++) acc[e] *= sc;
#pragma unroll
        for (int j = 0; j < CB; j++) {
            if (ch0 + j >= nch || mc[j] == -INFINITY) continue;
            const float w = exp2f(mc[j] - Mn);
            L += w * lc[j];
#pragma unroll
            for (int e = 0; e < 16; e++) acc[e] += w * v[j][e];
        }
        M = Mn;
    }
    const int qrow = qt * 32 + c;
    const float lt = L + __shfl_xor(L, 32, 64);
    if (qrow >= a.T) return;
    const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
    f16* out = a.out + ((size_t)qrow * a.nq + g * r + hidx) * D;
#pragma unroll
    for (int e = 0; e < 16; e++) out[i * 32 + 8 * (e / 4) + 4 * h + (e % 4)] = act_f16(acc[e] * inv);
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

AttnPrefillPlan attn_prefill_plan(int T, int L, int nq, int nkv, int d, int num_cus) {
    AttnPrefillPlan p;
    const int r = nq / nkv;
    const int hb = r < PF_MAXHB ? r : PF_MAXHB;
    p.ngrp = (r + hb - 1) / hb;
    p.threads = 64 * hb;
    const int nqt = (T + 31) / 32;
    // key stages of all query tiles of one block row, then chunks of at
    // least 2 stages (128 keys) sized so that the grid holds about two
    // blocks per CU
    long long stages = 0;
    for (int qt = 0; qt < nqt; qt++) stages += (L + std::min(T, 32 * (qt + 1)) + PF_KST - 1) / PF_KST;
    const long long rows = (long long)nkv * p.ngrp;
    long long cs = (stages * rows + 2LL * num_cus - 1) / (2LL * num_cus);
    cs = std::max(2LL, cs);
    p.chunk_keys = (int)(PF_KST * cs);
    p.items = 0;
    bool multi = false;
    for (int qt = 0; qt < nqt; qt++) {
        const int n = (L + std::min(T, 32 * (qt + 1)) + p.chunk_keys - 1) / p.chunk_keys;
        p.items += n;
        multi |= n > 1;
    }
    p.merge = multi;
    const int nreg = 2 + 16 * (d / 32);
    const size_t per_item = (size_t)rows * PF_MAXHB * nreg * 64 * sizeof(float);
    p.part_bytes = multi ? (size_t)p.items * per_item : 0;
    // chunks are at least 128 keys: a bound that grows with L, for workspace sizing
    p.part_bound = (size_t)nqt * ((L + T + 127) / 128) * per_item;
    p.lds_bytes = (size_t)4 * PF_KST * d * 2;
    return p;
}

int launch_attn_prefill(const AttnPrefillArgs& a, const AttnPrefillPlan& p, hipStream_t stream) {
    if (p.items < 1 || (p.part_bytes && !a.part)) return -1;
    AttnPrefillArgs b = a;
    b.chunk_keys = p.chunk_keys;
    b.ngrp = p.ngrp;
    b.items = p.items;
    const dim3 grid(p.items, a.nkv * p.ngrp);
    const dim3 mgrid((a.T + 31) / 32, a.nkv * p.ngrp, a.d / 32);
    static LdsLimit lim128, lim64;
    if (a.d == 128) {
        if (ensure_lds_limit(lim128, (const void*)attn_prefill_kernel<128>, p.lds_bytes)) return -1;
        hipLaunchKernelGGL(attn_prefill_kernel<128>, grid, dim3(p.threads), p.lds_bytes, stream, b);
        if (p.merge) hipLaunchKernelGGL(attn_prefill_merge_kernel<128>, mgrid, dim3(p.threads), 0, stream, b);
    } else if (a.d == 64) {
        if (ensure_lds_limit(lim64, (const void*)attn_prefill_kernel<64>, p.lds_bytes)) return -1;
        hipLaunchKernelGGL(attn_prefill_kernel<64>, grid, dim3(p.threads), p.lds_bytes, stream, b);
        if (p.merge) hipLaunchKernelGGL(attn_prefill_merge_kernel<64>, mgrid, dim3(p.threads), 0, stream, b);
    } else {
        return -1;
    }
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
