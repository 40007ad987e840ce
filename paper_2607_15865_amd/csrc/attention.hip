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
// layout and the V^T fragments of O^T = V^T P^T come from it by transposing
// LDS reads (lds_read_tr16).  Scores are formed transposed, S^T = K Q^T, with the 32 key rows
// of a tile fed in a permuted order (bits 2 and 3 of the row index swapped)
// so that register e of the score tile holds key 16*(e/8) + 8*(lane/32) +
// e%8 of query lane%32: exactly the operand layout of P^T.  Every lane
// therefore owns one query: the online softmax (running max and sum) lives
// in registers; the max moves only when a score passes it by more than 8
// (log2 units), so the weights stay below 2^8.  P is fed to the MFMA as a
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
// Decode: one query per sequence.  Split-KV: a block stages one 64-key chunk
// of one kv head's cache in LDS once for all the query heads of its group,
// forms scores and P V on the 16x16x32 bf16 MFMA, writes a partial (max,
// sum, unnormalised output), and a combine kernel merges the chunks with the
// log-sum-exp rule.
#include "common.h"
#include "launch.h"

namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));

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
#pragma unroll
            for (int e = 0; e < 32; e++) p[e] = (e < 16 ? sa[e] : sb[e - 16]) * a.scale_log2;
            if (diag) {            // (only the stages that straddle the diagonal)
#pragma unroll
                for (int e = 0; e < 32; e++) {
                    const int kslot = kbase + 32 * (e / 16) + 16 * ((e % 16) / 8) + 8 * h + (e % 8);
                    if (kslot > qslot) p[e] = -INFINITY;
                }
            }
            float mt = -INFINITY;
#pragma unroll
            for (int e = 0; e < 32; e++) mt = fmaxf(mt, p[e]);
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float m_new = fmaxf(m, mt);
            // The running max m moves (and o, l are rescaled) only when some
            // lane's scores pass it by more than 8 (log2 units); until then the
            // weights are taken against the older m and stay below 2^8, which
            // the hi + lo split of P carries as well as weights below 1.  While
            // every key so far is masked, m is -inf and the weights are 0.
            if (__builtin_amdgcn_ballot_w64(m_new > m + 8.0f) != 0) {
                const float alpha = exp2_hw(m - (m_new == -INFINITY ? 0.f : m_new));
                l *= alpha;
#pragma unroll
                for (int i = 0; i < D / 32; i++)
#pragma unroll
                    for (int e = 0; e < 16; e++) o[i][e] *= alpha;
                m = m_new;
            }
            const float mb = m == -INFINITY ? 0.f : m;
            float ls = 0.f;
#pragma unroll
            for (int e = 0; e < 32; e++) {
                p[e] = exp2_hw(p[e] - mb);
                ls += p[e];
            }
            l += ls;
            // O^T += V^T P^T over the 4 key groups of 16 (tile, step)
#pragma unroll
            for (int ks = 0; ks < 4; ks++) {
                bf16x8 phi, plo;
#pragma unroll
                for (int j = 0; j < 8; j += 2) {          // pairs: one packed conversion each
                    const bf16x2 hi = __builtin_convertvector(f32x2{p[8 * ks + j], p[8 * ks + j + 1]}, bf16x2);
                    const bf16x2 lo = __builtin_convertvector(
                        f32x2{p[8 * ks + j] - (float)hi[0], p[8 * ks + j + 1] - (float)hi[1]}, bf16x2);
                    phi[j] = hi[0]; phi[j + 1] = hi[1];
                    plo[j] = lo[0]; plo[j + 1] = lo[1];
                }
                // this lane's 8 keys 16 ks + 8 h .. + 7, dim i * 32 + c, by two
                // transposing reads: lane s of its 16-lane group points at key
                // 16 ks + 8 h + s / 4 (+ 4), dims 16 (c / 16) + 4 (s % 4) .. + 3
                const __bf16* vrow = V + (16 * ks + 8 * h + ((lane & 15) >> 2)) * D + 16 * (c >> 4) + 4 * (lane & 3);
#pragma unroll
                for (int i = 0; i < D / 32; i++) {
                    const i16x4 v0 = lds_read_tr16(vrow + i * 32), v1 = lds_read_tr16(vrow + 4 * D + i * 32);
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
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
        bool bad = false;
#pragma unroll
        for (int i = 0; i < D / 32; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) out[i * 32 + 8 * (e / 4) + 4 * h + (e % 4)] = act_f16(o[i][e] * inv, bad);
        flag_range(a.err, bad);
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
    bool bad = false;
#pragma unroll
    for (int e = 0; e < 16; e++) out[i * 32 + 8 * (e / 4) + 4 * h + (e % 4)] = act_f16(acc[e] * inv, bad);
    flag_range(a.err, bad);
}

// ---------------------------------------------------------------- decode

constexpr int MAXR = 8;      // query heads per kv head
constexpr int DEC_CH = 64;       // keys per chunk of the decode split kernel

// One chunk of DEC_CH keys of one (row, kv head) for all r query heads of
// the group, on the 16x16x32 bf16 MFMA (the design of the persistent decode's
// attention units): the chunk's K and V rows go straight from memory to LDS
// (16-byte chunks XOR-swizzled by row), the heads are the MFMA columns
// (padded to 16), and each of the two 32-key groups goes to two waves that
// both form its scores S^T = K Q^T and softmax in registers and each take
// half of the dims of O^T = V^T P^T (P as a bf16 pair hi + lo).  Rows past
// the chunk's keys read the chunk's first row (a written cache slot, so V
// stays finite) and get probability 0.  The two groups' states are merged
// in LDS into the chunk partial (max, sum, unnormalised output).
template <int D>
__global__ void __launch_bounds__(256) attn_decode_split_kernel(AttnDecodeArgs a) {
    constexpr int NCK = D / 8, KROWS = 1024 / (2 * D), CH = DEC_CH;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    unsigned char* Kst = smem;                                         // [CH][D] bf16
    unsigned char* Vst = smem + CH * D * 2;                            // [CH][D] bf16
    float* ored = reinterpret_cast<float*>(Vst + CH * D * 2);          // [2][MAXR][D]
    float* gst = ored + 2 * MAXR * D;                                  // [2][MAXR][2]
    float* mst = gst + 2 * MAXR * 2;                                   // [CH]
    uint16_t* qb = reinterpret_cast<uint16_t*>(mst + CH);              // [MAXR][D]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int b = blockIdx.x / a.nkv, g = blockIdx.x % a.nkv;
    const int chunk = blockIdx.y;
    const int ctx = a.ctx_lens ? a.ctx_lens[b] : a.ctx_base + b;
    const int start = chunk * CH, end = min(start + CH, ctx + 1);
    if (start >= end) return;
    const int nkeys = end - start, ng = (nkeys + 31) / 32;
    const int r = a.nq / a.nkv;
    const uint16_t* kc = a.k_cache + (size_t)b * a.stride_b + (size_t)g * a.stride_h;
    const uint16_t* vc = a.v_cache + (size_t)b * a.stride_b + (size_t)g * a.stride_h;
    auto kswz = [](int k) { return ((k & 3) | ((k >> 1) & 12)) & (NCK - 1); };
    auto vswz = [](int k) { return 2 * ((k >> 3) & 3); };

    // K, V rows (and the mask values) straight to LDS, q of the group's heads
    for (int i = wave; i < CH / KROWS; i += 4) {
        const int row = i * KROWS + lane / NCK, pc = lane % NCK;
        const size_t src = (size_t)(start + (row < nkeys ? row : 0)) * D;
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(kc + src + (pc ^ kswz(row)) * 8),
                                         (__attribute__((address_space(3))) void*)(Kst + i * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(vc + src + (pc ^ vswz(row)) * 8),
                                         (__attribute__((address_space(3))) void*)(Vst + i * 1024), 16, 0, 0);
    }
    if (a.mask && wave == 0)
        __builtin_amdgcn_global_load_lds(
            reinterpret_cast<const void*>(a.mask + (size_t)b * a.max_seq + start + (lane < nkeys ? lane : 0)),
            (__attribute__((address_space(3))) void*)mst, 4, 0, 0);
    for (int i = tid; i < r * D / 8; i += 256)
        reinterpret_cast<u32x4*>(qb)[i] =
            *reinterpret_cast<const u32x4*>(a.q + ((size_t)b * a.nq + g * r) * D + i * 8);
    __syncthreads();           // also: the stage loads have landed

    const int n16 = lane & 15, q4 = lane >> 4;
    const int gw = wave >> 1, part = wave & 1;
    const float LOG2E = 1.4426950408889634f;
    if (gw < ng) {
        // S^T of tiles t = 0, 1: A row n16 of tile t is key 32 gw + 8 (n16 / 4)
        // + 4 t + n16 % 4, so register j of lane (n16, q4) is key 8 q4 + 4 t + j
        // of the group, head n16
        f32x4 sacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
        const int row0 = 32 * gw + 8 * (n16 >> 2) + (n16 & 3), row1 = row0 + 4;
        const unsigned char* K0 = Kst + (size_t)row0 * D * 2;
        const unsigned char* K1 = Kst + (size_t)row1 * D * 2;
        const uint16_t* qsrc = qb + (n16 < r ? n16 : 0) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < D / 32; s++) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(qsrc + 32 * s);
            const bf16x8 qf = __builtin_bit_cast(bf16x8, n16 < r ? w : u32x4{0u, 0u, 0u, 0u});
            const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(K0 + (((4 * s + q4) ^ kswz(row0)) << 4));
            const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(K1 + (((4 * s + q4) ^ kswz(row1)) << 4));
            sacc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qf, sacc[0], 0, 0, 0);
            sacc[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qf, sacc[1], 0, 0, 0);
        }
        float sv[8];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const int kk = 32 * gw + 8 * q4 + e;
            float v = sacc[e / 4][e % 4] * a.scale_log2;
            if (a.mask) v += mst[kk] * LOG2E;
            v = kk < nkeys ? v : -INFINITY;
            sv[e] = v;
            mx = fmaxf(mx, v);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        bf16x8 phi, plo;
        float ls = 0.f;
        const float mb = mx == -INFINITY ? 0.f : mx;     // (every key masked: all weights 0)
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const float pv = exp2_hw(sv[e] - mb);
            ls += pv;
            const __bf16 hi = (__bf16)pv;
            phi[e] = hi;
            plo[e] = (__bf16)(pv - (float)hi);
        }
        ls += __shfl_xor(ls, 16, 64);
        ls += __shfl_xor(ls, 32, 64);
        // O^T += V^T P^T over this wave's half of the 16-dim blocks: lane
        // (n16, q4) holds V of keys 8 q4 .. + 7, dim 16 db + n16
        // (two transposing reads: lane n16 of its group points at key
        // 8 q4 + n16 / 4 (+ 4), dims 16 db + 4 (n16 % 4) .. + 3, in their
        // swizzled chunk)
        const uint16_t* Vw = reinterpret_cast<const uint16_t*>(Vst + (size_t)(32 * gw + 8 * q4 + (n16 >> 2)) * D * 2);
#pragma unroll
        for (int d0 = 0; d0 < D / 32; d0++) {
            const int db = part * (D / 32) + d0;
            const int off = (((2 * db + ((n16 & 3) >> 1)) ^ (2 * q4)) << 3) | (4 * (n16 & 1));
            const i16x4 v0 = lds_read_tr16(Vw + off), v1 = lds_read_tr16(Vw + 4 * D + off);
            const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
            f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, phi, o, 0, 0, 0);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, plo, o, 0, 0, 0);
            if (n16 < r) *reinterpret_cast<f32x4*>(ored + (gw * MAXR + n16) * D + 16 * db + 4 * q4) = o;
        }
        if (n16 < r && q4 == 0 && part == 0) {
            gst[(gw * MAXR + n16) * 2] = mx;
            gst[(gw * MAXR + n16) * 2 + 1] = ls;
        }
    }
    __syncthreads();
    // the chunk partial of every head: the groups rescaled to their common max
    for (int idx = tid; idx < r * D; idx += 256) {
        const int i = idx / D, dim = idx - i * D;
        const float m0 = gst[i * 2], m1 = ng > 1 ? gst[(MAXR + i) * 2] : -INFINITY;
        const float M = fmaxf(m0, m1);
        float v = 0.f, l = 0.f;
        if (M != -INFINITY) {
            const float s0 = m0 == -INFINITY ? 0.f : exp2f(m0 - M);
            const float s1 = m1 == -INFINITY ? 0.f : exp2f(m1 - M);
            v = s0 * ored[i * D + dim] + (ng > 1 ? s1 * ored[(MAXR + i) * D + dim] : 0.f);
            l = s0 * gst[i * 2 + 1] + (ng > 1 ? s1 * gst[(MAXR + i) * 2 + 1] : 0.f);
        }
        float* pp = a.part + (((size_t)b * a.nq + g * r + i) * a.nchunks + chunk) * (D + 2);
        pp[dim] = v;
        if (dim == 0) { pp[D] = M; pp[D + 1] = l; }
    }
}

// Merge of the chunk partials of one (row, head): thread group gq (of
// DEC_CG groups of D threads, one thread per dim) merges the chunks
// gq, gq + DEC_CG, ... in order, in batches of CB whose states are requested
// together; the groups' states then meet in LDS and group 0 merges them in
// group order.
constexpr int DEC_CG = 4;

template <int D>
__global__ void __launch_bounds__(D * DEC_CG) attn_decode_combine_kernel(AttnDecodeArgs a) {
    __shared__ float gm[DEC_CG], gl[DEC_CG], go[DEC_CG][D];
    const int b = blockIdx.x / a.nq, head = blockIdx.x % a.nq;
    const int dim = threadIdx.x % D, gq = threadIdx.x / D;
    const int ctx = a.ctx_lens ? a.ctx_lens[b] : a.ctx_base + b;
    const int nch = (ctx + 1 + a.chunk - 1) / a.chunk;
    const float* pp = a.part + ((size_t)b * a.nq + head) * a.nchunks * (D + 2);
    constexpr int CB = 8;
    float M = -INFINITY, L = 0.f, O = 0.f;
    for (int c0 = gq; c0 < nch; c0 += CB * DEC_CG) {
        float mc[CB], lc[CB], oc[CB];
#pragma unroll
        for (int j = 0; j < CB; j++) {
            const int ch0 = c0 + j * DEC_CG;
            const int ch = ch0 < nch ? ch0 : gq;
            mc[j] = pp[ch * (D + 2) + D];
            lc[j] = pp[ch * (D + 2) + D + 1];
            oc[j] = pp[ch * (D + 2) + dim];
        }
        float Mn = M;
#pragma unroll
        for (int j = 0; j < CB; j++)
            if (c0 + j * DEC_CG < nch) Mn = fmaxf(Mn, mc[j]);
        if (Mn == -INFINITY) continue;
        const float sc = (M == -INFINITY) ? 0.f : exp2f(M - Mn);
        L *= sc;
        O *= sc;
#pragma unroll
        for (int j = 0; j < CB; j++) {
            if (c0 + j * DEC_CG >= nch || mc[j] == -INFINITY) continue;
            const float w = exp2f(mc[j] - Mn);
            L += w * lc[j];
            O += w * oc[j];
        }
        M = Mn;
    }
    if (dim == 0) { gm[gq] = M; gl[gq] = L; }
    go[gq][dim] = O;
    __syncthreads();
    if (gq != 0) return;
    float Mt = -INFINITY;
#pragma unroll
    for (int q = 0; q < DEC_CG; q++) Mt = fmaxf(Mt, gm[q]);
    float Lt = 0.f, Ot = 0.f;
    if (Mt != -INFINITY) {
#pragma unroll
        for (int q = 0; q < DEC_CG; q++) {
            if (gm[q] == -INFINITY) continue;
            const float w = exp2f(gm[q] - Mt);
            Lt += w * gl[q];
            Ot += w * go[q][dim];
        }
    }
    const float v = (Lt > 0.f) ? Ot / Lt : 0.f;
    bool bad = false;
    a.out[((size_t)b * a.nq + head) * D + dim] = act_f16(v, bad);
    flag_range(a.err, bad);
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
    if (a.chunk != DEC_CH || a.nq / a.nkv > MAXR) return -1;
    dim3 g1(a.B * a.nkv, a.nchunks), g2(a.B * a.nq);
    // K and V stages, the two groups' outputs and statistics, mask values, q
    const size_t lds = (size_t)2 * DEC_CH * a.d * 2 + (2 * MAXR * a.d + 4 * MAXR + DEC_CH) * 4 + (size_t)MAXR * a.d * 2;
    if (a.d == 128) {
        hipLaunchKernelGGL(attn_decode_split_kernel<128>, g1, dim3(256), lds, stream, a);
        hipLaunchKernelGGL(attn_decode_combine_kernel<128>, g2, dim3(128 * DEC_CG), 0, stream, a);
    } else if (a.d == 64) {
        hipLaunchKernelGGL(attn_decode_split_kernel<64>, g1, dim3(256), lds, stream, a);
        hipLaunchKernelGGL(attn_decode_combine_kernel<64>, g2, dim3(64 * DEC_CG), 0, stream, a);
    } else {
        return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
