// Decode stage in one persistent launch (one block of 16 waves per CU), run
// as a dataflow graph without grid barriers.
//
// The decode step is a chain of dependent products (Sec. 4.4):
//   P1  q/k/v GEMV on RMSNorm(x)
//   P2  split-KV attention (RoPE and bf16 of q/k/v at the consumer), then the
//       combine of the chunks into the attention output A
//   P3  o_proj GEMV                    -> partial sums of A Wo
//   P4  h = x + A Wo; gate/up GEMV on RMSNorm(h) -> g = silu(gate) * up
//   P5  down GEMV                      -> y = h + g Wd
//
// Work split: in every GEMV the block owns whole column tiles (32 columns) or
// a k-part of one, and its 16 waves split the block's k range; the waves'
// partials meet in LDS.  A block's weight tiles for the next product are
// requested (gemv_core ring) as soon as its current run is done, so the
// weight stream keeps going while the block waits for its inputs.
//
// Synchronisation: every value that one block hands to another is a 64-bit
// word (32-bit payload | 32-bit launch epoch) written with one agent-scope
// store.  A consumer polls the words it needs until each carries this
// launch's epoch; a 64-bit access is single-copy atomic, so a word with the
// right tag holds this launch's payload.  There are no counters, fences or
// grid barriers, and a consumer waits only for the producers of its own
// inputs.  Sums are formed in a fixed order: results do not depend on
// timing.  Polls are bounded: on a timeout the kernel raises an error flag
// and runs to completion.  The launch is an ordinary one with one block per
// CU (a block's LDS leaves no room for a second), so all blocks are resident
// once the CUs are free; were one not, its consumers would time out, flag
// the error and end rather than hang.
#include "common.h"
#include "gemv_core.h"
#include "launch.h"
#include "decode_fused.h"

namespace {

constexpr int NWAVE = 16;
constexpr int NTHR = NWAVE * 64;
constexpr int RING = 4;            // weight tiles in flight per wave (gate/up, down)
constexpr int RING_QKV = 4;        // q/k/v: its run is about 4 tiles per wave
constexpr int RING_O = 4;          // o_proj: its run is 2 to 4 tiles per wave
constexpr int MAXS = 2;            // k-parts of a column tile
constexpr int MAXR = 8;            // query heads per kv head

#define GLOBAL_AS __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ GLOBAL_AS T* gptr(const T* p) {
    return (GLOBAL_AS T*)(const_cast<T*>(p));
}

__device__ __forceinline__ void put_tagged(uint64_t* p, uint32_t payload, uint32_t ep) {
    __hip_atomic_store(gptr(p), ((uint64_t)ep << 32) | payload, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t get_tagged(const uint64_t* p) {
    return __hip_atomic_load(gptr(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Poll budget of a thread for the whole launch: once it is spent, waits
// give up at once (after raising the error flag), so a launch whose producer
// never writes still ends.
struct Waiter {
    int* err;
    int left;
};

// Payloads of N words at p[i] (skipped where use[i] is false), given first
// loads v[i]: poll until every tag is ep.  The late words are loaded again
// together, so a round of polling costs one memory round trip however many
// words are late.
template <int N>
__device__ __forceinline__ void settle_all(const uint64_t* const (&p)[N], uint64_t (&v)[N], const bool (&use)[N],
                                           uint32_t ep, Waiter& wt) {
    for (;;) {
        bool late = false;
#pragma unroll
        for (int i = 0; i < N; i++) late |= use[i] && (uint32_t)(v[i] >> 32) != ep;
        if (!late) return;
        if (--wt.left < 0) {
            if (wt.left == -1) raise_flag(wt.err, W4_FLAG_WAIT_TIMEOUT);
            return;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int i = 0; i < N; i++)
            if (use[i] && (uint32_t)(v[i] >> 32) != ep) v[i] = get_tagged(p[i]);
    }
}

// Block-wide read of n elements: element i is the float sum over parts
// s < S (in s order) of the tagged word at addr(i) + s * sstride, handed to
// sink(i, sum).  The loads of 4 elements per thread (all parts) go out
// together before any poll.
template <typename Addr, typename Sink>
__device__ __forceinline__ void gather_sum(int n, int S, size_t sstride, uint32_t ep, Waiter& wt, Addr addr, Sink sink) {
    constexpr int BATCH = 4, NWD = BATCH * MAXS;
    for (int base = threadIdx.x; base < n; base += NTHR * BATCH) {
        const uint64_t* p[NWD];
        uint64_t v[NWD];
        bool use[NWD];
#pragma unroll
        for (int j = 0; j < BATCH; j++) {
            const int i = base + j * NTHR;
#pragma unroll
            for (int s = 0; s < MAXS; s++) {
                const int w = j * MAXS + s;
                use[w] = i < n && s < S;
                p[w] = addr(use[w] ? i : base) + (use[w] ? (size_t)s * sstride : 0);
                v[w] = use[w] ? get_tagged(p[w]) : 0;
            }
        }
        settle_all(p, v, use, ep, wt);
#pragma unroll
        for (int j = 0; j < BATCH; j++) {
            const int i = base + j * NTHR;
            if (i >= n) break;
            float sum = 0.f;
#pragma unroll
            for (int s = 0; s < MAXS; s++)
                if (s < S) sum += __uint_as_float((uint32_t)v[j * MAXS + s]);
            sink(i, sum);
        }
    }
}

// Block-wide read of n raw payloads: element i is the tagged word at addr(i)
// (skipped when addr(i) is null), handed to sink(i, payload).
template <typename Addr, typename Sink>
__device__ __forceinline__ void gather_raw(int n, uint32_t ep, Waiter& wt, Addr addr, Sink sink) {
    constexpr int BATCH = 8;
    for (int base = threadIdx.x; base < n; base += NTHR * BATCH) {
        const uint64_t* p[BATCH];
        uint64_t v[BATCH];
        bool use[BATCH];
#pragma unroll
        for (int j = 0; j < BATCH; j++) {
            const int i = base + j * NTHR;
            p[j] = i < n ? addr(i) : nullptr;
            use[j] = p[j] != nullptr;
            v[j] = use[j] ? get_tagged(p[j]) : 0;
        }
        settle_all(p, v, use, ep, wt);
#pragma unroll
        for (int j = 0; j < BATCH; j++) {
            const int i = base + j * NTHR;
            if (i >= n) break;
            if (use[j]) sink(i, (uint32_t)v[j]);
        }
    }
}

// RMSNorm of B rows (fp32, row b at src + b * K, in LDS) into activation
// rows prepared for the GEMV core (gemv_prep): x' as fp16 at xs[b * ldx + k]
// and the correction table c64.  gamma: bf16 bits in LDS.  K a multiple of
// 128.  red8: 8 + NWAVE * B floats of LDS scratch.  Each thread takes 4
// adjacent elements per pass, so the 16 lanes of a DPP row hold one 64-k tile.
__device__ __forceinline__ void norm_prep_rows(const float* src, const uint16_t* gamma, float eps, int B, int K,
                                               f16* xs, int ldx, float* c64, float* red8, int* err) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int b = 0; b < B; b++) {
        float ss = 0.f;
        for (int k = 4 * tid; k < K; k += 4 * NTHR) {
            const float4 v = *reinterpret_cast<const float4*>(src + b * K + k);
            ss += (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
        }
        ss = wave_sum(ss);
        if (lane == 0) red8[8 + b * NWAVE + wave] = ss;
    }
    __syncthreads();
    if (tid < B) {
        float t = 0.f;
        for (int w = 0; w < NWAVE; w++) t += red8[8 + tid * NWAVE + w];
        red8[tid] = 1.0f / sqrtf(t / (float)K + eps);
    }
    __syncthreads();
    const f16 sixteenth = (f16)0.0625f;
    bool bad = false;
    for (int b = 0; b < B; b++) {
        const float rb = red8[b];
        for (int k0 = 0; k0 < K; k0 += 4 * NTHR) {          // uniform passes
            const int k = k0 + 4 * tid;
            float e = 0.f, o = 0.f;
            if (k < K) {
                // elements k % 8 = 0, 1 (or 4, 5) as they are, 2, 3 (or 6, 7) divided by 16
                const float4 v = *reinterpret_cast<const float4*>(src + b * K + k);
                const uint2 g = *reinterpret_cast<const uint2*>(gamma + k);
                const f16 y0 = act_f16(v.x * rb * __uint_as_float(g.x << 16), bad);
                const f16 y1 = act_f16(v.y * rb * __uint_as_float(g.x & 0xFFFF0000u), bad);
                const f16 y2 = act_f16(v.z * rb * __uint_as_float(g.y << 16), bad) * sixteenth;
                const f16 y3 = act_f16(v.w * rb * __uint_as_float(g.y & 0xFFFF0000u), bad) * sixteenth;
                e = (float)y0 + (float)y1;
                o = (float)y2 + (float)y3;
                f16 q[4] = {y0, y1, y2, y3};
                *reinterpret_cast<uint2*>(xs + b * ldx + k) = *reinterpret_cast<const uint2*>(q);
            }
            e = row_sum<16>(e);
            o = row_sum<16>(o);
            if (k < K && (lane & 15) == 0) c64[(k >> 6) * GEMV_ROWS + b] = gemv_c64(e, o);
        }
    }
    flag_range(err, bad);
    __syncthreads();
}

// Device position (inside a head) of dim j: the head's 32-dim blocks are
// stored in the order that puts RoPE partners in adjacent tiles.
template <int D>
__device__ __forceinline__ int devpos(int j) {
    constexpr int half = D / 64;
    const int jb = j >> 5;
    const int p = jb < half ? 2 * jb : 2 * (jb - half) + 1;
    return p * 32 + (j & 31);
}

// Chunk partial of head i, dim `dim` from the ng key groups' (max, sum,
// output) in LDS (gst [group][MAXR][2], ored [group][MAXR][D]), rescaled to
// their common max M.  NGR >= ng bounds the unrolled loop; the slots past
// ng read group 0 and weigh 0, so the loads need no branches.
template <int NGR, int D>
__device__ __forceinline__ void group_merge(const float* gst, const float* ored, int ng, int i, int dim, float& M,
                                            float& v, float& l) {
    float mw[NGR];
#pragma unroll
    for (int w = 0; w < NGR; w++) mw[w] = gst[((w < ng ? w : 0) * MAXR + i) * 2];
    M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NGR; w++) M = w < ng ? fmaxf(M, mw[w]) : M;
    v = 0.f;
    l = 0.f;
#pragma unroll
    for (int w = 0; w < NGR; w++) {
        const int ww = w < ng ? w : 0;
        const float sc = (w < ng && mw[w] != -INFINITY) ? exp2f(mw[w] - M) : 0.f;
        v += sc * ored[(ww * MAXR + i) * D + dim];
        l += sc * gst[(ww * MAXR + i) * 2 + 1];
    }
}

// ---------------------------------------------------------------- kernel

template <int D, int MAXB>
__global__ void __launch_bounds__(NTHR) decode_fused_kernel(DecodeFusedArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int blk = blockIdx.x, P = gridDim.x;
    const int B = a.B, H = a.H, nq = a.nq, nkv = a.nkv, r = nq / nkv;
    const int qd = nq * D, kd = nkv * D;
    const uint32_t ep = a.epoch;
    Waiter wt{a.err, a.spin_max};
    const int ldx = a.ldx;
    const int h = lane >> 5, c = lane & 31;
    f16* xs = reinterpret_cast<f16*>(smem);
    float* hbuf = reinterpret_cast<float*>(smem + a.off_h);       // [B][H]
    const int SLOTS = a.slots;                                    // column tiles per block in one product
    float* red = reinterpret_cast<float*>(smem + a.off_red);      // [NWAVE][SLOTS][B][32]
    float* red8 = red + NWAVE * SLOTS * MAXB * 32;                // 8 + NWAVE * MAXB
    float* own = red8 + 8 + NWAVE * MAXB;                         // [MAXB][32]
    int* meta = reinterpret_cast<int*>(own + MAXB * 32);          // ctx_lens[B], pos[B]
    uint16_t* gam = reinterpret_cast<uint16_t*>(smem + a.off_gam);           // RMSNorm weights [2][H]
    const bool gam_lds = MAXB == 1 || a.gam_lds;                             // (one row always has room)
    f16* zero64 = reinterpret_cast<f16*>(smem + a.off_zero);                  // 64 zeros (GEMV phases)
    float* c64 = reinterpret_cast<float*>(smem + a.off_c64);                  // GEMV corrections

    if (a.stamps && blk == 0 && tid == 0) {
        a.stamps[0] = wall_clock64();
        a.stamps[1] = (unsigned long long)P;
    }
    // stamp slot ph of this block: 0..4 end of the five phases, 5.. detail
    auto stamp_done = [&](int ph) {
        if (a.stamps && tid == 0) a.stamps[8 + ph * P + blk] = wall_clock64();
    };
    stamp_done(5);

    // ---- this block's work: column tiles and k ranges per product, computed
    // here (a table in memory would put a dependent load before the first
    // weight request).  pl[0..3] q/k/v, pl[4..7] o_proj: column tile (-1:
    // none), k-tile range [ka, kz), k part; pl[8..9] gate/up: column tiles
    // [t0, t1) (whole gate/up pairs); pl[10..13] down.  A product of nt column
    // tiles cut into S k parts (S <= 2) gives block blk tile blk / S, part
    // blk % S, if blk < nt S.
    static_assert(MAXS == 2, "k parts: 1 or 2");
    int pl[16];
    {
        auto part = [&](const DevLinear& W, int S, int* e) {
            const int nt = W.N_dev / 32, kb = W.K_pad / 64;
            const bool on = blk < nt * S;
            const int s = S == 1 ? 0 : blk & 1;
            e[0] = on ? (S == 1 ? blk : blk >> 1) : -1;
            e[1] = on ? s * kb / S : 0;
            e[2] = on ? (s + 1) * kb / S : 0;
            e[3] = on ? s : 0;
        };
        part(a.qkv, a.S_qkv, pl);
        part(a.o, a.S_o, pl + 4);
        const unsigned np = (unsigned)a.gu.N_dev / 64;
        pl[8] = 2 * (int)((unsigned)blk * np / (unsigned)P);
        pl[9] = 2 * (int)((unsigned)(blk + 1) * np / (unsigned)P);
        part(a.down, a.S_down, pl + 10);
        pl[14] = pl[15] = 0;
    }
    const int Nq = a.qkv.N_dev;
    // this wave's run of product ph (1 q/k/v, 3 o_proj, 4 gate/up, 5 down)
    auto wave_run = [&](int ph) {
        int t0, tz, ka, kz;
        if (ph == 4) { t0 = pl[8]; tz = pl[9]; ka = 0; kz = a.gu.K_pad / 64; }
        else {
            const int e = ph == 1 ? 0 : ph == 3 ? 4 : 10;
            t0 = pl[e]; tz = t0 + 1; ka = pl[e + 1]; kz = pl[e + 2];
        }
        return Run{t0, tz, ka + wave * (kz - ka) / NWAVE, ka + (wave + 1) * (kz - ka) / NWAVE};
    };
    auto owns = [&](int ph) { return ph == 4 ? pl[9] > pl[8] : pl[ph == 1 ? 0 : ph == 3 ? 4 : 10] >= 0; };

    // one ring per product, sized for its usual run length; a product's ring
    // is filled as soon as the previous product's tiles are all consumed
    TileRing<RING_QKV, false> R1;
    TileRing<RING_O, false> R3;
    TileRing<RING, false> R4, R5;
    RunCursor q1, q3, q4, q5;
    auto prefetch = [&](int ph) {
        if (!owns(ph)) return;
        const Run run = wave_run(ph);
        if (run.ka >= run.kz) return;
        if (ph == 1) ring_prefetch<RING_QKV, false, false>(a.qkv, run, R1, q1);
        if (ph == 3) ring_prefetch<RING_O, false, false>(a.o, run, R3, q3);
        if (ph == 4) ring_prefetch<RING, false, false>(a.gu, run, R4, q4);
        if (ph == 5) ring_prefetch<RING, false, false>(a.down, run, R5, q5);
    };
    // this wave's part of the block partial of slot `slot`
    auto to_red = [&](int slot, const float (&out)[4]) {
#pragma unroll
        for (int qq = 0; qq < 4; qq++) {
            const int b = 4 * h + qq;
            if (b < B) red[((wave * SLOTS + slot) * B + b) * 32 + c] = out[qq];
        }
    };
    // (after a block barrier: the last product's partials may still be read)
    auto clear_red = [&]() {
        __syncthreads();
        for (int i = lane; i < SLOTS * B * 32; i += 64) red[wave * SLOTS * B * 32 + i] = 0.f;
    };
    // block sum of slot `slot`, row b, column cc (after a __syncthreads)
    auto red_sum = [&](int slot, int b, int cc) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < NWAVE; w++) v += red[((w * SLOTS + slot) * B + b) * 32 + cc];
        return v;
    };

    // x, the RMSNorm weights and the per-row metadata into LDS: every load of a
    // thread is issued before its first wait, and before the weight prefetch
    {
        float4 xv[2];
        u32x4 g1, g2;
        const int i0 = tid * 4, i1 = i0 + NTHR * 4;
        xv[0] = i0 < B * H ? *reinterpret_cast<const float4*>(a.x + i0) : float4{0.f, 0.f, 0.f, 0.f};
        xv[1] = i1 < B * H ? *reinterpret_cast<const float4*>(a.x + i1) : float4{0.f, 0.f, 0.f, 0.f};
        const int gi = tid * 8 < H ? tid * 8 : 0;
        g1 = *reinterpret_cast<const u32x4*>(a.attn_norm + gi);
        g2 = *reinterpret_cast<const u32x4*>(a.mlp_norm + gi);
        int m0 = 0;
        if (tid < B) m0 = a.ctx_lens ? a.ctx_lens[tid] : a.ctx_base + tid;
        else if (tid >= MAXB && tid < MAXB + B) m0 = a.pos[tid - MAXB];
        prefetch(1);
        if (i0 < B * H) *reinterpret_cast<float4*>(hbuf + i0) = xv[0];
        if (i1 < B * H) *reinterpret_cast<float4*>(hbuf + i1) = xv[1];
        if (gam_lds && tid * 8 < H) {
            *reinterpret_cast<u32x4*>(gam + tid * 8) = g1;
            *reinterpret_cast<u32x4*>(gam + H + tid * 8) = g2;
        }
        if (tid < MAXB + B) meta[tid] = m0;
        if (tid < 8) reinterpret_cast<u32x4*>(zero64)[tid] = u32x4{0u, 0u, 0u, 0u};
        for (int i = i1 + NTHR * 4; i < B * H; i += NTHR * 4)      // rows past 2 * NTHR * 4 floats
            *reinterpret_cast<float4*>(hbuf + i) = *reinterpret_cast<const float4*>(a.x + i);
        for (int i = tid * 8 + NTHR * 8; gam_lds && i < H; i += NTHR * 8) {
            *reinterpret_cast<u32x4*>(gam + i) = *reinterpret_cast<const u32x4*>(a.attn_norm + i);
            *reinterpret_cast<u32x4*>(gam + H + i) = *reinterpret_cast<const u32x4*>(a.mlp_norm + i);
        }
        __syncthreads();
    }
    stamp_done(23);

    // ================= P1: q/k/v partial sums =================
    if (owns(1)) {
        const int t1 = pl[0], s1 = pl[3];
        const Run run1 = wave_run(1);
        // (the RMSNorm weights are in LDS unless the block's LDS has no room)
        norm_prep_rows(hbuf, gam_lds ? gam : a.attn_norm, a.eps, B, H, xs, ldx, c64, red8, a.err);
        stamp_done(6);
        clear_red();
        const GemvAct xa{xs, ldx, c64, nullptr, zero64};
        if (run1.ka < run1.kz)
            gemv_run<RING_QKV, false, false, MAXB == 1>(a.qkv, run1, xa, B, R1, q1, [&](int, const float (&out)[4]) { to_red(0, out); });
        stamp_done(7);
        __syncthreads();
        for (int i = tid; i < B * 32; i += NTHR) {
            const int b = i >> 5, cc = i & 31;
            put_tagged(a.qkv_part + ((size_t)s1 * B + b) * Nq + t1 * 32 + cc, __float_as_uint(red_sum(0, b, cc)), ep);
        }
    }
    // ================= P2: attention units =================
    // A unit is one chunk of keys of one (row, kv head).  Its K and V rows go
    // straight from memory to LDS; the r query heads of the group are the
    // columns of the 16x16x32 bf16 MFMA.  Key group k (keys 32k .. 32k + 31)
    // goes to two waves: each forms the group's scores S^T = K Q^T as two
    // 16-key tiles whose rows are fed in the order that leaves the
    // probabilities in the operand layout of P^T, the softmax over the
    // group's keys in registers, then half of the dims of O^T = V^T P^T with
    // P as a bf16 pair hi + lo.  The groups' (max, sum, output) meet in LDS
    // and leave as one chunk partial (up to 8 groups: 256 keys).
    {
        constexpr int NCK = D / 8;                   // 16-byte chunks per K / V row
        constexpr int KROWS = 1024 / (2 * D);         // rows per 1 KB stage load
        const int CH = a.chunk, NCH = a.nchunk;
        const int CHP = (CH + 31) & ~31, NG = CHP / 32;
        unsigned char* Kst = smem;                                           // [CHP][D] bf16
        unsigned char* Vst = smem + (size_t)CHP * D * 2;                     // [CHP][D] bf16
        float* ored = reinterpret_cast<float*>(Vst + (size_t)CHP * D * 2);   // [NG][MAXR][D]
        float* gst = ored + NG * MAXR * D;                                   // [NG][MAXR][2]
        // q/k/v of the unit's row (r + 2 rows), then k/v of up to 3 earlier
        // rows (shared-cache mode)
        float* qkvf = gst + NG * MAXR * 2;                                   // [r + 2 + 6][D] device order
        uint16_t* qb = reinterpret_cast<uint16_t*>(qkvf + (MAXR + 8) * D);    // [r][D] bf16
        uint16_t* knb = qb + MAXR * D;                                       // [D]
        uint16_t* vnb = knb + D;                                             // [D]
        float* mst = reinterpret_cast<float*>(vnb + D);                      // [CHP] mask values
        // 16-byte chunk c of stage row k sits at c ^ kswz(k) (K) or c ^ vswz(k)
        // (V): the fragment reads below then hit distinct banks
        auto kswz = [](int k) { return ((k & 3) | ((k >> 1) & 12)) & (NCK - 1); };
        auto vswz = [](int k) { return 2 * ((k >> 3) & 3); };
        const float LOG2E = 1.4426950408889634f;
        const int n16 = lane & 15, q4 = lane >> 4;
        const int units = B * nkv * NCH;
        // K and V rows start .. start + 32 ng - 1 of unit u into the stages;
        // rows past the history (the new key, the padding) read row 0 and
        // are rewritten before use
        auto load_stage = [&](int u) {
            const int b = u / (nkv * NCH), g = (u / NCH) % nkv, chunk = u % NCH;
            const int ctx = meta[b];
            const int start = chunk * CH, end = min(start + CH, ctx + 1);
            const int hist_end = min(end, a.shared ? a.ctx_base : ctx), ng = (end - start + 31) / 32;
            if (a.mask && wave < ng / 2 + (ng & 1)) {     // mask values of keys start + 64 wave + lane
                const int kk = 64 * wave + lane;
                __builtin_amdgcn_global_load_lds(
                    reinterpret_cast<const void*>(a.mask + (size_t)b * a.max_seq + (start + kk < end ? start + kk : start)),
                    (__attribute__((address_space(3))) void*)(mst + 64 * wave), 4, 0, 0);
            }
            const uint16_t* kc = a.k_cache + (size_t)b * a.sb + (size_t)g * a.sh;
            const uint16_t* vc = a.v_cache + (size_t)b * a.sb + (size_t)g * a.sh;
            for (int i = wave; i < ng * 32 / KROWS; i += NWAVE) {
                const int row = i * KROWS + lane / NCK, pc = lane % NCK;
                const int key = start + row;
                const size_t src = (size_t)(key < hist_end ? key : 0) * D;
                __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(kc + src + (pc ^ kswz(row)) * 8),
                                                 (__attribute__((address_space(3))) void*)(Kst + i * 1024), 16, 0, 0);
                __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(vc + src + (pc ^ vswz(row)) * 8),
                                                 (__attribute__((address_space(3))) void*)(Vst + i * 1024), 16, 0, 0);
            }
        };
        // The o_proj weights are requested once the q/k/v results went out
        // (the memory pipeline serves a wave's requests in order), then the
        // first unit's K and V; P1 has finished with the activation rows that
        // the stages overwrite.
        prefetch(3);
        if (blk < units) load_stage(blk);
        stamp_done(0);
        for (int u = blk; u < units; u += P) {
            const int b = u / (nkv * NCH), g = (u / NCH) % nkv, chunk = u % NCH;
            const int ctx = meta[b];
            const int start = chunk * CH, end = min(start + CH, ctx + 1);
            if (start >= end) continue;
            const int nkeys = end - start;
            const int ng = (nkeys + 31) / 32;
            // two waves per key group: each repeats the group's scores and
            // softmax and takes half of its 16-dim blocks of P V
            constexpr int ns = 2;
            const int gw = wave / ns, part = wave % ns;
            if (u != blk) load_stage(u);
            // the RoPE factors of this thread's dim, requested before the wait
            // for q/k/v
            const int ps = meta[MAXB + b];
            const int jr = tid % (D / 2);            // the RoPE dim of every item of this thread
            const float rc = a.rope_cos[(size_t)ps * (D / 2) + jr], rs = a.rope_sin[(size_t)ps * (D / 2) + jr];
            // Shared-cache mode (rows are consecutive tokens of one sequence):
            // the earlier rows o_lo .. o_lo + np - 1 hold slots of this chunk
            // that no launch has written yet; their keys and values come from
            // their q/k/v parts, rotated with their own positions.
            const int o_lo = a.shared ? max(0, start - a.ctx_base) : 0;
            const int np = a.shared ? max(0, min(b, end - a.ctx_base) - o_lo) : 0;
            float rco[3], rso[3];
#pragma unroll
            for (int j = 0; j < 3; j++) {
                const int pj = j < np ? meta[MAXB + o_lo + j] : 0;
                rco[j] = j < np ? a.rope_cos[(size_t)pj * (D / 2) + jr] : 0.f;
                rso[j] = j < np ? a.rope_sin[(size_t)pj * (D / 2) + jr] : 0.f;
            }
            // q (r heads), k_new, v_new of row b, then k and v of the earlier
            // rows: sums of the q/k/v parts
            const uint64_t* qrow = a.qkv_part + (size_t)b * Nq;
            gather_sum((r + 2 + 2 * np) * D, a.S_qkv, (size_t)B * Nq, ep, wt,
                       [&](int i) -> const uint64_t* {
                           if (i >= (r + 2) * D) {
                               const int jo = (i - (r + 2) * D) / (2 * D), rem = i - (r + 2) * D - jo * 2 * D;
                               const int col = rem < D ? qd + g * D + rem : qd + kd + g * D + (rem - D);
                               return a.qkv_part + (size_t)(o_lo + jo) * Nq + col;
                           }
                           const int col = i < r * D ? g * r * D + i
                                         : i < (r + 1) * D ? qd + g * D + (i - r * D)
                                                           : qd + kd + g * D + (i - (r + 1) * D);
                           return qrow + col;
                       },
                       [&](int i, float v) { qkvf[i] = v; });
            __syncthreads();           // also: the stage loads have landed
            stamp_done(8);
            // RoPE of q and k (Sec. 3.1, table of Sec. 4.6.2), bf16; the new
            // key and value also replace stage row ctx - start when the chunk
            // holds it, and the padding rows of V become zeros (their
            // probabilities are 0, and 0 times a stale NaN would not be)
            const int nrow = ctx - start;
            const bool has_new = ctx < end;
            for (int i = tid; i < (r + 1 + np) * (D / 2); i += NTHR) {
                const int hh = i / (D / 2), j = jr;
                const int jo = hh - r - 1;                    // earlier row (hh > r)
                const float* src = hh <= r ? qkvf + hh * D : qkvf + (r + 2) * D + jo * 2 * D;
                const float cs = jo < 0 ? rc : jo == 0 ? rco[0] : jo == 1 ? rco[1] : rco[2];
                const float sn = jo < 0 ? rs : jo == 0 ? rso[0] : jo == 1 ? rso[1] : rso[2];
                const float v0 = src[devpos<D>(j)], v1 = src[devpos<D>(j + D / 2)];
                const uint16_t e0 = bf16_bits_rne(v0 * cs - v1 * sn), e1 = bf16_bits_rne(v1 * cs + v0 * sn);
                if (hh < r) {
                    qb[hh * D + j] = e0;
                    qb[hh * D + j + D / 2] = e1;
                } else {
                    if (hh == r) {
                        knb[j] = e0;
                        knb[j + D / 2] = e1;
                    }
                    const int row = hh == r ? nrow : a.ctx_base + o_lo + jo - start;
                    if (hh > r || has_new) {
                        uint16_t* kr = reinterpret_cast<uint16_t*>(Kst + (size_t)row * D * 2);
                        kr[(((j >> 3) ^ kswz(row)) << 3) | (j & 7)] = e0;
                        kr[((((j + D / 2) >> 3) ^ kswz(row)) << 3) | (j & 7)] = e1;
                    }
                }
            }
            for (int j = tid; j < D * (1 + np); j += NTHR) {
                const int ro = j / D, dm = j - ro * D;         // ro 0: this row's value, ro > 0: earlier row ro - 1
                const float* src = ro == 0 ? qkvf + (r + 1) * D : qkvf + (r + 2) * D + (ro - 1) * 2 * D + D;
                const uint16_t e = bf16_bits_rne(src[devpos<D>(dm)]);
                if (ro == 0) vnb[dm] = e;
                const int row = ro == 0 ? nrow : a.ctx_base + o_lo + ro - 1 - start;
                if (ro > 0 || has_new)
                    reinterpret_cast<uint16_t*>(Vst + (size_t)row * D * 2)[(((dm >> 3) ^ vswz(row)) << 3) | (dm & 7)] = e;
            }
            for (int i = tid; i < (ng * 32 - nkeys) * NCK; i += NTHR)
                reinterpret_cast<u32x4*>(Vst + (size_t)nkeys * D * 2)[i] = u32x4{0u, 0u, 0u, 0u};
            __syncthreads();
            stamp_done(16);
            if (chunk == 0) {     // the new row goes to cache slot ctx (read by later launches only)
                uint16_t* kw = a.k_cache + (size_t)b * a.sb + (size_t)g * a.sh + (size_t)ctx * D;
                uint16_t* vw = a.v_cache + (size_t)b * a.sb + (size_t)g * a.sh + (size_t)ctx * D;
                for (int j = tid; j < D; j += NTHR) { kw[j] = knb[j]; vw[j] = vnb[j]; }
            }
            if (gw < ng) {
                // S^T of the tiles t = 0, 1: A row n16 of tile t is key
                // 32 gw + 8 (n16 / 4) + 4 t + n16 % 4, so output register j of
                // lane (n16, q4) is key 8 q4 + 4 t + j of the group's 32, head n16.
                // Q^T (B operand): head n16 (zero past r), dims 32 s + 8 q4 .. + 7
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
                // scores in the log2 domain, masked past the chunk; max and sum
                // over the group's keys (registers, then lanes n16 + 16 q4)
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
                // O^T += V^T P^T per 16-dim block: lane (n16, q4) holds V of keys
                // 8 q4 .. + 7, dim 16 db + n16
                // (two transposing reads: lane n16 of its group points at key
                // 8 q4 + n16 / 4 (+ 4), dims 16 db + 4 (n16 % 4) .. + 3, in
                // their swizzled chunk)
                const uint16_t* Vw = reinterpret_cast<const uint16_t*>(Vst + (size_t)(32 * gw + 8 * q4 + (n16 >> 2)) * D * 2);
                const int nb = D / 16 / ns;
#pragma unroll
                for (int d0 = 0; d0 < D / 16; d0++) {
                    if (d0 >= nb) break;
                    const int db = part * nb + d0;
                    const int off = (((2 * db + ((n16 & 3) >> 1)) ^ (2 * q4)) << 3) | (4 * (n16 & 1));
                    const i16x4 v0 = lds_read_tr16(Vw + off), v1 = lds_read_tr16(Vw + 4 * D + off);
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
                    f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
                    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, phi, o, 0, 0, 0);
                    o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, plo, o, 0, 0, 0);
                    // register j: dim 16 db + 4 q4 + j of head n16
                    if (n16 < r)
                        *reinterpret_cast<f32x4*>(ored + (gw * MAXR + n16) * D + 16 * db + 4 * q4) = o;
                }
                if (n16 < r && q4 == 0 && part == 0) {
                    gst[(gw * MAXR + n16) * 2] = mx;
                    gst[(gw * MAXR + n16) * 2 + 1] = ls;
                }
            }
            __syncthreads();
            stamp_done(17);
            // the chunk partial: the groups' outputs rescaled to the common max
            uint64_t* ap = a.apart + ((size_t)b * nq + g * r) * NCH * (D + 2) + (size_t)chunk * (D + 2);
            for (int idx = tid; idx < r * D; idx += NTHR) {
                const int i = idx / D, dim = idx - i * D;
                float M, v, l;
                if (ng <= 4) group_merge<4, D>(gst, ored, ng, i, dim, M, v, l);
                else group_merge<8, D>(gst, ored, ng, i, dim, M, v, l);
                uint64_t* aph = ap + (size_t)i * NCH * (D + 2);
                put_tagged(aph + dim, __float_as_uint(v), ep);
                if (dim == 0) {
                    put_tagged(aph + D, __float_as_uint(M), ep);
                    put_tagged(aph + D + 1, __float_as_uint(l), ep);
                }
            }
            // the next unit writes the stages and q/k/v only after its own
            // first barrier, and the group outputs after its second: every
            // thread has finished this unit's reads by then
        }
        __syncthreads();
        stamp_done(9);

        // ---- combine: this block's slice [v0, v1) of A (an even count).  LPV
        // lanes share one value (each holds one chunk or more), so the max and
        // the two sums over the chunks are lane shuffles.
        const int V = B * qd, per = a.comb_per;
        const int v0 = min(V, blk * per), v1 = min(V, v0 + per), nv = v1 - v0;
        uint16_t* abuf = reinterpret_cast<uint16_t*>(smem);
        if (nv > 0) {
            bool bad = false;
            const int LPV = a.comb_lpv, VPW = 64 / LPV;          // lanes per value (power of two)
            const int cpl = (NCH + LPV - 1) / LPV;                // chunks per lane (<= 4)
            for (int vb = wave * VPW; vb < nv; vb += NWAVE * VPW) {
                const int j = vb + lane / LPV, cl = lane % LPV;
                const bool valid = j < nv;
                const int vv = v0 + (valid ? j : 0);
                const int head = vv / D, dim = vv - head * D;     // head over all rows: b * nq + head
                const int b = head / nq;
                const int nch = (meta[b] + 1 + CH - 1) / CH;
                const uint64_t* base = a.apart + (size_t)head * NCH * (D + 2);
                // words of chunk qq: 3 qq (output dim), 3 qq + 1 (max), 3 qq + 2 (sum)
                const uint64_t* pw[12];
                uint64_t tw[12];
                bool uw[12];
#pragma unroll
                for (int qq = 0; qq < 4; qq++) {
                    const int ch = cl + qq * LPV;
                    const bool use = valid && qq < cpl && ch < nch;
                    const uint64_t* p = base + (size_t)(use ? ch : 0) * (D + 2);
                    pw[3 * qq] = p + dim;
                    pw[3 * qq + 1] = p + D;
                    pw[3 * qq + 2] = p + D + 1;
#pragma unroll
                    for (int e = 0; e < 3; e++) {
                        uw[3 * qq + e] = use;
                        tw[3 * qq + e] = use ? get_tagged(pw[3 * qq + e]) : 0;
                    }
                }
                settle_all(pw, tw, uw, ep, wt);
                float m[4], l[4], o[4];
#pragma unroll
                for (int qq = 0; qq < 4; qq++) {
                    if (uw[3 * qq]) {
                        o[qq] = __uint_as_float((uint32_t)tw[3 * qq]);
                        m[qq] = __uint_as_float((uint32_t)tw[3 * qq + 1]);
                        l[qq] = __uint_as_float((uint32_t)tw[3 * qq + 2]);
                    } else {
                        o[qq] = 0.f; m[qq] = -INFINITY; l[qq] = 0.f;
                    }
                }
                float M = fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3]));
                for (int off = 1; off < LPV; off <<= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
                float L = 0.f, O = 0.f;
                if (M != -INFINITY) {
#pragma unroll
                    for (int qq = 0; qq < 4; qq++) {
                        if (m[qq] == -INFINITY) continue;
                        const float w = exp2f(m[qq] - M);
                        L += w * l[qq];
                        O += w * o[qq];
                    }
                }
                for (int off = 1; off < LPV; off <<= 1) {
                    L += __shfl_xor(L, off, 64);
                    O += __shfl_xor(O, off, 64);
                }
                if (valid && cl == 0) abuf[j] = __builtin_bit_cast(uint16_t, act_f16(L > 0.f ? O / L : 0.f, bad));
            }
            flag_range(a.err, bad);
            __syncthreads();
            stamp_done(10);
            for (int j = 2 * tid; j < nv; j += 2 * NTHR)
                put_tagged(a.A + (v0 + j) / 2, (uint32_t)abuf[j] | ((uint32_t)abuf[j + 1] << 16), ep);
        }
        __syncthreads();
    }
    stamp_done(1);

    // ================= P3: o_proj partial sums =================
    if (owns(3)) {
        const int t3 = pl[4], ka3 = pl[5], kz3 = pl[6], s3 = pl[7];
        const Run run3 = wave_run(3);
        const int klo = ka3 * 64, kh = (kz3 - ka3) * 32;       // k range in fp16 pairs
        for (int b = 0; b < B; b++) {
            const uint64_t* src = a.A + ((size_t)b * qd + klo) / 2;
            f16* dst = xs + b * ldx;
            gather_raw(kh, ep, wt, [&](int i) -> const uint64_t* { return src + i; },
                       [&](int i, uint32_t p) { *reinterpret_cast<uint32_t*>(dst + 2 * i) = p; });
        }
        stamp_done(11);
        clear_red();
        if (tid < 8) reinterpret_cast<u32x4*>(zero64)[tid] = u32x4{0u, 0u, 0u, 0u};   // (attention reused it)
        gemv_prep(xs - klo, ldx, c64 - ka3 * GEMV_ROWS, nullptr, B, klo, 2 * kh, tid, NTHR);
        __syncthreads();
        stamp_done(19);
        const GemvAct xa{xs - klo, ldx, c64 - ka3 * GEMV_ROWS, nullptr, zero64};
        if (run3.ka < run3.kz)
            gemv_run<RING_O, false, false, MAXB == 1>(a.o, run3, xa, B, R3, q3, [&](int, const float (&out)[4]) { to_red(0, out); });
        stamp_done(20);
        __syncthreads();
        stamp_done(21);
        for (int i = tid; i < B * 32; i += NTHR) {
            const int b = i >> 5, cc = i & 31;
            put_tagged(a.o_part + ((size_t)s3 * B + b) * H + t3 * 32 + cc, __float_as_uint(red_sum(0, b, cc)), ep);
        }
    }
    prefetch(4);
    stamp_done(2);

    // ================= P4: h, RMSNorm(h), gate/up, SwiGLU =================
    gather_sum(B * H, a.S_o, (size_t)B * H, ep, wt, [&](int i) { return a.o_part + i; },
               [&](int i, float v) { hbuf[i] += v; });
    __syncthreads();
    stamp_done(12);
    if (owns(4)) {
        const int ta4 = pl[8], tb4 = pl[9];
        const Run run4 = wave_run(4);
        if (tid < 8) reinterpret_cast<u32x4*>(zero64)[tid] = u32x4{0u, 0u, 0u, 0u};   // (attention reused it)
        norm_prep_rows(hbuf, gam_lds ? gam + H : a.mlp_norm, a.eps, B, H, xs, ldx, c64, red8, a.err);
        stamp_done(22);
        clear_red();
        const GemvAct xa{xs, ldx, c64, nullptr, zero64};
        if (run4.ka < run4.kz)
            gemv_run<RING, false, false, MAXB == 1>(a.gu, run4, xa, B, R4, q4,
                                         [&](int t, const float (&out)[4]) { to_red(t - ta4, out); });
        stamp_done(13);
        __syncthreads();
        stamp_done(24);
        const int np = (tb4 - ta4) / 2;
        bool bad = false;
        for (int i = tid; i < np * B * 16; i += NTHR) {
            const int pp = i / (B * 16), rem = i - pp * B * 16, b = rem >> 4, cc = 2 * (rem & 15);
            const f16 g0 = act_f16(silu(red_sum(2 * pp, b, cc)) * red_sum(2 * pp + 1, b, cc), bad);
            const f16 g1 = act_f16(silu(red_sum(2 * pp, b, cc + 1)) * red_sum(2 * pp + 1, b, cc + 1), bad);
            const uint32_t word = (uint32_t)__builtin_bit_cast(uint16_t, g0) | ((uint32_t)__builtin_bit_cast(uint16_t, g1) << 16);
            put_tagged(a.g + ((size_t)b * a.F_pad + (ta4 / 2 + pp) * 32 + cc) / 2, word, ep);
        }
        flag_range(a.err, bad);
    }
    prefetch(5);
    stamp_done(3);

    // ================= P5: down, y = h + g Wd =================
    if (owns(5)) {
        const int t5 = pl[10], ka5 = pl[11], kz5 = pl[12], s5 = pl[13];
        const Run run5 = wave_run(5);
        const int klo = ka5 * 64, kh = (kz5 - ka5) * 32;
        for (int b = 0; b < B; b++) {
            const uint64_t* src = a.g + ((size_t)b * a.F_pad + klo) / 2;
            f16* dst = xs + b * ldx;
            gather_raw(kh, ep, wt, [&](int i) -> const uint64_t* { return src + i; },
                       [&](int i, uint32_t p) { *reinterpret_cast<uint32_t*>(dst + 2 * i) = p; });
        }
        stamp_done(14);
        clear_red();
        if (tid < 8) reinterpret_cast<u32x4*>(zero64)[tid] = u32x4{0u, 0u, 0u, 0u};   // (attention reused it)
        gemv_prep(xs - klo, ldx, c64 - ka5 * GEMV_ROWS, nullptr, B, klo, 2 * kh, tid, NTHR);
        __syncthreads();
        const GemvAct xa{xs - klo, ldx, c64 - ka5 * GEMV_ROWS, nullptr, zero64};
        if (run5.ka < run5.kz)
            gemv_run<RING, false, false, MAXB == 1>(a.down, run5, xa, B, R5, q5, [&](int, const float (&out)[4]) { to_red(0, out); });
        stamp_done(15);
        __syncthreads();
        if (s5 > 0) {
            for (int i = tid; i < B * 32; i += NTHR) {
                const int b = i >> 5, cc = i & 31;
                put_tagged(a.down_part + ((size_t)s5 * B + b) * H + t5 * 32 + cc, __float_as_uint(red_sum(0, b, cc)), ep);
            }
        } else {
            for (int i = tid; i < B * 32; i += NTHR) own[i] = red_sum(0, i >> 5, i & 31);
            __syncthreads();
            gather_sum(B * 32, a.S_down - 1, (size_t)B * H, ep, wt,
                       [&](int i) { return a.down_part + ((size_t)1 * B + (i >> 5)) * H + t5 * 32 + (i & 31); },
                       [&](int i, float v) {
                           const int b = i >> 5, col = t5 * 32 + (i & 31);
                           a.y[(size_t)b * H + col] = hbuf[b * H + col] + (own[i] + v);
                       });
        }
    }
    stamp_done(4);
}

template <int D, int MAXB>
LdsLimit& lds_limit() {
    static LdsLimit lim;
    return lim;
}

template <int D, int MAXB>
int launch_t(const DecodeFusedArgs& a, hipStream_t stream) {
    auto fn = decode_fused_kernel<D, MAXB>;
    if (ensure_lds_limit(lds_limit<D, MAXB>(), (const void*)fn, a.lds_bytes)) return -1;
    // An ordinary launch: one block per CU (the LDS of a block leaves room for
    // no second one), so every block is resident once the CUs are free.  A
    // cooperative launch would guarantee the same at about 20 us per launch.
    hipLaunchKernelGGL(fn, dim3(a.nblocks), dim3(NTHR), a.lds_bytes, stream, a);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int decode_fused_max_chunk(int) { return 256; }   // 8 key groups

int decode_fused_blocks(int head_dim, int B, size_t lds_bytes) {
    int dev = 0, cus = 0, occ = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    const void* fn = nullptr;
    LdsLimit* lim = nullptr;
    if (head_dim == 128) {
        fn = B <= 1 ? (const void*)decode_fused_kernel<128, 1> : (const void*)decode_fused_kernel<128, 4>;
        lim = B <= 1 ? &lds_limit<128, 1>() : &lds_limit<128, 4>();
    } else {
        fn = B <= 1 ? (const void*)decode_fused_kernel<64, 1> : (const void*)decode_fused_kernel<64, 4>;
        lim = B <= 1 ? &lds_limit<64, 1>() : &lds_limit<64, 4>();
    }
    if (ensure_lds_limit(*lim, fn, lds_bytes)) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, NTHR, lds_bytes) != hipSuccess) return 0;
    return occ >= 1 ? cus : 0;
}

int launch_decode_fused(const DecodeFusedArgs& a, hipStream_t stream) {
    if (a.B > 4 || a.S_qkv > MAXS || a.S_o > MAXS || a.S_down > MAXS) return -1;
    if (a.S_qkv < 1 || a.S_o < 1 || a.S_down < 1 || a.nblocks < 1) return -1;
    if (a.shared ? (a.ctx_lens != nullptr || a.sb != 0 || a.ctx_base < 0) : a.ctx_lens == nullptr) return -1;
    if (a.slots < 1 || (a.B == 1 && !a.gam_lds)) return -1;
    if (a.chunk < 1 || a.chunk > decode_fused_max_chunk(a.d) || a.nkv < 1 || a.nq % a.nkv || a.nq / a.nkv > MAXR)
        return -1;
    if (a.off_h < decode_fused_attn_bytes(a.chunk, a.d)) return -1;
    if (a.d == 128) return a.B <= 1 ? launch_t<128, 1>(a, stream) : launch_t<128, 4>(a, stream);
    if (a.d == 64) return a.B <= 1 ? launch_t<64, 1>(a, stream) : launch_t<64, 4>(a, stream);
    return -1;
}
