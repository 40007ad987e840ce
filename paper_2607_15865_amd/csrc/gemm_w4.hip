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
// by the scale of the last group of the k range.  (Rounding the scaled weight
// to fp16 instead would save those multiplies, but its 2^-12 relative error
// flips the bf16 rounding of q/k/v and of the SwiGLU output often enough to
// break the parity bound on full-size layers.)
//
// Block: 256 threads = 4 waves side by side along N.  Block tile BM x 256
// with BM = 32 * TM; wave tile BM x 64 (TM x 2 MFMA tiles), so a wave's two
// 32-column weight tiles are a RoPE pair or a gate/up pair and every
// dequantised weight fragment feeds TM MFMAs.
//
// Pipeline, per iteration of BK = 128 k (two 64-k weight tiles per column):
// at its start a block requests everything the next iteration needs, and
// the barrier at its end (whose workgroup release waits for the block's
// outstanding loads) makes it visible:
//   * the X tile (BM x 128 fp16) goes straight from memory to LDS with
//     direct-to-LDS loads (one 1 KB wave load per 4 rows), so it costs no
//     registers; rows are 256 bytes without padding, and the 16-byte chunk c
//     of row r is stored at chunk c ^ (r & 15), so the A-fragment reads of
//     16 consecutive rows hit 16 different bank groups;
//   * each wave loads its 4 weight tiles (1 KB each, one 16-byte load per
//     lane) into the free half of a register ring of 8 tile slots;
//   * inside the iteration the A fragments (LDS) and B fragments of step
//     t + 1 are prepared while the MFMAs of step t run;
//   * the scale ratio that the accumulators take at the end of an iteration
//     (the next iteration's first group) was requested an iteration earlier,
//     so no instruction of an iteration waits for that iteration's loads.
// Every load is issued unconditionally with clamped addresses (X rows past M
// read row M - 1; their outputs are dropped).  K_pad is a multiple of 128, so
// every k range holds whole iterations.
//
// Split K: with S > 1 the k tiles are cut into S ranges, one block each.
// Every block stores its fp32 partial tile, and the last block of a tile to
// arrive (a per-tile counter) adds the S partials in range order and runs
// the epilogue, so the result does not depend on the arrival order.  The
// counters live in the caller's workspace and need no clearing: each is a
// 64-bit word (launch tag << 32 | arrivals), and an arrival that finds
// another launch's tag starts the count afresh.
//
// Block order: the blocks of one column block (its row blocks and k ranges)
// are placed on the same XCD (consecutive block ids go round robin over the
// 8 XCDs), so each weight column block is read from HBM into one L2.
#include "common.h"
#include "launch.h"

namespace {

constexpr int BN = 256;
constexpr int NXCD = 8;

struct GemmShape {
    int M, nrb, ncb, S, KB;
    float* part;                 // [S][M][N_dev] (S > 1)
    unsigned long long* cnt;     // [nrb * ncb] tagged arrival counters (S > 1)
    unsigned tag;                // this launch's tag, unique among launches that share cnt
};

// Instruction order of one k16 step for the scheduler: every MFMA is
// followed by an LDS read of the next step's A fragments (the first TM of
// them) and a few VALU operations (dequantisation of the next step).
template <int TM, int NVALU>
__device__ __forceinline__ void sched_step() {
#pragma unroll
    for (int j = 0; j < 2 * TM; j++) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        if (j < TM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
        __builtin_amdgcn_sched_group_barrier(0x002, NVALU, 0);   // VALU
    }
}

template <int TM>
constexpr size_t lds_bytes() { return (size_t)2 * 32 * TM * 256; }

// k range of split sp in 64-k tiles; inner split points are even so that
// iterations hold whole tile pairs
__host__ __device__ inline void split_range(int sp, int S, int KB, int& lo, int& hi) {
    const int pairs = KB / 2;
    lo = (int)((long long)sp * pairs / S) * 2;
    hi = sp == S - 1 ? KB : (int)((long long)(sp + 1) * pairs / S) * 2;
}

// GT: group size class, 0 = groups of 32 (two per 64-k tile), 1 = groups of
// 64, 2 = groups of 128 or more (starting only at the first tile of an
// iteration); ZP: the linear has zero points; WF: weight format
// (WeightFormat).  The 8- and 16-bit formats differ only in the tile bytes
// (2 or 4 quads of 16 bytes per lane) and the fragment unpack (dequant8_u8,
// f16_frag); their scales (one per column, in groups of 128) ride the same
// ratio scheme (every ratio 1).
template <int EPI, int TM, int GT, bool ZP, int WF>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
gemm_w4_kernel(const f16* __restrict__ X, int ldx, DevLinear W, EpiArgs ep, GemmShape gs) {
    constexpr int BM = 32 * TM;
    constexpr int XL = BM / 16;                         // X direct-to-LDS loads per wave and iteration
    constexpr int NH = GT == 0 ? 2 : 1;                 // group parameters per tile
    constexpr int RS = 8;                               // weight tile slots: two iterations
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    unsigned char* const As0 = smem;
    unsigned char* const As1 = smem + BM * 256;
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
    const bool wave_on = nt0 * 32 < W.N_dev;            // columns past N_dev: the wave computes on
                                                        // tile 0 and stores nothing
    const int KB = gs.KB;
    int kb_lo, kb_hi;
    split_range(sp, gs.S, KB, kb_lo, kb_hi);
    const int nit = (kb_hi - kb_lo + 1) / 2;
    const int Gm1 = (1 << W.lgG) - 1;
    const int col0 = (wave_on ? nt0 : 0) * 32 + c, col1 = col0 + 32;
    const DqConst dq = dq_const();

    // ---- X tile of the iteration that starts at 64-k tile kb, straight to
    // LDS: load i of wave w fills rows 4 (4 i + w) .. + 3; lane L writes
    // chunk L & 15 of row 4 (4 i + w) + L / 16, which holds logical chunk
    // (L & 15) ^ (row & 15).
    const uint32_t xrow_bytes = (uint32_t)ldx * 2u;
    const char* const Xb = reinterpret_cast<const char*>(X);
    // row & 15 = (4 wave + lane / 16) & 15 for every load i, so the logical
    // chunk of this lane is the same in all its loads
    const int xlc = (lane & 15) ^ ((4 * wave + (lane >> 4)) & 15);
    uint32_t xoff[XL];                                  // per load: row offset + chunk (bytes)
#pragma unroll
    for (int i = 0; i < XL; i++) {
        const int r = 4 * (4 * i + wave) + (lane >> 4);
        const int m = m0 + r < M ? m0 + r : M - 1;
        xoff[i] = (uint32_t)m * xrow_bytes + (uint32_t)xlc * 16u;
    }
    // Pipeline depth P: the loads of iteration it + P are requested in
    // iteration it.  Row tiles of 32 and 64 (short iterations) stage X in
    // registers, so the barrier of an iteration waits for LDS writes only and
    // the deeper loads stay in flight; row tiles of 128 load X straight into
    // LDS one iteration ahead (their registers hold the accumulators).
    constexpr bool XREG = TM < 4;
    // (the 8- and 16-bit formats hold 2 or 4 times the weight registers per
    // tile: the shallowest pipeline)
    constexpr int P = WF != WF_INT4 ? 2 : TM == 1 ? 4 : (TM == 2 && GT != 0) ? 3 : 2;
    constexpr int U = P % 2 == 0 ? P : 2 * P;          // unroll: X stage (mod P) and LDS buffer (mod 2) static
    constexpr int XS = XREG ? P : 1;
    u32x4 xr[XS][XL];
    auto xbytes = [&](int kb) __attribute__((always_inline)) {
        return (uint32_t)(kb < kb_hi ? kb : kb_lo) * 128u;
    };
    // DMA variant: the X tile of the iteration that starts at kb into As
    auto load_x_lds = [&](int kb, unsigned char* As) __attribute__((always_inline)) {
        const uint32_t kbytes = xbytes(kb);
#pragma unroll
        for (int i = 0; i < XL; i++)
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(Xb + (xoff[i] + kbytes)),
                                             (__attribute__((address_space(3))) void*)(As + (4 * i + wave) * 1024),
                                             16, 0, 0);
    };
    // register variant: load into stage st, later written to LDS at the place
    // the direct-to-LDS load would fill (lane L: 16 bytes at L * 16)
    auto load_x_reg = [&](int st, int kb) __attribute__((always_inline)) {
        const uint32_t kbytes = xbytes(kb);
#pragma unroll
        for (int i = 0; i < XL; i++)
            xr[XREG ? st : 0][i] = *reinterpret_cast<const u32x4*>(Xb + (xoff[i] + kbytes));
    };
    auto store_x = [&](int st, unsigned char* As) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < XL; i++)
            *reinterpret_cast<u32x4*>(As + (4 * i + wave) * 1024 + lane * 16) = xr[XREG ? st : 0][i];
    };

    // ---- weight ring: group g (slots 4 g .. 4 g + 3) holds the tiles of one
    // iteration, slot 4 g + 2 half + column with the ratios (and zero points)
    // of their groups.  Loads past the range re-read the range's first tile
    // (never used).
    constexpr int NG = XREG ? P : 2;
    constexpr int NQ = 1 << WF;                         // 16-byte quads per lane and tile
    constexpr uint32_t TB = 1024u << WF;                // tile bytes
    const char* const Wb = reinterpret_cast<const char*>(W.qw);
    const uint32_t woff0 = (uint32_t)(wave_on ? nt0 : 0) * (uint32_t)KB * TB + (uint32_t)lane * 16u;
    const uint32_t wcol1 = (uint32_t)KB * TB;
    const char* const Rb = reinterpret_cast<const char*>(W.ratios);
    // FS (INT4, 128-row tiles, SwiGLU and residual epilogues): a weight
    // fragment is multiplied by its group's fp16 scale (4 packed multiplies,
    // which the fragment's 8 MFMAs share) instead of the accumulators by the
    // running ratio at each group boundary (128 multiplies per group); the
    // product (q - z) s is rounded to fp16.  With fewer row tiles a fragment
    // serves fewer MFMAs and the ratio costs less, so those keep it; so does
    // the q/k/v GEMM, whose exact sums decide the bf16 rounding of the
    // cached keys and values.
    constexpr bool FS = WF == WF_INT4 && TM == 4 && EPI != EPI_QKV;
    u32x4 rw[4 * NG][NQ];
    float rr[4 * NG][NH];
    f16 rs[4 * NG][NH];
    uint32_t rz[4 * NG][NH];
    auto load_w = [&](int q, int kb) __attribute__((always_inline)) {
        const int kk = kb < kb_hi ? kb : kb_lo;
        const int col = (q & 1) ? col1 : col0;
#pragma unroll
        for (int j = 0; j < NQ; j++)
            rw[q][j] = *reinterpret_cast<const u32x4*>(Wb + (woff0 + ((q & 1) ? wcol1 : 0u) + (uint32_t)kk * TB + 1024u * j));
#pragma unroll
        for (int hh = 0; hh < NH; hh++) {
            const uint32_t gi = (uint32_t)((kk * 64 + 32 * hh) >> W.lgG) * (uint32_t)W.N_dev + (uint32_t)col;
            if constexpr (FS) rs[q][hh] = __builtin_bit_cast(f16, W.scales[gi]);
            else rr[q][hh] = *reinterpret_cast<const float*>(Rb + gi * 4u);
            if (ZP) rz[q][hh] = (uint32_t)W.zeros[gi];
        }
    };
    // DMA variant: the scale ratio of the first tile of the iteration that
    // starts at kb (both columns), two iterations ahead in a ring of two
    // slots, so the group boundary at the end of an iteration never waits
    // for loads of the same iteration (slot it % 2 holds the ratio of
    // iteration it + 2 from the start of iteration it on).
    float rn[2][2];
    auto load_rn = [&](int slot, int kb) __attribute__((always_inline)) {
        if constexpr (FS) return;
        const int kk = kb < kb_hi ? kb : kb_lo;
        const uint32_t g0 = (uint32_t)((kk * 64) >> W.lgG) * (uint32_t)W.N_dev;
        rn[slot][0] = *reinterpret_cast<const float*>(Rb + (g0 + (uint32_t)col0) * 4u);
        rn[slot][1] = *reinterpret_cast<const float*>(Rb + (g0 + (uint32_t)col1) * 4u);
    };
    auto load_group = [&](int g, int kb) __attribute__((always_inline)) {
        load_w(4 * g, kb);
        load_w(4 * g + 1, kb);
        load_w(4 * g + 2, kb + 1);
        load_w(4 * g + 3, kb + 1);
    };

    f32x16 acc[TM][2];
#pragma unroll
    for (int i = 0; i < TM; i++) { acc[i][0] = f32x16{}; acc[i][1] = f32x16{}; }
    ZeroOff zo0 = zero_off(8.0f), zo1 = zo0;
    // A fragment of row tile i, step s, tile half: logical chunk 8 half + 2 s + h
    // of row 32 i + c, stored at chunk ^ (row & 15) (row & 15 == c & 15)
    const uint32_t arow = (uint32_t)c * 256u;

    // the MFMAs of the iteration that starts at kb, on the X tile in As and
    // weight group qb; qn: the group of the next iteration (its first ratio)
    auto compute = [&](int kb, const unsigned char* As, int qb, int qn) __attribute__((always_inline)) {
        f16x8 a[2][TM], b[2][2];
        auto prep = [&](int t, int p) __attribute__((always_inline)) {
            const int half = t >> 2, s = t & 3, q = qb + 2 * half, hh = NH == 2 ? (s >> 1) : 0;
            if (ZP && (s == 0 || (NH == 2 && s == 2))) {
                zo0 = zero_off((float)rz[q][hh]);
                zo1 = zero_off((float)rz[q + 1][hh]);
            }
            const uint32_t chunk = (uint32_t)((8 * half + 2 * s + h) ^ (c & 15)) * 16u;
#pragma unroll
            for (int i = 0; i < TM; i++)
                a[p][i] = *reinterpret_cast<const f16x8*>(As + (uint32_t)i * 8192u + arow + chunk);
            if constexpr (WF == WF_INT8) {
                b[p][0] = dequant8_u8(rw[q][s >> 1][2 * (s & 1)], rw[q][s >> 1][2 * (s & 1) + 1], zo0.even);
                b[p][1] = dequant8_u8(rw[q + 1][s >> 1][2 * (s & 1)], rw[q + 1][s >> 1][2 * (s & 1) + 1], zo1.even);
            } else if constexpr (WF == WF_F16) {
                b[p][0] = f16_frag(rw[q][s][0], rw[q][s][1], rw[q][s][2], rw[q][s][3]);
                b[p][1] = f16_frag(rw[q + 1][s][0], rw[q + 1][s][1], rw[q + 1][s][2], rw[q + 1][s][3]);
            } else {
                b[p][0] = dequant8(rw[q][0][s], zo0, dq);
                b[p][1] = dequant8(rw[q + 1][0][s], zo1, dq);
                if constexpr (FS) {
                    const f16 s0 = rs[q][hh], s1 = rs[q + 1][hh];
                    b[p][0] = b[p][0] * f16x8{s0, s0, s0, s0, s0, s0, s0, s0};
                    b[p][1] = b[p][1] * f16x8{s1, s1, s1, s1, s1, s1, s1, s1};
                }
            }
        };
        // After step t, if step t + 1 (step 0 of the next iteration for
        // t = 7) starts a group inside the range, the accumulators take
        // its ratio s_prev / s_new.  Doing it here, interleaved with the
        // last MFMAs of the old group, keeps the multiplies off the
        // boundary between the groups' MFMA streams.
        auto next_group = [](int t) { return t == 7 || (GT <= 1 && t == 3) || (GT == 0 && (t & 1) == 1); };
        prep(0, 0);
#pragma unroll
        for (int t = 0; t < 8; t++) {
            const int p = t & 1;
            if (t + 1 < 8) prep(t + 1, p ^ 1);
#pragma unroll
            for (int i = 0; i < TM; i++) {
                acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[p][i], b[p][0], acc[i][0], 0, 0, 0);
                acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[p][i], b[p][1], acc[i][1], 0, 0, 0);
            }
            if (!FS && next_group(t)) {
                const int tn = (t + 1) & 7;                       // the next step
                const int half = tn >> 2, hh = NH == 2 ? ((tn & 3) >> 1) : 0;
                const int q = (t == 7 ? qn : qb) + 2 * half;
                const int k = (kb + (t == 7 ? 2 : 0) + half) * 64 + (tn & 3) * 16;
                const bool start = k < kb_hi * 64 && (k & Gm1) == 0;
                float r0 = rr[q][hh], r1 = rr[q + 1][hh];
                if (!XREG && t == 7) {          // the next iteration's first tile (NH == 1)
                    r0 = rn[(qb >> 2) ^ 1][0];
                    r1 = rn[(qb >> 2) ^ 1][1];
                }
                const float f0 = start ? r0 : 1.0f, f1 = start ? r1 : 1.0f;
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int e = 0; e < 16; e++) {
                        acc[i][0][e] *= f0;
                        acc[i][1][e] *= f1;
                    }
                sched_step<TM, TM == 4 ? 16 : 20>();
            } else {
                sched_step<TM, TM == 4 ? 4 : 6>();
            }
        }
    };

    if constexpr (XREG) {
        // iteration it (u = it mod U): X of it + P into stage u mod P (X of it
        // is in LDS already), the MFMAs of it on LDS buffer u mod 2 and weight
        // group u mod P, then the weights of it + P into that group, X of
        // it + 1 into the other LDS buffer, and the barrier.  Iterations past
        // the range (the loop runs a multiple of U) only load, store and wait.
#pragma unroll
        for (int j = 0; j < P; j++) {
            load_x_reg(j, kb_lo + 2 * j);
            load_group(j, kb_lo + 2 * j);
        }
        store_x(0, As0);
        __syncthreads();
        for (int it0 = 0; it0 < nit; it0 += U) {
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int kb = kb_lo + 2 * (it0 + u);
                const int st = u % P;
                load_x_reg(st, kb + 2 * P);
                if (kb < kb_hi) compute(kb, (u & 1) ? As1 : As0, 4 * st, 4 * ((u + 1) % P));
                load_group(st, kb + 2 * P);
                store_x((u + 1) % P, (u & 1) ? As0 : As1);
                __syncthreads();
            }
        }
    } else {
        // iteration it: X and weights of it + 1 requested (X straight to LDS),
        // the MFMAs of it, then the barrier, whose workgroup release waits for
        // the block's outstanding loads.  With it == nit (the odd partner of
        // the last iteration) only the loads and the barrier run.
        auto iteration = [&](int it, const unsigned char* As, unsigned char* As_next, int qb, int qn)
            __attribute__((always_inline)) {
            const int kb = kb_lo + 2 * it;
            load_rn(qb >> 2, kb + 4);
            load_x_lds(kb + 2, As_next);
            load_group(qn / 4, kb + 2);
            if (kb < kb_hi) compute(kb, As, qb, qn);
            __syncthreads();
        };
        load_x_lds(kb_lo, As0);
        load_group(0, kb_lo);
        load_rn(1, kb_lo + 2);
        __syncthreads();
        for (int it = 0; it < nit; it += 2) {
            iteration(it, As0, As1, 0, 4);
            iteration(it + 1, As1, As0, 4, 0);
        }
    }

    // ---- scale of the range's last group (1 with fragment scales)
    const int glast = ((kb_hi * 64) - 1) >> W.lgG;
    const float sl0 = FS ? 1.0f : (float)__builtin_bit_cast(f16, W.scales[(size_t)glast * W.N_dev + col0]);
    const float sl1 = FS ? 1.0f : (float)__builtin_bit_cast(f16, W.scales[(size_t)glast * W.N_dev + col1]);

    // Epilogue of row tile i: v0[e], v1[e] are the sums of columns col0 and
    // col1 for row m0 + 32 i + 8 (e / 4) + 4 h + e % 4.  Every value the
    // epilogue reads (residual, positions, RoPE factors) is requested for
    // all 16 rows before the first store: a store could alias a later read,
    // so interleaved they would cost a memory round trip per row.
    auto tile_epilogue = [&](int i, const float (&v0)[16], const float (&v1)[16]) __attribute__((always_inline)) {
        int mr[16];
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
            mr[e] = m < M ? m : -1;
        }
        auto row = [&](int e) { return mr[e] < 0 ? M - 1 : mr[e]; };
        if (EPI == EPI_RESID) {
            float r0[16], r1[16];
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const size_t o = (size_t)row(e) * W.N;
                r0[e] = ep.resid[o + col0];
                r1[e] = ep.resid[o + col1];
            }
#pragma unroll
            for (int e = 0; e < 16; e++) {
                if (mr[e] < 0) continue;
                const size_t o = (size_t)mr[e] * W.N;
                ep.out_f32[o + col0] = r0[e] + v0[e];
                ep.out_f32[o + col1] = r1[e] + v1[e];
            }
        } else if (EPI == EPI_SWIGLU) {
            const int f = (nt0 / 2) * 32 + c;          // tile pair (2j, 2j+1) = gate block j, up block j
            bool bad = false;
#pragma unroll
            for (int e = 0; e < 16; e++)
                if (mr[e] >= 0) ep.act_out[(size_t)mr[e] * ep.F_pad + f] = act_f16(silu(v0[e]) * v1[e], bad);
            flag_range(ep.err, bad);
        } else {
            // q/k/v: the column pair (nt0 * 32 + c, + 32) holds dims dim0 and
            // dim1 of one head (see epi_qkv_pair); RoPE on q and k
            const int d = ep.head_dim, qd = ep.nq * d, kd = ep.nkv * d;
            int n = nt0 * 32, kind, head;
            if (n < qd) { kind = 0; head = n / d; n -= head * d; }
            else if (n < qd + kd) { kind = 1; n -= qd; head = n / d; n -= head * d; }
            else { kind = 2; n -= qd + kd; head = n / d; n -= head * d; }
            const int p0 = n / 32;
            const int dim0 = 32 * rope_block(p0, d) + c;
            const int dim1 = 32 * rope_block(p0 + 1, d) + c;
            float cs[16], sn[16];
            if (kind < 2) {
                int ps[16];
#pragma unroll
                for (int e = 0; e < 16; e++) ps[e] = ep.pos[row(e)];
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    cs[e] = ep.rope_cos[(size_t)ps[e] * (d / 2) + dim0];
                    sn[e] = ep.rope_sin[(size_t)ps[e] * (d / 2) + dim0];
                }
            }
#pragma unroll
            for (int e = 0; e < 16; e++) {
                if (mr[e] < 0) continue;
                float o0 = v0[e], o1 = v1[e];
                if (kind < 2) {
                    o0 = v0[e] * cs[e] - v1[e] * sn[e];
                    o1 = v1[e] * cs[e] + v0[e] * sn[e];
                }
                const uint16_t b0 = bf16_bits_rne(o0), b1 = bf16_bits_rne(o1);
                uint16_t* dst;
                if (kind == 0) {
                    dst = ep.q_out + ((size_t)mr[e] * ep.nq + head) * d;
                } else {
                    uint16_t* cache = (kind == 1) ? ep.k_cache : ep.v_cache;
                    dst = cache + (size_t)head * ep.cache_stride_h + (size_t)(ep.slot_base + mr[e]) * d;
                }
                dst[dim0] = b0;
                dst[dim1] = b1;
            }
        }
    };

    if (gs.S == 1) {
        if (!wave_on) return;
#pragma unroll
        for (int i = 0; i < TM; i++) {
            float v0[16], v1[16];
#pragma unroll
            for (int e = 0; e < 16; e++) {
                v0[e] = acc[i][0][e] * sl0;
                v1[e] = acc[i][1][e] * sl1;
            }
            tile_epilogue(i, v0, v1);
        }
        return;
    }

    // ---- split K: store the partial tile; the last block of the tile to
    // arrive adds the S partials in range order and runs the epilogue.  The
    // partials are written and read with device-coherent (relaxed, agent
    // scope) accesses, which go past the non-coherent per-XCD L2, so the
    // count only has to follow their completion: no cache write-back or
    // invalidation is needed.
    float* part = gs.part + (size_t)sp * M * W.N_dev;
    if (wave_on) {
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
                if (m < M) {
                    __hip_atomic_store(part + (size_t)m * W.N_dev + col0, acc[i][0][e] * sl0, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(part + (size_t)m * W.N_dev + col1, acc[i][1][e] * sl1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's partial stores are complete
    __syncthreads();
    if (tid == 0) {
        unsigned long long* cnt = gs.cnt + rb * gs.ncb + cb;
        unsigned long long v = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), nv;
        do {
            nv = (unsigned)(v >> 32) == gs.tag ? v + 1 : ((unsigned long long)gs.tag << 32 | 1u);
        } while (!__hip_atomic_compare_exchange_weak(cnt, &v, nv, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT));
        last_flag = ((unsigned)nv == (unsigned)gs.S);
    }
    __syncthreads();
    if (!last_flag || !wave_on) return;
    // The sum, row tile by row tile: the 32 values of a range are requested
    // together (one memory round trip per range), rows past M read row M - 1
    // and are dropped.
#pragma unroll
    for (int i = 0; i < TM; i++) {
        float t0[16], t1[16];
#pragma unroll
        for (int e = 0; e < 16; e++) { t0[e] = 0.f; t1[e] = 0.f; }
        for (int s = 0; s < gs.S; s++) {
            if (s == sp) {
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    t0[e] += acc[i][0][e] * sl0;
                    t1[e] += acc[i][1][e] * sl1;
                }
            } else {
                const float* ps = gs.part + (size_t)s * M * W.N_dev;
                float v0[16], v1[16];
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const int m = m0 + i * 32 + 8 * (e / 4) + 4 * h + (e % 4);
                    const size_t ro = (size_t)(m < M ? m : M - 1) * W.N_dev;
                    v0[e] = __hip_atomic_load(ps + ro + col0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    v1[e] = __hip_atomic_load(ps + ro + col1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    t0[e] += v0[e];
                    t1[e] += v1[e];
                }
            }
        }
        tile_epilogue(i, t0, t1);
    }
}

template <int EPI, int TM, int GT, bool ZP, int WF = WF_INT4>
int launch_v(const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmShape& gs, hipStream_t stream) {
    const int blocks = gs.nrb * gs.ncb * gs.S;
    const size_t lds = lds_bytes<TM>();
    static LdsLimit lim;
    if (ensure_lds_limit(lim, (const void*)gemm_w4_kernel<EPI, TM, GT, ZP, WF>, lds)) return -1;
    hipLaunchKernelGGL((gemm_w4_kernel<EPI, TM, GT, ZP, WF>), dim3(blocks), dim3(256), lds, stream, X, ldx, W, ep, gs);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// row tiles of 128 only for groups of 64 or more without zero points; the
// other variants use at most 64
template <int EPI>
int launch_epi(int TM, const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmShape& gs,
               hipStream_t stream) {
    const bool zp = W.zeros != nullptr;
    const int gt = W.lgG == 5 ? 0 : W.lgG == 6 ? 1 : 2;
    // 8-bit: zero points, groups of 128 (row tiles of 32 or 64); 16-bit: neither
    // (row tiles of 32)
    if (W.wf == WF_INT8) {
        if (!zp || gt != 2 || TM == 4) return -1;
        return TM == 2 ? launch_v<EPI, 2, 2, true, WF_INT8>(X, ldx, W, ep, gs, stream)
                       : launch_v<EPI, 1, 2, true, WF_INT8>(X, ldx, W, ep, gs, stream);
    }
    if (W.wf == WF_F16) {
        if (zp || gt != 2 || TM != 1) return -1;
        return launch_v<EPI, 1, 2, false, WF_F16>(X, ldx, W, ep, gs, stream);
    }
    if (!zp && gt == 2) {
        if (TM == 4) return launch_v<EPI, 4, 2, false>(X, ldx, W, ep, gs, stream);
        if (TM == 2) return launch_v<EPI, 2, 2, false>(X, ldx, W, ep, gs, stream);
        return launch_v<EPI, 1, 2, false>(X, ldx, W, ep, gs, stream);
    }
    if (!zp && gt == 1) {
        if (TM == 4) return launch_v<EPI, 4, 1, false>(X, ldx, W, ep, gs, stream);
        if (TM == 2) return launch_v<EPI, 2, 1, false>(X, ldx, W, ep, gs, stream);
        return launch_v<EPI, 1, 1, false>(X, ldx, W, ep, gs, stream);
    }
    if (TM == 4) return -1;
    if (zp) {
        if (gt == 0) return TM == 2 ? launch_v<EPI, 2, 0, true>(X, ldx, W, ep, gs, stream)
                                    : launch_v<EPI, 1, 0, true>(X, ldx, W, ep, gs, stream);
        if (gt == 1) return TM == 2 ? launch_v<EPI, 2, 1, true>(X, ldx, W, ep, gs, stream)
                                    : launch_v<EPI, 1, 1, true>(X, ldx, W, ep, gs, stream);
        return TM == 2 ? launch_v<EPI, 2, 2, true>(X, ldx, W, ep, gs, stream)
                       : launch_v<EPI, 1, 2, true>(X, ldx, W, ep, gs, stream);
    }
    return TM == 2 ? launch_v<EPI, 2, 0, false>(X, ldx, W, ep, gs, stream)
                   : launch_v<EPI, 1, 0, false>(X, ldx, W, ep, gs, stream);
}

}  // namespace

// Launch plan.  The row tile is the largest (most MFMAs per dequantised
// fragment) that still gives 0.75 tiles per CU; k splits then raise the grid
// to 0.75 blocks per CU, or, while splits stay long (6144 k or more), up to
// 1.2 blocks per CU.  Each split keeps at least 4 iterations.  (The
// thresholds follow a measured sweep over the prefill shapes of the
// Llama-3-8B-shaped layer at 128 and 512 rows.)
GemmPlan gemm_w4_plan(int M, const DevLinear& W, int num_cus) {
    GemmPlan p;
    const int ncb = (W.N_dev + BN - 1) / BN, KB = W.K_pad / 64;
    // the kernel variants that exist (the 16-bit format's weight registers
    // leave room for row tiles of 32 only)
    const int tm_max = W.wf == WF_F16 ? 1 : (W.zeros || W.lgG == 5 || W.wf != WF_INT4) ? 2 : 4;
    auto nrb = [&](int tm) { return (M + 32 * tm - 1) / (32 * tm); };
    p.TM = tm_max;
    // (a k range of 12288 or more also takes a row tile with 0.375 tiles per
    // CU: two k splits then fill the CUs, and each dequantised fragment feeds
    // twice the MFMAs -- the 512 x 4096 x 14336 down GEMM: 80 -> 76 us)
    const int tile_need = KB * 64 >= 4 * 3072 ? num_cus * 3 / 2 : num_cus * 3;
    while (p.TM > 1 && nrb(p.TM) * ncb * 4 < tile_need) p.TM /= 2;
    const int tiles = nrb(p.TM) * ncb;
    p.S = 1;
    while (p.S < 16 && KB / (p.S * 2) >= 8) {
        const int blocks = tiles * p.S;
        const bool small = blocks * 4 < num_cus * 3;
        const bool long_k = KB * 64 / p.S >= 2 * 3072 && blocks * 5 < num_cus * 6;
        if (!small && !long_k) break;
        p.S *= 2;
    }
    p.nrb = nrb(p.TM);
    p.ncb = ncb;
    p.part_bytes = p.S > 1 ? (size_t)p.S * M * W.N_dev * 4 : 0;
    p.tiles = tiles;
    return p;
}

int launch_gemm_w4(int epi, const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmPlan& p,
                   int M, float* part, unsigned long long* cnt, unsigned tag, hipStream_t stream) {
    if (p.S > 1 && (!part || !cnt)) return -1;
    GemmShape gs{M, p.nrb, p.ncb, p.S, W.K_pad / 64, part, cnt, tag};
    switch (epi) {
        case EPI_QKV: return launch_epi<EPI_QKV>(p.TM, X, ldx, W, ep, gs, stream);
        case EPI_RESID: return launch_epi<EPI_RESID>(p.TM, X, ldx, W, ep, gs, stream);
        case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(p.TM, X, ldx, W, ep, gs, stream);
        default: return -1;
    }
}
