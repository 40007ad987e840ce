// Decode GEMV core: one wave's walk over a run of weight tiles, for B <= 8
// activation rows (the decode batch).
//
// A run is the set of tiles (t, kb) with column tile t in [t0, t1) and k-tile
// kb in [ka, kz), walked column by column.  The wave streams the tiles
// through a ring of D register slots: a slot is refilled as soon as its
// tile has been consumed, so D tiles (D KB per wave) stay in flight.  All
// run bookkeeping is wave-uniform (scalar registers) and kept as byte and
// element offsets that are advanced, not recomputed, per tile.
//
// Arithmetic per tile.  The four weight words of a lane are not brought to
// (code - zero): each code pair becomes the fp16 pair it makes when OR-ed
// into 0x6400 (dequant8_raw, five bit operations per word), which is
// 1024 + q for the codes in bits 0..3 of a byte and 1024 + 16 q for the codes
// in bits 4..7.  The activations are prepared to match (gemv_prep): the
// elements at k % 8 in {2, 3, 6, 7} (the bits 4..7 codes) are divided by 16,
// and per row and 32-k segment the sums E (other elements) and O (divided
// elements) are kept.  The product over a segment is then
//     sum x'(raw) = sum x (q - z) + 1024 (E + O) + z (E + 16 O),
// so one subtraction per output recovers the exact-weight sum.
//
// The product runs on the 16x16x32 fp16 MFMA with the 32-column tile as is:
// lane l of the B operand is the lane's word s (column 32 t + l % 32,
// k = 16 s + 8 (l / 32) + 0..7), which the MFMA takes as k block l / 16 and
// column l % 16.  The column's high bit (l / 16) % 2 thus sits in the k
// block, and the A operand separates it again: MFMA row m stands for batch
// row b = 4 (m / 8) + m % 4 and column half c = (m / 4) % 2, and lane l
// supplies x'[b] only where c equals its own column half (zeros elsewhere).
// Output register r of lane l is then batch row 4 (l / 32) + r, column
// 32 t + l % 32: the lane's own column, so the lane's own group scale
// applies.  Four 16-cycle MFMAs per tile instead of four 32-cycle ones.
//
// Group parameters: the raw fp16 scale bits (or scale | zero << 16 when the
// linear has zero points, ZP) of the group of k 0..31 of a tile, and with
// groups of 32 (G32) also of k 32..63, travel with the tile in the ring.
#pragma once
#include "common.h"

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// fp16 pairs (1024 + q) / (1024 + 16 q) of the eight codes of a word, in k
// order (pairs at bits 4p and 16 + 4p): five bit operations.
__device__ __forceinline__ f16x8 dequant8_raw(uint32_t w, const DqConst& k) {
    const uint32_t w8 = w >> 8;
    u32x4 r;
    r[0] = (w & k.lo) | k.magic;
    r[1] = (w & k.hi) | k.magic;
    r[2] = (w8 & k.lo) | k.magic;
    r[3] = (w8 & k.hi) | k.magic;
    return __builtin_bit_cast(f16x8, r);
}

// INT8 fragment for the GEMV: fp16 pairs 1024 + q at k % 8 in {0, 1, 4, 5}
// and 16 (1024 + q) at {2, 3, 6, 7} (0x64 | q and 0x74 | q), from the codes
// of bytes lo[0..3], hi[0..3] in k order: four v_perm.
__device__ __forceinline__ f16x8 dequant8_u8_raw(uint32_t lo, uint32_t hi) {
    const uint32_t m = 0x74746464u;
    u32x4 r;
    r[0] = __builtin_amdgcn_perm(m, lo, 0x04010400u);
    r[1] = __builtin_amdgcn_perm(m, lo, 0x06030602u);
    r[2] = __builtin_amdgcn_perm(m, hi, 0x04010400u);
    r[3] = __builtin_amdgcn_perm(m, hi, 0x06030602u);
    return __builtin_bit_cast(f16x8, r);
}

constexpr int GEMV_ROWS = 8;     // row stride of the correction tables

// Activation rows prepared by gemv_prep, all indexed by the absolute k of the
// linear (the pointers are offset by the first k of the range held):
//   xs[b * ldx + k]                       x' (fp16), rows b < B;
//   c64[(k / 64) * GEMV_ROWS + b]         1024 (E + O) + 8 (E + 16 O) over the
//                                         64-k tile (the correction for z = 8);
//   uv32[(k / 32) * GEMV_ROWS + b]        (E + O, E + 16 O) over the 32-k
//                                         segment (any zero point); may be
//                                         null when only z = 8 with groups of
//                                         64 or more is used;
//   zero                                  64 zero fp16 (the A operand of the
//                                         lanes whose column half does not
//                                         match).
struct GemvAct {
    const f16* xs;
    int ldx;
    const float* c64;
    const float2* uv32;
    const f16* zero;
};

// Correction table entries from the sums e (other elements) and o (divided
// elements) of x' over a 64-k tile: the correction for the zero point 8.
__device__ __forceinline__ float gemv_c64(float e, float o) {
    return 1024.0f * (e + o) + 8.0f * (e + 16.0f * o);
}

// Prepare rows b < B, absolute k in [k0, k0 + klen) (klen a multiple of 64)
// in place: x (bf16 values held as fp16) -> x', and write the correction
// tables (pointers as in GemvAct, non-const).  One 8-element chunk per thread
// and pass; the 8 chunks of a 64-k tile sit in 8 adjacent lanes, which meet
// with DPP row operations.  Called by all nthr threads of the block (nthr a
// multiple of 64); the caller synchronises before and after.
__device__ __forceinline__ void gemv_prep(f16* xs, int ldx, float* c64, float2* uv32, int B, int k0, int klen,
                                          int tid, int nthr) {
    const int nc = klen >> 3, total = B * nc;
    const f16x2 sixteenth = f16x2{(f16)0.0625f, (f16)0.0625f};
    for (int base = 0; base < total; base += nthr) {       // uniform passes
        const int i = base + tid;
        const bool ok = i < total;
        const int b = ok ? i / nc : 0, c = ok ? i - b * nc : 0;
        const int k = k0 + 8 * c;
        float e = 0.f, o = 0.f;
        if (ok) {
            u32x4* p = reinterpret_cast<u32x4*>(xs + b * ldx + k);
            const u32x4 w = *p;
            // element pairs (0,1) (2,3) (4,5) (6,7); the words are taken into
            // scalars first (see as_bf16x2)
            const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3];
            const f16x2 x0 = __builtin_bit_cast(f16x2, w0), x2 = __builtin_bit_cast(f16x2, w2);
            const f16x2 x1 = __builtin_bit_cast(f16x2, w1) * sixteenth;
            const f16x2 x3 = __builtin_bit_cast(f16x2, w3) * sixteenth;
            e = ((float)x0[0] + (float)x0[1]) + ((float)x2[0] + (float)x2[1]);
            o = ((float)x1[0] + (float)x1[1]) + ((float)x3[0] + (float)x3[1]);
            *p = u32x4{w0, __builtin_bit_cast(uint32_t, x1), w2, __builtin_bit_cast(uint32_t, x3)};
        }
        // sums over the 4 chunks of a 32-k segment, then the 8 of a 64-k tile
        e += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(e), 0xB1, 0xF, 0xF, false));
        o += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(o), 0xB1, 0xF, 0xF, false));
        e += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(e), 0x4E, 0xF, 0xF, false));
        o += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(o), 0x4E, 0xF, 0xF, false));
        if (uv32 && ok && (c & 3) == 0) uv32[(k >> 5) * GEMV_ROWS + b] = float2{e + o, e + 16.0f * o};
        e += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(e), 0x141, 0xF, 0xF, false));
        o += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(o), 0x141, 0xF, 0xF, false));
        if (ok && (c & 7) == 0) c64[(k >> 6) * GEMV_ROWS + b] = gemv_c64(e, o);
    }
}

// D tiles of a lane: quad j of tile slot u in w[u][j] (1, 2 or 4 quads
// for the 4-, 8- and 16-bit formats).
template <int D, bool G32, int WF = WF_INT4>
struct TileRing {
    u32x4 w[D][1 << WF];
    uint32_t sa[D];
    uint32_t sb[G32 ? D : 1];
};

struct Run {
    int t0, t1, ka, kz;
    __device__ int size() const { return (t1 - t0) * (kz - ka); }
};

// Wave-uniform position in a run: the tile's byte offset in the tile array,
// the element offset of its group parameters (group row + column), and kb.
struct RunCursor {
    uint32_t woff;     // ((t * KBf + kb) * tile bytes (1024 << wf))
    uint32_t grow;     // (kb * 64 >> lgG) * N_dev
    uint32_t gcol;     // t * 32
    int kb;

    __device__ __forceinline__ void start(const DevLinear& W, const Run& run) {
        const int KBf = W.K_pad >> 6;
        woff = (uint32_t)(run.t0 * KBf + run.ka) << (10 + W.wf);
        grow = (uint32_t)((run.ka * 64) >> W.lgG) * (uint32_t)W.N_dev;
        gcol = (uint32_t)run.t0 * 32u;
        kb = run.ka;
    }
    // next tile of the run (past the end the cursor runs on harmlessly)
    __device__ __forceinline__ void next(const DevLinear& W, const Run& run) {
        const int KBf = W.K_pad >> 6;
        kb++;
        woff += 1024u << W.wf;
        if (W.lgG < 6) grow += (uint32_t)W.N_dev << (6 - W.lgG);   // groups of 32: two per tile
        else if (((kb * 64) & ((1 << W.lgG) - 1)) == 0) grow += (uint32_t)W.N_dev;
        if (kb == run.kz) {
            kb = run.ka;
            woff += (uint32_t)(KBf - (run.kz - run.ka)) << (10 + W.wf);
            grow = (uint32_t)((run.ka * 64) >> W.lgG) * (uint32_t)W.N_dev;
            gcol += 32u;
        }
    }
};

// Load the tile at cursor q into slot u.
template <int D, bool ZP, bool G32, int WF = WF_INT4>
__device__ __forceinline__ void ring_load(const DevLinear& W, TileRing<D, G32, WF>& R, int u, const RunCursor& q) {
    const int lane = threadIdx.x & 63;
    const uint32_t lo = (uint32_t)lane * 16u;
#pragma unroll
    for (int j = 0; j < (1 << WF); j++)
        R.w[u][j] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(W.qw) + (q.woff + 1024u * j + lo));
    const uint32_t gi = q.grow + q.gcol + (uint32_t)(lane & 31);
    if (ZP) R.sa[u] = W.sz[gi];
    else R.sa[u] = W.scales[gi];
    if (G32) {   // the k 32..63 half starts a new group
        const uint32_t gj = gi + (uint32_t)W.N_dev;
        if (ZP) R.sb[G32 ? u : 0] = W.sz[gj];
        else R.sb[G32 ? u : 0] = W.scales[gj];
    }
}

// Fill the ring with the first D tiles of the run; the cursor q is left at
// tile D.  Weights do not depend on the activations, so this may run before
// the activations are ready.  Slots past the end of the run load the run's
// first tile again (a cache hit): ring slots are written unconditionally, so
// no slot value has to be merged across branches (that would force a wait
// for the load).
template <int D, bool ZP, bool G32, int WF = WF_INT4>
__device__ __forceinline__ void ring_prefetch(const DevLinear& W, const Run& run, TileRing<D, G32, WF>& R,
                                              RunCursor& q) {
    const int n = run.size();
    RunCursor first;
    first.start(W, run);
    q = first;
#pragma unroll
    for (int u = 0; u < D; u++) {
        ring_load<D, ZP, G32, WF>(W, R, u, u < n ? q : first);
        q.next(W, run);
    }
}

// Group scale (fp16 bits in the low half) and zero point of a group word.
__device__ __forceinline__ float gscale(uint32_t v) {
    return (float)__builtin_bit_cast(f16, (uint16_t)(v & 0xFFFFu));
}
template <bool ZP>
__device__ __forceinline__ float gzero(uint32_t v) {
    return ZP ? (float)((v >> 16) & 0xFFu) : 8.0f;
}

// Walk a run whose first D tiles are in R (ring_prefetch, which also set the
// load cursor q), on activation rows prepared by gemv_prep.  For every column
// tile t of the run, emit(t, out) is called once (wave-uniformly) with
// out[r] = the run's partial sum over its k-tiles for row 4 * (lane / 32) + r
// and column 32 t + lane % 32 (rows >= B hold no meaningful value).
//
// The walk is rounded up to a multiple of D tiles; the steps past the end do
// no arithmetic, but every step refills its slot (past the end with the
// run's first tile) so that no load sits under a branch.  With DRAIN (the
// persistent decode) no tile past the end is requested and the run returns
// with all its loads complete.  A wave's memory counter counts loads and
// stores together, in issue order, so a load still in flight when the wave
// stores its results would make any later wait that covers it (the wait
// before the ring's registers are reused) also wait for those stores to
// complete.
//
// The 8- and 16-bit formats (WF) take the same activations x'.  INT8: the B
// fragment pairs are 0x64 | code = 1024 + q at k % 8 in {0, 1, 4, 5} and
// 0x74 | code = 16 (1024 + q) at the divided elements, so the product over
// a 64-k tile is sum x (1024 + q) = sum x (q - z) + (1024 + z) S with S the
// tile's sum of x (E + 16 O over its two 32-k segments): one correction per
// output with the column's zero point.  F16: the divided elements' weights
// are held times 16, so the product is the exact-weight sum (scale 1).
template <int D, bool ZP, bool G32, bool DRAIN = false, typename Emit, int WF = WF_INT4>
__device__ __forceinline__ void gemv_run(const DevLinear& W, const Run& run, const GemvAct& xa, int B,
                                         TileRing<D, G32, WF>& R, RunCursor& q, Emit&& emit) {
    const int lane = threadIdx.x & 63, h = lane >> 5;
    const DqConst dq = dq_const();
    // A operand of this lane: MFMA row m = lane % 16 (batch row bm, column
    // half cm), k block lane / 16 (column half c1, k half h)
    const int m = lane & 15, cm = (m >> 2) & 1, bm = 4 * (m >> 3) + (m & 3), c1 = (lane >> 4) & 1;
    const bool valid = cm == c1 && bm < B;
    const f16* abase = valid ? xa.xs + bm * xa.ldx + 8 * h : xa.zero + 8 * h;
    const int astride = valid ? 64 : 0;
    const int n = run.size();
    RunCursor first;
    first.start(W, run);
    int pt = run.t0, pkb = run.ka;                        // tile being processed
    float out[4] = {0.f, 0.f, 0.f, 0.f};
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    for (int base = 0; base < n; base += D) {
#pragma unroll
        for (int u = 0; u < D; u++) {
            if (base + u < n) {                           // wave-uniform
                const f16* xk = abase + pkb * astride;
                const f16x8 a0 = *reinterpret_cast<const f16x8*>(xk);
                const f16x8 a1 = *reinterpret_cast<const f16x8*>(xk + 16);
                const f16x8 a2 = *reinterpret_cast<const f16x8*>(xk + 32);
                const f16x8 a3 = *reinterpret_cast<const f16x8*>(xk + 48);
                const float sa = gscale(R.sa[u]);
                if constexpr (WF == WF_INT8) {
                    f32x4_t acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, dequant8_u8_raw(R.w[u][0][0], R.w[u][0][1]), zero, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, dequant8_u8_raw(R.w[u][0][2], R.w[u][0][3]), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a2, dequant8_u8_raw(R.w[u][1][0], R.w[u][1][1]), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a3, dequant8_u8_raw(R.w[u][1][2], R.w[u][1][3]), acc, 0, 0, 0);
                    const float zc = 1024.0f + gzero<true>(R.sa[u]);
                    const float2* uv = xa.uv32 + (2 * pkb) * GEMV_ROWS + 4 * h;
                    const float2* uw = uv + GEMV_ROWS;
#pragma unroll
                    for (int r = 0; r < 4; r++) out[r] = __builtin_fmaf(sa, acc[r] - zc * (uv[r].y + uw[r].y), out[r]);
                } else if constexpr (WF == WF_F16) {
                    f32x4_t acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, __builtin_bit_cast(f16x8, R.w[u][0]), zero, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, __builtin_bit_cast(f16x8, R.w[u][1]), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a2, __builtin_bit_cast(f16x8, R.w[u][2]), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a3, __builtin_bit_cast(f16x8, R.w[u][3]), acc, 0, 0, 0);
#pragma unroll
                    for (int r = 0; r < 4; r++) out[r] += acc[r];
                } else {
                f32x4_t acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, dequant8_raw(R.w[u][0][0], dq), zero, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, dequant8_raw(R.w[u][0][1], dq), acc, 0, 0, 0);
                if (G32) {
                    // k 0..31 and k 32..63 are two groups
                    const float za = gzero<ZP>(R.sa[u]);
                    const float sb = gscale(R.sb[G32 ? u : 0]), zb = gzero<ZP>(R.sb[G32 ? u : 0]);
                    const float2* uv = xa.uv32 + (2 * pkb) * GEMV_ROWS + 4 * h;
#pragma unroll
                    for (int r = 0; r < 4; r++)
                        out[r] = __builtin_fmaf(sa, acc[r] - __builtin_fmaf(za, uv[r].y, 1024.0f * uv[r].x), out[r]);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a2, dequant8_raw(R.w[u][0][2], dq), zero, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a3, dequant8_raw(R.w[u][0][3], dq), acc, 0, 0, 0);
                    const float2* uw = uv + GEMV_ROWS;
#pragma unroll
                    for (int r = 0; r < 4; r++)
                        out[r] = __builtin_fmaf(sb, acc[r] - __builtin_fmaf(zb, uw[r].y, 1024.0f * uw[r].x), out[r]);
                } else {
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a2, dequant8_raw(R.w[u][0][2], dq), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a3, dequant8_raw(R.w[u][0][3], dq), acc, 0, 0, 0);
                    if (ZP) {
                        const float za = gzero<ZP>(R.sa[u]);
                        const float2* uv = xa.uv32 + (2 * pkb) * GEMV_ROWS + 4 * h;
                        const float2* uw = uv + GEMV_ROWS;
#pragma unroll
                        for (int r = 0; r < 4; r++) {
                            const float cr = __builtin_fmaf(za, uv[r].y + uw[r].y, 1024.0f * (uv[r].x + uw[r].x));
                            out[r] = __builtin_fmaf(sa, acc[r] - cr, out[r]);
                        }
                    } else {
                        const f32x4_t cc = *reinterpret_cast<const f32x4_t*>(xa.c64 + pkb * GEMV_ROWS + 4 * h);
#pragma unroll
                        for (int r = 0; r < 4; r++) out[r] = __builtin_fmaf(sa, acc[r] - cc[r], out[r]);
                    }
                }
                }
                if (pkb == run.kz - 1) {
                    emit(pt, out);
#pragma unroll
                    for (int r = 0; r < 4; r++) out[r] = 0.f;
                    pkb = run.ka;
                    pt++;
                } else {
                    pkb++;
                }
            }
            // refill the slot with tile base + u + D (or the first tile)
            if constexpr (DRAIN) {
                if (base + u + D < n) ring_load<D, ZP, G32, WF>(W, R, u, q);
            } else {
                ring_load<D, ZP, G32, WF>(W, R, u, base + u + D < n ? q : first);
            }
            q.next(W, run);
        }
    }
    if constexpr (DRAIN) __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
}
