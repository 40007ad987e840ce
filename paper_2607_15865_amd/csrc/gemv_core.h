// Decode GEMV core: one wave's walk over a run of weight tiles, for B <= 8
// activation rows (the decode batch).
//
// A run is the set of tiles (t, kb) with column tile t in [t0, t1) and k-tile
// kb in [ka, kz), walked column by column.  The wave streams the tiles
// through a ring of D register slots: a slot is refilled as soon as its
// tile has been dequantised, so D tiles (D KB per wave) stay in flight.  All
// run bookkeeping is wave-uniform (scalar registers) and kept as byte and
// element offsets that are advanced, not recomputed, per tile.
//
// Arithmetic per tile: the four weight words of a lane are turned into exact
// fp16 (code - zero) values (dequant8) and multiplied on the 32x32x16 fp16
// MFMA with the activation rows (bf16 values held as fp16, read from LDS):
// A = activations (row l % 32 of lane l, clamped to the last real row),
// B = weights (the tile's lane layout is the MFMA B fragment).  Rows 0..7 of
// the product sit in accumulator registers 0..3 (row 4h + r in lane half h);
// the other registers carry rows nobody reads.  Each tile's product (each
// half tile with groups of 32) starts from zero, is multiplied by its group
// scale in fp32 and added to the output.
//
// Group parameters: the raw fp16 scale bits (or scale | zero << 16 when the
// linear has zero points, ZP) of the group of k 0..31 of a tile, and with
// groups of 32 (G32) also of k 32..63, travel with the tile in the ring.
#pragma once
#include "common.h"

template <int D, bool G32>
struct TileRing {
    u32x4 w[D];
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
    uint32_t woff;     // ((t * KBf + kb) * 1024)
    uint32_t grow;     // (kb * 64 >> lgG) * N_dev
    uint32_t gcol;     // t * 32
    int kb;

    __device__ __forceinline__ void start(const DevLinear& W, const Run& run) {
        const int KBf = W.K_pad >> 6;
        woff = (uint32_t)(run.t0 * KBf + run.ka) << 10;
        grow = (uint32_t)((run.ka * 64) >> W.lgG) * (uint32_t)W.N_dev;
        gcol = (uint32_t)run.t0 * 32u;
        kb = run.ka;
    }
    // next tile of the run (past the end the cursor runs on harmlessly)
    __device__ __forceinline__ void next(const DevLinear& W, const Run& run) {
        const int KBf = W.K_pad >> 6;
        kb++;
        woff += 1024u;
        if (((kb * 64) & ((1 << W.lgG) - 1)) == 0) grow += (uint32_t)W.N_dev;
        if (kb == run.kz) {
            kb = run.ka;
            woff += (uint32_t)(KBf - (run.kz - run.ka)) << 10;
            grow = (uint32_t)((run.ka * 64) >> W.lgG) * (uint32_t)W.N_dev;
            gcol += 32u;
        }
    }
};

// Load the tile at cursor q into slot u.
template <int D, bool ZP, bool G32>
__device__ __forceinline__ void ring_load(const DevLinear& W, TileRing<D, G32>& R, int u, const RunCursor& q) {
    const int lane = threadIdx.x & 63;
    const uint32_t lo = (uint32_t)lane * 16u;
    R.w[u] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(W.qw) + (q.woff + lo));
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
template <int D, bool ZP, bool G32>
__device__ __forceinline__ void ring_prefetch(const DevLinear& W, const Run& run, TileRing<D, G32>& R, RunCursor& q) {
    const int n = run.size();
    RunCursor first;
    first.start(W, run);
    q = first;
#pragma unroll
    for (int u = 0; u < D; u++) {
        ring_load<D, ZP, G32>(W, R, u, u < n ? q : first);
        q.next(W, run);
    }
}

template <bool ZP>
__device__ __forceinline__ float take_gparam(uint32_t v, ZeroOff& zo) {
    if (ZP) zo = zero_off((float)((v >> 16) & 0xFFu));
    return (float)__builtin_bit_cast(f16, (uint16_t)(v & 0xFFFFu));
}

// Walk a run whose first D tiles are in R (ring_prefetch, which also set the
// load cursor q).  xs: activation rows in LDS, row b at xs + b * ldx, indexed
// by the absolute k of the linear.  For every column tile t of the run,
// emit(t, out) is called once (wave-uniformly) with out[r] = the run's
// partial sum over its k-tiles for row 4 * (lane / 32) + r and column
// 32 t + lane % 32.
//
// The walk is rounded up to a multiple of D tiles; the steps past the end do
// no arithmetic, but every step refills its slot (past the end with the
// run's first tile) so that no load sits under a branch.
template <int D, bool ZP, bool G32, typename Emit>
__device__ __forceinline__ void gemv_run(const DevLinear& W, const Run& run, const f16* xs, int ldx, int B,
                                         TileRing<D, G32>& R, RunCursor& q, Emit&& emit) {
    const int lane = threadIdx.x & 63, h = lane >> 5, c = lane & 31;
    const DqConst dq = dq_const();
    const int row = c < B ? c : B - 1;
    const f16* xrow = xs + row * ldx + h * 8;
    const int n = run.size();
    RunCursor first;
    first.start(W, run);
    int pt = run.t0, pkb = run.ka;                        // tile being processed
    float out[4] = {0.f, 0.f, 0.f, 0.f};
    const f32x16 zero = {};
    for (int base = 0; base < n; base += D) {
#pragma unroll
        for (int u = 0; u < D; u++) {
            if (base + u < n) {                           // wave-uniform
                ZeroOff zo = zero_off(8.0f), zo_hi = zo;
                const float sa = take_gparam<ZP>(R.sa[u], zo);
                float sb = sa;
                if (G32) sb = take_gparam<ZP>(R.sb[G32 ? u : 0], zo_hi);
                else zo_hi = zo;
                const f16x8 b0 = dequant8(R.w[u][0], zo, dq), b1 = dequant8(R.w[u][1], zo, dq);
                const f16x8 b2 = dequant8(R.w[u][2], zo_hi, dq), b3 = dequant8(R.w[u][3], zo_hi, dq);
                const f16* xk = xrow + pkb * 64;
                f32x16 acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const f16x8*>(xk), b0, zero, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const f16x8*>(xk + 16), b1, acc, 0, 0, 0);
                if (G32) {
#pragma unroll
                    for (int r = 0; r < 4; r++) out[r] = __builtin_fmaf(sa, acc[r], out[r]);
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const f16x8*>(xk + 32), b2, zero, 0, 0, 0);
                } else {
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const f16x8*>(xk + 32), b2, acc, 0, 0, 0);
                }
                acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const f16x8*>(xk + 48), b3, acc, 0, 0, 0);
#pragma unroll
                for (int r = 0; r < 4; r++) out[r] = __builtin_fmaf(sb, acc[r], out[r]);
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
            ring_load<D, ZP, G32>(W, R, u, base + u + D < n ? q : first);
            q.next(W, run);
        }
    }
}
