// Decode stage in one persistent launch (one block of 8 waves per CU).
// Deterministic: every column sum is formed from per-wave partials added in a
// fixed order, no floating-point atomics.
//
// The decode step is a chain of five dependent phases (Sec. 4.4):
//   P1  q/k/v GEMV on RMSNorm(x)      -> RoPE, bf16, new K/V into the cache
//   P2  split-KV attention            -> attention output A
//   P3  o_proj GEMV                   -> h = x + A Wo
//   P4  gate/up GEMV on RMSNorm(h)    -> g = silu(gate) * up
//   P5  down GEMV                     -> y = h + g Wd
// Separate kernels pay a launch boundary (~2.3 us) per phase and run each
// phase on a partly idle machine; here the blocks stay resident and meet at
// grid barriers (~1.6 us, fence-free tree).  Every GEMV phase splits the
// layer's 1 KB weight tiles evenly over all waves (each wave a contiguous run
// of tiles in column-major order), so no phase has a tail of idle CUs.
// Epilogues that need a column's complete sum (RoPE, SwiGLU) are run by the
// wave that contributes the last partial of a column pair (or column tile
// for the residual epilogues); the attention
// combine of a kv group by the block that finishes its last chunk.
//
// Memory ordering: the L2 of each XCD is not coherent with the others, so
// every value one block produces for another in the same launch moves
// through agent-scope (sc1) stores/loads or atomics, and a writer waits for
// its stores (s_waitcnt vmcnt(0)) before it signals with an atomic.  Weights
// and the KV cache history are produced by earlier launches and use ordinary
// loads.  The new K/V row is read back from a coherent side buffer, not from
// the cache.  Barrier spins are bounded: on timeout the kernel raises an
// error flag and runs to completion.
#include "common.h"
#include "launch.h"
#include "decode_fused.h"

namespace {

constexpr int NWAVE = 8;
constexpr int NTHR = NWAVE * 64;
constexpr int SPIN_MAX = 1 << 22;
constexpr int MAXR_F = 8;        // query heads per kv head

__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

#define GLOBAL_AS __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ GLOBAL_AS T* gptr(const T* p) {
    return (GLOBAL_AS T*)(const_cast<T*>(p));
}
__device__ __forceinline__ void st_coh(float* p, float v) {
    __hip_atomic_store(gptr(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coh(const float* p) {
    return __hip_atomic_load(gptr(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh16(uint16_t* p, uint16_t v) {
    __hip_atomic_store(gptr(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh64(void* p, uint64_t v) {
    __hip_atomic_store(gptr(reinterpret_cast<uint64_t*>(p)), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_coh64(const void* p) {
    return __hip_atomic_load(gptr(reinterpret_cast<const uint64_t*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned atom_add(unsigned* p, unsigned v) {
    return __hip_atomic_fetch_add(gptr(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned atom_ld(const unsigned* p) {
    return __hip_atomic_load(gptr(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void atom_st(unsigned* p, unsigned v) {
    __hip_atomic_store(gptr(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Tree barrier over the grid, in two halves so that loads can be issued
// between arriving and waiting.  bar[0]: release generation; bar[16]: root
// counter; bar[32 + 16 g]: counter of group g (16 blocks), each on its own
// 64-byte line.  Counters return to 0 after every barrier.
__device__ __forceinline__ unsigned grid_arrive(unsigned* bar) {
    wait_stores();           // every wave: its stores are performed
    __syncthreads();
    unsigned gen = 0;
    if (threadIdx.x == 0) {
        gen = atom_ld(&bar[0]);
        const unsigned nb = gridDim.x, G = 16, ngroups = (nb + G - 1) / G;
        const unsigned grp = blockIdx.x / G, gsize = min(G, nb - grp * G);
        unsigned* gc = &bar[32 + 16 * grp];
        if (atom_add(gc, 1u) + 1 == gsize) {
            atom_st(gc, 0u);
            wait_stores();
            if (atom_add(&bar[16], 1u) + 1 == ngroups) {
                atom_st(&bar[16], 0u);
                wait_stores();
                atom_st(&bar[0], gen + 1);
            }
        }
    }
    return gen;              // meaningful in thread 0 only
}

__device__ __forceinline__ void grid_wait(unsigned* bar, unsigned gen, int* err) {
    if (threadIdx.x == 0) {
        int n = 0;
        while (atom_ld(&bar[0]) == gen) {
            __builtin_amdgcn_s_sleep(1);
            if (++n > SPIN_MAX) { atomicExch(err, 1); break; }
        }
        compiler_fence();
    }
    __syncthreads();
}

__device__ __forceinline__ void grid_sync(unsigned* bar, int* err) { grid_wait(bar, grid_arrive(bar), err); }

__device__ __forceinline__ float scale_of(const DevLinear& W, int n, int g) {
    return (float)__builtin_bit_cast(f16, W.scales[(size_t)n * W.KG + g]);
}

// RMSNorm of B fp32 rows into LDS (fp16-held bf16 values).  coherent: the
// rows were produced in this launch.  Every thread loads its slice of all
// rows at once (one memory round trip), then a block reduction.
template <int MAXB>
__device__ __forceinline__ void norm_rows(const float* src, bool coherent, const uint16_t* gamma, float eps, int B, int K,
                          f16* xs, float* red) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int PER = 8;                        // floats per thread per row
    float v[MAXB][PER];
    const int k0 = tid * PER;                     // K <= NTHR * PER * passes
    float ss[MAXB];
#pragma unroll
    for (int b = 0; b < MAXB; b++) ss[b] = 0.f;
    for (int kk = k0; kk < K; kk += NTHR * PER) {
#pragma unroll
        for (int b = 0; b < MAXB; b++) {
            if (b >= B) break;
#pragma unroll
            for (int j = 0; j < PER; j += 2) {
                const float* p = src + (size_t)b * K + kk + j;
                if (coherent) {
                    const uint64_t u = ld_coh64(p);
                    v[b][j] = __uint_as_float((uint32_t)u);
                    v[b][j + 1] = __uint_as_float((uint32_t)(u >> 32));
                } else {
                    const float2 f = *reinterpret_cast<const float2*>(p);
                    v[b][j] = f.x;
                    v[b][j + 1] = f.y;
                }
            }
        }
#pragma unroll
        for (int b = 0; b < MAXB; b++) {
            if (b >= B) break;
#pragma unroll
            for (int j = 0; j < PER; j++) ss[b] += v[b][j] * v[b][j];
        }
    }
#pragma unroll
    for (int b = 0; b < MAXB; b++) {
        if (b >= B) break;
        const float w = wave_sum(ss[b]);
        if (lane == 0) red[8 + b * NWAVE + wave] = w;
    }
    __syncthreads();
    if (tid < B) {
        float t = 0.f;
        for (int w = 0; w < NWAVE; w++) t += red[8 + tid * NWAVE + w];
        red[tid] = 1.0f / sqrtf(t / (float)K + eps);
    }
    __syncthreads();
    // second pass: the values of the first pass are still in registers when K
    // fits one pass (the common case); otherwise reload
    if (K <= NTHR * PER) {
        if (k0 < K) {
#pragma unroll
            for (int b = 0; b < MAXB; b++) {
                if (b >= B) break;
                const float rb = red[b];
#pragma unroll
                for (int j = 0; j < PER; j++)
                    xs[(size_t)b * K + k0 + j] = act_f16(v[b][j] * rb * bf16_bits_to_f32(gamma[k0 + j]));
            }
        }
    } else {
        for (int i = tid * 2; i < B * K; i += NTHR * 2) {
            const int b = i / K, k = i - b * K;
            float x0, x1;
            if (coherent) {
                const uint64_t u = ld_coh64(src + i);
                x0 = __uint_as_float((uint32_t)u);
                x1 = __uint_as_float((uint32_t)(u >> 32));
            } else {
                x0 = src[i];
                x1 = src[i + 1];
            }
            xs[i] = act_f16(x0 * red[b] * bf16_bits_to_f32(gamma[k]));
            xs[i + 1] = act_f16(x1 * red[b] * bf16_bits_to_f32(gamma[k + 1]));
        }
    }
    __syncthreads();
}

// Load B coherent fp16 rows [B][K] (4 halves per 8-byte load) into LDS.
__device__ __forceinline__ void load_rows_f16(const f16* src, int B, int K, f16* xs) {
    for (int i = threadIdx.x * 4; i < B * K; i += NTHR * 4)
        *reinterpret_cast<uint64_t*>(xs + i) = ld_coh64(src + i);
    __syncthreads();
}

// Even split of T tiles over all waves: wave w owns [w*TPW, min((w+1)*TPW, T)).
struct Split {
    int KB, TPW, total;
    __device__ int first_wave(int t) const { return (t * KB) / TPW; }
    __device__ int nseg(int t) const { return ((t + 1) * KB - 1) / TPW - (t * KB) / TPW + 1; }
};

constexpr int GDEPTH = 8;   // tiles per batch (16 bytes per lane each)

struct Prefetch {
    u32x4 w[GDEPTH];
    float sc[GDEPTH][2];     // scale of the tile's group(s): k 0..31 and 32..63
};

// Tile i of the wave's run (column tile t, k-tile kb) and the scales of its
// two k halves (equal unless the group size is 32).
__device__ __forceinline__ void load_tile(const DevLinear& W, int i, int i1, int t, int kb, int lane, u32x4& w,
                                          float (&sc)[2]) {
    if (i < i1) {
        const int col = t * 32 + (lane & 31);
        w = reinterpret_cast<const u32x4*>(W.qw)[(size_t)i * 64 + lane];
        const int g0 = (kb * 64) >> W.lgG, g1 = (kb * 64 + 32) >> W.lgG;
        sc[0] = scale_of(W, col, g0);
        sc[1] = (g1 != g0) ? scale_of(W, col, g1) : sc[0];
    } else {
        w = u32x4{0, 0, 0, 0};
        sc[0] = sc[1] = 0.f;
    }
}

// Issue the first batch of this wave's tiles (weights do not depend on earlier
// phases, so this can run ahead of a grid barrier).
__device__ __forceinline__ void gemv_prefetch(const DevLinear& W, const Split& sp, Prefetch& pf) {
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * NWAVE + (threadIdx.x >> 6);
    const int i0 = wave * sp.TPW, i1 = min(i0 + sp.TPW, sp.total);
    const int t0 = i0 / sp.KB, bnd = (t0 + 1) * sp.KB;
#pragma unroll
    for (int u = 0; u < GDEPTH; u++) {
        const int i = i0 + u, t = (i >= bnd) ? t0 + 1 : t0;
        load_tile(W, i, i1, t, i - t * sp.KB, lane, pf.w[u], pf.sc[u]);
    }
}

// One wave's share of a GEMV phase: its contiguous run of tiles [i0, i1)
// (column-major) covers at most two column tiles (the host keeps the number
// of column tiles below the number of waves).  Batches are pipelined: the
// next batch is in flight while the current one is dotted.  The B sums per
// lane column of each column tile go to emit(t, seg, acc).
template <int MAXB, typename Emit>
__device__ __forceinline__ void gemv_share(const DevLinear& W, const Split& sp, const f16* xs, int ldx, int B, Prefetch& pf,
                           Emit emit) {
    const int lane = threadIdx.x & 63, h = lane >> 5, c = lane & 31;
    const int wave = blockIdx.x * NWAVE + (threadIdx.x >> 6);
    const int i0 = wave * sp.TPW, i1 = min(i0 + sp.TPW, sp.total);
    if (i0 >= i1) return;
    const int t0 = i0 / sp.KB, bnd = (t0 + 1) * sp.KB;
    float acc[MAXB], gacc[MAXB], acc0[MAXB];
#pragma unroll
    for (int b = 0; b < MAXB; b++) { acc[b] = 0.f; gacc[b] = 0.f; acc0[b] = 0.f; }
    int t_cur = t0, cur_g = -1;
    float sc = 0.f;
    f16x2 zo = zero_offset_pair(nullptr, 0);
    for (int pos = i0; pos < i1; pos += GDEPTH) {
        Prefetch nx;
#pragma unroll
        for (int u = 0; u < GDEPTH; u++) {
            const int i = pos + GDEPTH + u, t = (i >= bnd) ? t0 + 1 : t0;
            load_tile(W, i, i1, t, i - t * sp.KB, lane, nx.w[u], nx.sc[u]);
        }
#pragma unroll
        for (int u = 0; u < GDEPTH; u++) {
            const int i = pos + u;
            if (i >= i1) break;
            const int t = (i >= bnd) ? t0 + 1 : t0, kb = i - t * sp.KB;
            if (t != t_cur) {                       // second column tile of the run
#pragma unroll
                for (int b = 0; b < MAXB; b++) { acc0[b] = acc[b] + sc * gacc[b]; acc[b] = 0.f; gacc[b] = 0.f; }
                t_cur = t;
                cur_g = -1;
                sc = 0.f;
            }
            const int col = t * 32 + c;
            const uint32_t wd4[4] = {pf.w[u][0], pf.w[u][1], pf.w[u][2], pf.w[u][3]};
#pragma unroll
            for (int s = 0; s < 4; s++) {
                const int k = kb * 64 + s * 16 + h * 8;
                const int g = (kb * 64 + s * 16) >> W.lgG;
                if (g != cur_g) {
#pragma unroll
                    for (int b = 0; b < MAXB; b++) { acc[b] += sc * gacc[b]; gacc[b] = 0.f; }
                    cur_g = g;
                    sc = pf.sc[u][s >= 2 ? 1 : 0];
                    if (W.zeros) zo = zero_offset_pair(W.zeros, (size_t)col * W.KG + g);
                }
                const uint32_t wd = wd4[s];
                const f16x2 d0 = dequant_pair(wd, 0, zo), d1 = dequant_pair(wd, 1, zo);
                const f16x2 d2 = dequant_pair(wd, 2, zo), d3 = dequant_pair(wd, 3, zo);
#pragma unroll
                for (int b = 0; b < MAXB; b++) {
                    if (b < B) {
                        const f16x8 xv = *reinterpret_cast<const f16x8*>(xs + (size_t)b * ldx + k);
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
        pf = nx;
    }
#pragma unroll
    for (int b = 0; b < MAXB; b++) acc[b] += sc * gacc[b];
    if (t_cur != t0) {
#pragma unroll
        for (int b = 0; b < MAXB; b++) acc0[b] += __shfl_xor(acc0[b], 32, 64);
        emit(t0, wave - sp.first_wave(t0), acc0);
    }
#pragma unroll
    for (int b = 0; b < MAXB; b++) acc[b] += __shfl_xor(acc[b], 32, 64);
    emit(t_cur, wave - sp.first_wave(t_cur), acc);
}

// Partial of column tile t, segment seg: part[(t * SEGMAX + seg) * B + b][32].
template <int MAXB>
__device__ __forceinline__ void store_partial(float* part, int segmax, int t, int seg, int B, const float (&acc)[MAXB]) {
    const int lane = threadIdx.x & 63;
    if (lane < 32)
#pragma unroll
        for (int b = 0; b < MAXB; b++)
            if (b < B) st_coh(part + ((size_t)(t * segmax + seg) * B + b) * 32 + lane, acc[b]);
}

// Sum of the partials of column tile t for row b, lane column c, in segment
// order.  Up to 24 loads go out together (one round trip in practice).
__device__ __forceinline__ float sum_partials(const float* part, int segmax, const Split& sp, int t, int B, int b, int c) {
    float v = 0.f;
    const int ns = sp.nseg(t);
    for (int s0 = 0; s0 < ns; s0 += 24) {
        float x[24];
#pragma unroll
        for (int j = 0; j < 24; j++)
            x[j] = (s0 + j < ns) ? ld_coh(part + ((size_t)(t * segmax + s0 + j) * B + b) * 32 + c) : 0.f;
#pragma unroll
        for (int j = 0; j < 24; j++) v += x[j];
    }
    return v;
}

// Signal that a partial of unit p (a column tile or a pair of them) is
// stored; true for the wave that stored the last one (all lanes agree).
__device__ __forceinline__ bool pair_done(unsigned* cnt, int p, unsigned total) {
    const int lane = threadIdx.x & 63;
    wait_stores();
    unsigned old = 0;
    if (lane == 0) old = atom_add(&cnt[p], 1u);
    old = __shfl(old, 0, 64);
    const bool last = (old + 1 == total);
    if (last) {
        compiler_fence();
        if (lane == 0) atom_st(&cnt[p], 0u);
    }
    return last;
}

// ---------------------------------------------------------------- kernel

template <int D, int MAXB>
__global__ void __launch_bounds__(NTHR) decode_fused_kernel(DecodeFusedArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int B = a.B, H = a.H, d = D, nq = a.nq, nkv = a.nkv, r = nq / nkv;
    const int qd = nq * d;
    f16* xs = reinterpret_cast<f16*>(smem);                    // activation rows
    float* red = reinterpret_cast<float*>(smem + a.lds_act);   // small scratch
    // phase timestamps (block 0, thread 0): start and after each barrier
    auto stamp = [&](int i) {
        if (blockIdx.x == 0 && tid == 0 && a.stamps) a.stamps[i] = wall_clock64();
    };
    auto arrive = [&](int ph) {      // this block's arrival at the barrier ending phase ph
        if (tid == 0 && a.stamps) a.stamps[8 + ph * gridDim.x + blockIdx.x] = wall_clock64();
    };
    stamp(0);

    // ================= P1: q/k/v =================
    Prefetch pf;
    const Split sp_qkv{a.qkv.K_pad / 64, a.tpw_qkv, (a.qkv.N_dev / 32) * (a.qkv.K_pad / 64)};
    const Split sp_o{a.o.K_pad / 64, a.tpw_o, (a.o.N_dev / 32) * (a.o.K_pad / 64)};
    const Split sp_gu{a.gu.K_pad / 64, a.tpw_gu, (a.gu.N_dev / 32) * (a.gu.K_pad / 64)};
    const Split sp_dn{a.down.K_pad / 64, a.tpw_down, (a.down.N_dev / 32) * (a.down.K_pad / 64)};
    gemv_prefetch(a.qkv, sp_qkv, pf);
    norm_rows<MAXB>(a.x, false, a.attn_norm, a.eps, B, H, xs, red);
    {
        const Split& sp = sp_qkv;
        gemv_share<MAXB>(a.qkv, sp, xs, H, B, pf, [&](int t, int seg, const float (&acc)[MAXB]) {
            store_partial<MAXB>(a.part_qkv, a.segmax_qkv, t, seg, B, acc);
            const int p = t / 2;
            if (!pair_done(a.cnt_qkv, p, sp.nseg(2 * p) + sp.nseg(2 * p + 1))) return;
            // finalize the pair: RoPE for q/k, bf16, write q / cache / new-row buffer
            if (lane < 32) {
                for (int b = 0; b < B; b++) {
                    const float v0 = sum_partials(a.part_qkv, a.segmax_qkv, sp, 2 * p, B, b, lane);
                    const float v1 = sum_partials(a.part_qkv, a.segmax_qkv, sp, 2 * p + 1, B, b, lane);
                    // which, head, dims of the pair
                    int n = p * 64, kind, head;
                    const int kd = nkv * d;
                    if (n < qd) { kind = 0; head = n / d; n -= head * d; }
                    else if (n < qd + kd) { kind = 1; n -= qd; head = n / d; n -= head * d; }
                    else { kind = 2; n -= qd + kd; head = n / d; n -= head * d; }
                    const int p0 = n / 32;
                    const int dim0 = 32 * rope_block(p0, d) + lane, dim1 = 32 * rope_block(p0 + 1, d) + lane;
                    float o0 = v0, o1 = v1;
                    if (kind < 2) {
                        const int ps = a.pos[b];
                        const float cs = a.rope_cos[(size_t)ps * (d / 2) + dim0];
                        const float sn = a.rope_sin[(size_t)ps * (d / 2) + dim0];
                        o0 = v0 * cs - v1 * sn;
                        o1 = v1 * cs + v0 * sn;
                    }
                    const uint16_t b0 = bf16_bits_rne(o0), b1 = bf16_bits_rne(o1);
                    if (kind == 0) {
                        uint16_t* q = a.q_fin + ((size_t)b * nq + head) * d;
                        st_coh16(q + dim0, b0);
                        st_coh16(q + dim1, b1);
                    } else {
                        const int slot = a.ctx_lens[b];
                        uint16_t* cache = (kind == 1) ? a.k_cache : a.v_cache;
                        uint16_t* cp = cache + (size_t)b * a.sb + (size_t)head * a.sh + (size_t)slot * d;
                        cp[dim0] = b0;
                        cp[dim1] = b1;
                        uint16_t* nv = a.kv_new + (((size_t)b * 2 + (kind - 1)) * nkv + head) * d;
                        st_coh16(nv + dim0, b0);
                        st_coh16(nv + dim1, b1);
                    }
                }
            }
        });
    }
    arrive(0);
    grid_sync(a.bar, a.err);
    stamp(1);

    // ================= P2: attention =================
    {
        constexpr int LPK = D / 8, KPW = 64 / LPK;
        float* sc = reinterpret_cast<float*>(smem);                 // [r][chunk]
        float* ored = sc + MAXR_F * a.chunk;                        // [NWAVE][r][D]
        float* stat = ored + NWAVE * MAXR_F * D;                    // [r][2]
        const int units = B * nkv * a.nchunk;
        const int kl = lane / LPK, dseg = lane % LPK;
        const float LOG2E = 1.4426950408889634f;
        for (int u = blockIdx.x; u < units; u += gridDim.x) {
            const int b = u / (nkv * a.nchunk), rem = u % (nkv * a.nchunk);
            const int g = rem / a.nchunk, chunk = rem % a.nchunk;
            const int ctx = a.ctx_lens[b];
            const int start = chunk * a.chunk, end = min(start + a.chunk, ctx + 1);
            if (start >= end) continue;
            const uint16_t* kc = a.k_cache + (size_t)b * a.sb + (size_t)g * a.sh;
            const uint16_t* vc = a.v_cache + (size_t)b * a.sb + (size_t)g * a.sh;
            const uint16_t* kn = a.kv_new + (((size_t)b * 2 + 0) * nkv + g) * d;
            const uint16_t* vn = a.kv_new + (((size_t)b * 2 + 1) * nkv + g) * d;
            uint32_t qv[MAXR_F][4];
#pragma unroll
            for (int i = 0; i < MAXR_F; i++) {
                if (i < r) {
                    const uint16_t* qp = a.q_fin + ((size_t)b * nq + g * r + i) * d + dseg * 8;
                    const uint64_t lo = ld_coh64(qp), hi = ld_coh64(qp + 4);
                    qv[i][0] = (uint32_t)lo; qv[i][1] = (uint32_t)(lo >> 32);
                    qv[i][2] = (uint32_t)hi; qv[i][3] = (uint32_t)(hi >> 32);
                } else {
                    qv[i][0] = qv[i][1] = qv[i][2] = qv[i][3] = 0;
                }
            }
            const float* mrow = a.mask ? a.mask + (size_t)b * a.max_seq : nullptr;
            for (int k0 = start + wave * KPW; k0 < end; k0 += NWAVE * KPW) {
                const int key = k0 + kl;
                const bool valid = key < end;
                uint32_t kw[4] = {0, 0, 0, 0};
                if (valid) {
                    if (key == ctx) {
                        const uint64_t lo = ld_coh64(kn + dseg * 8), hi = ld_coh64(kn + dseg * 8 + 4);
                        kw[0] = (uint32_t)lo; kw[1] = (uint32_t)(lo >> 32); kw[2] = (uint32_t)hi; kw[3] = (uint32_t)(hi >> 32);
                    } else {
                        const u32x4 kk = *reinterpret_cast<const u32x4*>(kc + (size_t)key * d + dseg * 8);
                        kw[0] = kk[0]; kw[1] = kk[1]; kw[2] = kk[2]; kw[3] = kk[3];
                    }
                }
#pragma unroll
                for (int i = 0; i < MAXR_F; i++) {
                    if (i >= r) break;
                    float v = 0.f;
#pragma unroll
                    for (int pp = 0; pp < 4; pp++)
                        v = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(qv[i][pp]), as_bf16x2(kw[pp]), v, false);
#pragma unroll
                    for (int o = 1; o < LPK; o <<= 1) v += __shfl_xor(v, o, 64);
                    if (dseg == 0 && valid) {
                        float s = v * a.scale_log2;
                        if (mrow) s += mrow[key] * LOG2E;
                        sc[i * a.chunk + (key - start)] = s;
                    }
                }
            }
            __syncthreads();
            const int n = end - start;
            for (int i = wave; i < r; i += NWAVE) {
                float mx = -INFINITY;
                for (int j = lane; j < n; j += 64) mx = fmaxf(mx, sc[i * a.chunk + j]);
                mx = wave_max(mx);
                float sum = 0.f;
                for (int j = lane; j < n; j += 64) {
                    const float pv = (mx == -INFINITY) ? 0.f : exp2f(sc[i * a.chunk + j] - mx);
                    sc[i * a.chunk + j] = pv;
                    sum += pv;
                }
                sum = wave_sum(sum);
                if (lane == 0) { stat[2 * i] = mx; stat[2 * i + 1] = sum; }
            }
            __syncthreads();
            float ov[MAXR_F][8];
#pragma unroll
            for (int i = 0; i < MAXR_F; i++)
#pragma unroll
                for (int j = 0; j < 8; j++) ov[i][j] = 0.f;
            for (int k0 = start + wave * KPW; k0 < end; k0 += NWAVE * KPW) {
                const int key = k0 + kl;
                if (key >= end) continue;
                uint32_t vw[4];
                if (key == ctx) {
                    const uint64_t lo = ld_coh64(vn + dseg * 8), hi = ld_coh64(vn + dseg * 8 + 4);
                    vw[0] = (uint32_t)lo; vw[1] = (uint32_t)(lo >> 32); vw[2] = (uint32_t)hi; vw[3] = (uint32_t)(hi >> 32);
                } else {
                    const u32x4 vv = *reinterpret_cast<const u32x4*>(vc + (size_t)key * d + dseg * 8);
                    vw[0] = vv[0]; vw[1] = vv[1]; vw[2] = vv[2]; vw[3] = vv[3];
                }
                float vf[8];
#pragma unroll
                for (int pp = 0; pp < 4; pp++) {
                    vf[2 * pp] = __uint_as_float(vw[pp] << 16);
                    vf[2 * pp + 1] = __uint_as_float(vw[pp] & 0xFFFF0000u);
                }
#pragma unroll
                for (int i = 0; i < MAXR_F; i++) {
                    if (i >= r) break;
                    const float pv = sc[i * a.chunk + (key - start)];
#pragma unroll
                    for (int j = 0; j < 8; j++) ov[i][j] += pv * vf[j];
                }
            }
#pragma unroll
            for (int i = 0; i < MAXR_F; i++) {
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
                    for (int j = 0; j < 8; j++) ored[(wave * MAXR_F + i) * D + dseg * 8 + j] = ov[i][j];
            }
            __syncthreads();
            for (int idx = tid; idx < r * D; idx += NTHR) {
                const int i = idx / D, dim = idx % D;
                float v = 0.f;
#pragma unroll
                for (int w = 0; w < NWAVE; w++) v += ored[(w * MAXR_F + i) * D + dim];
                float* pp = a.apart + (((size_t)b * nq + g * r + i) * a.nchunk + chunk) * (D + 2);
                st_coh(pp + dim, v);
                if (dim == 0) { st_coh(pp + D, stat[2 * i]); st_coh(pp + D + 1, stat[2 * i + 1]); }
            }
            // last chunk of this (b, g) combines the heads of the group
            wait_stores();
            __syncthreads();
            __shared__ unsigned last_flag;
            if (tid == 0) {
                const unsigned nch = (unsigned)((ctx + 1 + a.chunk - 1) / a.chunk);
                const unsigned old = atom_add(&a.cnt_attn[b * nkv + g], 1u);
                last_flag = (old + 1 == nch);
                if (last_flag) atom_st(&a.cnt_attn[b * nkv + g], 0u);
            }
            __syncthreads();
            if (last_flag) {
                compiler_fence();
                const int nch = (ctx + 1 + a.chunk - 1) / a.chunk;
                float* ml = sc;   // [r][nch][2] (the scores are no longer needed)
                for (int idx = tid; idx < r * nch * 2; idx += NTHR) {
                    const int i = idx / (nch * 2), rem2 = idx % (nch * 2);
                    const int ch = rem2 / 2, which = rem2 % 2;
                    ml[idx] = ld_coh(a.apart + (((size_t)b * nq + g * r + i) * a.nchunk + ch) * (D + 2) + D + which);
                }
                __syncthreads();
                for (int idx = tid; idx < r * D; idx += NTHR) {
                    const int i = idx / D, dim = idx % D;
                    const float* pp = a.apart + (((size_t)b * nq + g * r + i) * a.nchunk) * (D + 2);
                    const float* mli = ml + i * nch * 2;
                    float M = -INFINITY;
                    for (int ch = 0; ch < nch; ch++) M = fmaxf(M, mli[2 * ch]);
                    float L = 0.f, O = 0.f;
                    if (M != -INFINITY) {
                        for (int c0 = 0; c0 < nch; c0 += 32) {
                            float ov8[32];
#pragma unroll
                            for (int j = 0; j < 32; j++)
                                ov8[j] = (c0 + j < nch) ? ld_coh(pp + (c0 + j) * (D + 2) + dim) : 0.f;
#pragma unroll
                            for (int j = 0; j < 32; j++) {
                                if (c0 + j >= nch) break;
                                const float mc = mli[2 * (c0 + j)];
                                if (mc == -INFINITY) continue;
                                const float w = exp2f(mc - M);
                                L += w * mli[2 * (c0 + j) + 1];
                                O += w * ov8[j];
                            }
                        }
                    }
                    const f16 val = act_f16(L > 0.f ? O / L : 0.f);
                    st_coh16(reinterpret_cast<uint16_t*>(a.A) + ((size_t)b * nq + g * r + i) * D + dim,
                             __builtin_bit_cast(uint16_t, val));
                }
            }
            __syncthreads();
        }
    }
    arrive(1);
    {
        const unsigned gen = grid_arrive(a.bar);
        gemv_prefetch(a.o, sp_o, pf);
        grid_wait(a.bar, gen, a.err);
    }
    stamp(2);

    // ================= P3: o_proj, h = x + A Wo =================
    load_rows_f16(a.A, B, qd, xs);
    {
        const Split& sp = sp_o;
        gemv_share<MAXB>(a.o, sp, xs, qd, B, pf, [&](int t, int seg, const float (&acc)[MAXB]) {
            store_partial<MAXB>(a.part_o, a.segmax_o, t, seg, B, acc);
            if (!pair_done(a.cnt_o, t, sp.nseg(t))) return;
            if (lane < 32)
                for (int b = 0; b < B; b++) {
                    const size_t i = (size_t)b * H + t * 32 + lane;
                    st_coh(a.h + i, a.x[i] + sum_partials(a.part_o, a.segmax_o, sp, t, B, b, lane));
                }
        });
    }
    arrive(2);
    {
        const unsigned gen = grid_arrive(a.bar);
        gemv_prefetch(a.gu, sp_gu, pf);
        grid_wait(a.bar, gen, a.err);
    }
    stamp(3);

    // ================= P4: gate/up on RMSNorm(h) =================
    norm_rows<MAXB>(a.h, true, a.mlp_norm, a.eps, B, H, xs, red);
    {
        const Split& sp = sp_gu;
        gemv_share<MAXB>(a.gu, sp, xs, H, B, pf, [&](int t, int seg, const float (&acc)[MAXB]) {
            store_partial<MAXB>(a.part_gu, a.segmax_gu, t, seg, B, acc);
            const int p = t / 2;
            if (!pair_done(a.cnt_gu, p, sp.nseg(2 * p) + sp.nseg(2 * p + 1))) return;
            if (lane < 32) {
                for (int b = 0; b < B; b++) {
                    const float gv = sum_partials(a.part_gu, a.segmax_gu, sp, 2 * p, B, b, lane);
                    const float uv = sum_partials(a.part_gu, a.segmax_gu, sp, 2 * p + 1, B, b, lane);
                    const f16 val = act_f16(silu(gv) * uv);
                    st_coh16(reinterpret_cast<uint16_t*>(a.g) + (size_t)b * a.F_pad + p * 32 + lane,
                             __builtin_bit_cast(uint16_t, val));
                }
            }
        });
    }
    arrive(3);
    {
        const unsigned gen = grid_arrive(a.bar);
        gemv_prefetch(a.down, sp_dn, pf);
        grid_wait(a.bar, gen, a.err);
    }
    stamp(4);

    // ================= P5: down, y = h + g Wd =================
    load_rows_f16(a.g, B, a.F_pad, xs);
    {
        const Split& sp = sp_dn;
        gemv_share<MAXB>(a.down, sp, xs, a.F_pad, B, pf, [&](int t, int seg, const float (&acc)[MAXB]) {
            store_partial<MAXB>(a.part_down, a.segmax_down, t, seg, B, acc);
            if (!pair_done(a.cnt_down, t, sp.nseg(t))) return;
            if (lane < 32)
                for (int b = 0; b < B; b++) {
                    const size_t i = (size_t)b * H + t * 32 + lane;
                    a.y[i] = ld_coh(a.h + i) + sum_partials(a.part_down, a.segmax_down, sp, t, B, b, lane);
                }
        });
    }
    arrive(4);
    if (a.stamps) {          // end: the last block to finish writes the time
        wait_stores();
        __syncthreads();
        if (tid == 0 && atom_add(&a.bar[8], 1u) + 1 == gridDim.x) {
            atom_st(&a.bar[8], 0u);
            a.stamps[5] = wall_clock64();
        }
    }
}

template <int D, int MAXB>
int launch_t(const DecodeFusedArgs& a, hipStream_t stream) {
    auto fn = decode_fused_kernel<D, MAXB>;
    if (hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)a.lds_bytes) != hipSuccess)
        return -1;
    DecodeFusedArgs args = a;
    void* kargs[] = {&args};
    return hipLaunchCooperativeKernel((const void*)fn, dim3(a.nblocks), dim3(NTHR), kargs, a.lds_bytes, stream) ==
                   hipSuccess
               ? 0
               : -1;
}

}  // namespace

int decode_fused_blocks(int head_dim, int B, size_t lds_bytes) {
    int dev = 0, cus = 0, occ = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    const void* fn = nullptr;
    if (head_dim == 128) fn = B <= 1 ? (const void*)decode_fused_kernel<128, 1> : (const void*)decode_fused_kernel<128, 4>;
    else fn = B <= 1 ? (const void*)decode_fused_kernel<64, 1> : (const void*)decode_fused_kernel<64, 4>;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, NTHR, lds_bytes) != hipSuccess) return 0;
    return occ >= 1 ? cus : 0;
}

int launch_decode_fused(const DecodeFusedArgs& a, hipStream_t stream) {
    if (a.B > 4) return -1;
    if (a.d == 128) return a.B <= 1 ? launch_t<128, 1>(a, stream) : launch_t<128, 4>(a, stream);
    if (a.d == 64) return a.B <= 1 ? launch_t<64, 1>(a, stream) : launch_t<64, 4>(a, stream);
    return -1;
}
