// Kernel launchers (internal) and the q/k/v epilogue shared by the GEMM and
// the GEMV.
#pragma once
#include "common.h"

// q/k/v epilogue for one row and one RoPE pair of device columns.
// n_base: device column of the first tile of the pair (multiple of 64);
// c: column inside the tile; v0, v1: sums of columns n_base + c and
// n_base + 32 + c, which hold dims i and i + d/2 of the same head.
// RoPE (Sec. 3.1 Listing 1, table of Sec. 4.6.2) is applied to q and k; the
// results are rounded to bf16 and written to the q buffer or the cache slot.
__device__ __forceinline__ void epi_qkv_pair(const EpiArgs& ep, int row, int n_base, int c,
                                             float v0, float v1, int slot, int seq) {
    const int d = ep.head_dim;
    const int qd = ep.nq * d, kd = ep.nkv * d;
    int n = n_base;
    int kind, head;
    if (n < qd) { kind = 0; head = n / d; n -= head * d; }
    else if (n < qd + kd) { kind = 1; n -= qd; head = n / d; n -= head * d; }
    else { kind = 2; n -= qd + kd; head = n / d; n -= head * d; }
    const int p0 = n / 32;
    const int dim0 = 32 * rope_block(p0, d) + c;
    const int dim1 = 32 * rope_block(p0 + 1, d) + c;
    float o0 = v0, o1 = v1;
    if (kind < 2) {
        const int pos = ep.pos[row];
        const float cs = ep.rope_cos[(size_t)pos * (d / 2) + dim0];
        const float sn = ep.rope_sin[(size_t)pos * (d / 2) + dim0];
        o0 = v0 * cs - v1 * sn;
        o1 = v1 * cs + v0 * sn;
    }
    const uint16_t b0 = bf16_bits_rne(o0), b1 = bf16_bits_rne(o1);
    if (kind == 0) {
        uint16_t* q = ep.q_out + ((size_t)row * ep.nq + head) * d;
        q[dim0] = b0;
        q[dim1] = b1;
    } else {
        uint16_t* cache = (kind == 1) ? ep.k_cache : ep.v_cache;
        uint16_t* p = cache + (size_t)seq * ep.cache_stride_b + (size_t)head * ep.cache_stride_h + (size_t)slot * d;
        p[dim0] = b0;
        p[dim1] = b1;
    }
}

// Prefill GEMM launch plan: row tile (32 * TM rows), k splits S, grid.
struct GemmPlan {
    int TM = 4, S = 1, nrb = 0, ncb = 0, tiles = 0;
    size_t part_bytes = 0;        // fp32 partial sums (S > 1)
};
GemmPlan gemm_w4_plan(int M, const DevLinear& W, int num_cus);
// part: plan.part_bytes of workspace; cnt: plan.tiles 64-bit arrival
// counters in any state; tag: non-zero, different from the tag of every
// earlier launch that used the same counters.  part and cnt are unused when
// plan.S == 1.
int launch_gemm_w4(int epi, const f16* X, int ldx, const DevLinear& W, const EpiArgs& ep, const GemmPlan& plan,
                   int M, float* part, unsigned long long* cnt, unsigned tag, hipStream_t stream);

struct GemvArgs {
    DevLinear W;
    const float* x_f32;      // NORM prologue input fp32 [B][K] (K = hidden)
    const uint16_t* gamma;   // bf16 bits [K]
    float eps;
    const f16* x_f16;        // activation input [B][ldx] (non-NORM)
    int ldx;
    int B;
    int ksplit;              // blocks along K
    EpiArgs ep;
    const float* copy_src;   // optional side copy (fp32), count copy_n
    float* copy_dst;
    int copy_n;
};
int launch_gemv_w4(int epi, bool norm, const GemvArgs& a, hipStream_t stream);

int launch_rmsnorm(const float* x, const uint16_t* gamma, float eps, int M, int H, f16* out, int* err,
                   hipStream_t stream);

struct AttnPrefillArgs {
    const uint16_t* q;       // bf16 [T][nq][d]
    const uint16_t* k_cache; // bf16 [nkv][max_seq][d] of the sequence
    const uint16_t* v_cache;
    long long cache_stride_h;
    f16* out;                // [T][nq*d]
    int T, L, nq, nkv, d;
    float scale_log2;        // log2(e) / sqrt(d)
    float* part;             // chunk partial states (plan.part_bytes)
    int chunk_keys, ngrp, items;   // set by the launcher from the plan
    int* err;                // the layer's error flag (W4_FLAG_F16_RANGE)
};
// Prefill attention launch plan: key chunk length, work items per block
// row, block size, workspace.
struct AttnPrefillPlan {
    int chunk_keys = 0, items = 0, ngrp = 1, threads = 64;
    bool merge = false;      // some query tile has more than one chunk
    size_t part_bytes = 0;
    size_t part_bound = 0;   // part_bytes of any history up to L (non-decreasing in L)
    size_t lds_bytes = 0;
};
AttnPrefillPlan attn_prefill_plan(int T, int L, int nq, int nkv, int d, int num_cus);
int launch_attn_prefill(const AttnPrefillArgs& a, const AttnPrefillPlan& p, hipStream_t stream);

struct AttnDecodeArgs {
    const uint16_t* q;       // bf16 [B][nq][d]
    const uint16_t* k_cache; // bf16 [B][nkv][max_seq][d]
    const uint16_t* v_cache;
    long long stride_b, stride_h;
    const int32_t* ctx_lens; // [B] device, or null: row b's context is ctx_base + b
    int ctx_base;
    const float* mask;       // [B][max_seq] or null
    int max_seq;
    float* part;             // [B][nq][nchunks][d + 2]
    f16* out;                // [B][nq*d]
    int B, nq, nkv, d, chunk, nchunks;
    float scale_log2;
    int* err;                // the layer's error flag (W4_FLAG_F16_RANGE)
};
int launch_attn_decode(const AttnDecodeArgs& a, hipStream_t stream);

int launch_kv_append(uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_new, const uint16_t* v_new,
                     int B, int T, int nkv, int d, long long stride_b, long long stride_h,
                     const int32_t* slot_start_host, hipStream_t stream);

int launch_debug_dequant(const DevLinear& W, const int32_t* col_map, int K, int N, float* out,
                         hipStream_t stream);
