// Arguments of the persistent decode kernel (decode_fused.hip).
#pragma once
#include "common.h"

struct DecodeFusedArgs {
    DevLinear qkv, o, gu, down;
    const uint16_t* attn_norm;
    const uint16_t* mlp_norm;
    float eps;
    const float* rope_cos;
    const float* rope_sin;
    int H, nq, nkv, d, F_pad, B;
    const float* x;            // [B][H]
    const int32_t* pos;        // [B]
    const int32_t* ctx_lens;   // [B], or null: row b's context is ctx_base + b
    int ctx_base;
    int shared;                // rows are consecutive tokens of one sequence: one cache
                               // (sb = 0), row b also attends to rows 0 .. b-1 (B <= 4)
    const float* mask;         // [B][max_seq] or null
    int max_seq;
    uint16_t* k_cache;
    uint16_t* v_cache;
    long long sb, sh;
    float* y;                  // [B][H]
    // workspace: tagged words (payload | epoch << 32)
    uint64_t* qkv_part;        // [S_qkv][B][N_qkv]      fp32 partial sums
    uint64_t* apart;           // [B][nq][nchunk][d + 2] fp32 chunk outputs, max, sum
    uint64_t* A;               // [B][nq*d / 2]          attention output, fp16 pairs
    uint64_t* o_part;          // [S_o][B][H]            fp32 partial sums
    uint64_t* g;               // [B][F_pad / 2]         SwiGLU output, fp16 pairs
    uint64_t* down_part;       // [S_down][B][H]         fp32 partial sums (s >= 1)
    uint32_t epoch;            // tag of this launch (never 0)
    int spin_max;              // polls per thread per launch before a wait gives up
    int* err;                  // the layer's error flag: W4_FLAG_WAIT_TIMEOUT, W4_FLAG_F16_RANGE
    unsigned long long* stamps;  // wall-clock stamps or null
    // work split (each block derives its share from these and its index)
    int S_qkv, S_o, S_down;    // k-parts per column tile (1 or 2)
    int comb_per, comb_lpv;    // attention outputs combined per block, lanes per output
    int slots;                 // column tiles per block in one product (LDS partial slots)
    int chunk, nchunk;         // attention keys per unit, units per (row, kv head)
    float scale_log2;
    int nblocks;
    int ldx;                   // fp16 elements per activation row in LDS
    size_t off_h, off_red, off_gam;  // LDS offsets (bytes)
    size_t off_zero, off_c64;  // LDS: 64 zero fp16; GEMV correction table [ldx / 64][8] fp32
                               // (inside the region the attention phase reuses)
    size_t lds_bytes;          // dynamic LDS per block
    int gam_lds;               // RMSNorm weights held in LDS (at off_gam) or read from memory
};

int launch_decode_fused(const DecodeFusedArgs& a, hipStream_t stream);
// Blocks of the persistent launch (one per CU) or 0 if it cannot be resident.
int decode_fused_blocks(int head_dim, int B, size_t lds_bytes);
// Largest attention chunk (keys per unit) the kernel supports for head_dim.
int decode_fused_max_chunk(int head_dim);
// LDS bytes of the attention phase for chunks of ch keys, head size d: the K
// and V stages ([ch rounded up to 32][d] bf16 each), the per-group outputs
// and statistics ([ch / 32][8 heads][d + 2] fp32), q/k/v in fp32
// ([16][d]: 8 query heads, k, v and the k, v of up to 3 earlier rows), the
// rotated q, k and v in bf16 ([10][d]) and the mask values (ch rounded up to
// 64, fp32).
inline size_t decode_fused_attn_bytes(int ch, int d) {
    const size_t chp = (size_t)(ch + 31) / 32 * 32, ng = chp / 32;
    return 4 * chp * d + (ng * 8 * d + ng * 16 + 16 * (size_t)d) * 4 + 10 * (size_t)d * 2 + (chp + 63) / 64 * 64 * 4;
}
