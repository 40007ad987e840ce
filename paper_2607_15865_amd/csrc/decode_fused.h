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
    const int32_t* ctx_lens;   // [B]
    const float* mask;         // [B][max_seq] or null
    int max_seq;
    uint16_t* k_cache;
    uint16_t* v_cache;
    long long sb, sh;
    float* y;                  // [B][H]
    // workspace
    float* h;                  // [B][H]
    float* part_qkv;           // [CT][segmax][B][32]
    float* part_gu;
    float* part_o;
    float* part_down;
    uint16_t* q_fin;           // bf16 [B][nq*d]
    uint16_t* kv_new;          // bf16 [B][2][nkv][d]
    float* apart;              // [B][nq][nchunk][d+2]
    f16* A;                    // [B][nq*d]
    f16* g;                    // [B][F_pad]
    // synchronisation state (per layer handle, zeroed at create)
    unsigned* bar;
    unsigned* cnt_qkv;
    unsigned* cnt_gu;
    unsigned* cnt_attn;
    unsigned* cnt_o;           // per column tile of o_proj
    unsigned* cnt_down;        // per column tile of down
    int* err;
    unsigned long long* stamps;  // [6] phase timestamps (wall clock) or null
    // work split
    int tpw_qkv, tpw_o, tpw_gu, tpw_down;
    int segmax_qkv, segmax_gu, segmax_o, segmax_down;
    int chunk, nchunk;
    float scale_log2;
    int nblocks;
    size_t lds_act;            // bytes of the activation rows in LDS
    size_t lds_bytes;          // dynamic LDS per block
};

int launch_decode_fused(const DecodeFusedArgs& a, hipStream_t stream);
// Blocks of the persistent launch (one per CU) or 0 if it cannot be resident.
int decode_fused_blocks(int head_dim, int B, size_t lds_bytes);
