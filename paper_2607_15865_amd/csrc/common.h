// Shared device helpers and the private device layout of the W4A16 layer.
//
// Device weight layout (written once by layer_create, read by every stage):
//
//   A linear with K rows and N columns is stored as "tiles" of 32 columns x
//   64 rows (k).  Tile (nb, kb) is 1 KB: 64 lanes x 4 words, so one wave
//   reads a whole tile with one 16-byte load per lane.  Lane l holds column
//   32*nb + (l % 32) and, for h = l / 32, the words that cover
//   k = 64*kb + 16*s + 8*h + (0..7) for s = 0..3 (word s of the lane).
//   Inside a word the eight 4-bit codes of k0..k0+7 sit at bit offsets
//   0, 16, 4, 20, 8, 24, 12, 28, so ((w >> 4p) & 0x000F000F) holds the codes
//   of k0+2p (low half) and k0+2p+1 (high half).  OR-ing 0x64006400 makes the
//   fp16 pair (1024 + q) exactly, and subtracting 1024 + z leaves the exact
//   code minus zero point.  This pair order is the operand order of the
//   32x32x16 MFMA, so a lane's word s is its B fragment of k16 step s.
//
//   Tile index: nb * (K_pad / 64) + kb (column strips contiguous along k).
//   Group parameters are group-major, so the 32 lanes of a tile read one
//   contiguous run: scales fp16 [K_pad / G][N_dev]; ratios for the prefill
//   GEMM fp32 [K_pad / G][N_dev] with ratio[g][n] = s[g-1][n] / s[g][n]
//   (g >= 1).  Zero points (optional): uint8 [K_pad / G][N_dev], and the same
//   again packed with the scale bits as uint32 (scale | zero << 16) for the
//   decode GEMV.
//
//   K_pad is a multiple of 128 and of G (the padded FFN width of the down
//   projection; the other K are multiples already); padded rows and groups
//   carry the zero point code (weight 0).  A group whose scale is 0 is stored
//   with all codes at the zero point and a non-zero stand-in scale, so every
//   scale is non-zero (the ratios are finite) and the group still contributes
//   0.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <mutex>

#include "w4layer.h"

typedef _Float16 f16;
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Transposing LDS read (gfx950 ds_read_b64_tr_b16).  In each group of 16
// lanes, source lane s reads the four 16-bit values at its own address p_s;
// output lane t receives, as element k, value t % 4 of source lane
// 4 k + t / 4.  So when lane s of a group points at row r0 + s / 4, columns
// c0 + 4 (s % 4) .. + 3 of a row-major 16-bit matrix, output lane t holds
// column c0 + t of rows r0 .. r0 + 3: a column segment, as the MFMA takes
// its operand.  p: 8-byte aligned, in LDS.
__device__ __forceinline__ i16x4 lds_read_tr16(const void* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4*)(const_cast<void*>(p)));
}
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define W4_TILE_N 32
#define W4_TILE_K 64
#define W4_TILE_WORDS 256   // 64 lanes x 4 words

// Column permutation inside a head for the fused q/k/v weight: the head's
// dims are cut into blocks of 32 and stored as pairs (b, b + d/64) so that a
// RoPE pair (i, i + d/2) lands in the same lane of two adjacent 32-column
// tiles.  Device block p of a head holds dim block rope_block(p).
__host__ __device__ inline int rope_block(int p, int head_dim) {
    int nb = head_dim / 32;          // 2 or 4
    int half = nb / 2;
    return (p % 2 == 0) ? (p / 2) : (p / 2 + half);
}

// Dynamic LDS above 64 KB has to be allowed per kernel with
// hipFuncSetAttribute; the setting lasts, so it is made once per kernel and
// device (again only when a larger size is asked for), not on every launch.
struct LdsLimit {
    int bytes[64] = {};      // per device: the size allowed so far
    std::mutex mu;
};
inline int ensure_lds_limit(LdsLimit& lim, const void* fn, size_t bytes) {
    if (bytes <= 64 * 1024) return 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
    std::lock_guard<std::mutex> g(lim.mu);
    if (lim.bytes[dev] >= (int)bytes) return 0;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) != hipSuccess) return -1;
    lim.bytes[dev] = (int)bytes;
    return 0;
}

// ---------------------------------------------------------------- numerics

// fp32 -> bf16 -> fp32, round to nearest even (finite inputs).
__device__ __forceinline__ float round_bf16(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

__device__ __forceinline__ uint16_t bf16_bits_rne(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Activation store: the value rounded to bf16 and held as fp16, the operand
// type of the W4 MFMA.  Every bf16 value of magnitude 2^-17 .. 65280 is an
// fp16 value, so the store is exact there; smaller magnitudes land on fp16's
// 2^-24 grid (an absolute change below 3e-8).  A bf16 value beyond fp16's
// range (65504) would become an infinity: `bad` records it (also NaN), and
// the kernel raises W4_FLAG_F16_RANGE in the layer's error flag.
__device__ __forceinline__ f16 act_f16(float x, bool& bad) {
    const float r = round_bf16(x);
    bad |= !(__builtin_fabsf(r) <= 65504.0f);
    return (f16)r;
}

// Raise flag bits in a device error word (read and cleared by the host).
__device__ __forceinline__ void raise_flag(int* err, int bits) {
    if (err) atomicOr(err, bits);
}
__device__ __forceinline__ void flag_range(int* err, bool bad) {
    if (bad) raise_flag(err, W4_FLAG_F16_RANGE);
}

// Dequantisation offsets of one zero point z: the fp16 pairs -(1024 + z) and
// -(64 + z).
struct ZeroOff {
    f16x2 even, odd;
};

__device__ __forceinline__ ZeroOff zero_off(float z) {
    ZeroOff r;
    const f16 e = (f16)(-(1024.0f + z)), o = (f16)(-(64.0f + z));
    r.even = f16x2{e, e};
    r.odd = f16x2{o, o};
    return r;
}

// The three bit patterns of dequant8, held in vector registers (opaque to the
// compiler, which would otherwise fold them into instruction literals and
// split every and-or into two instructions).
struct DqConst {
    uint32_t lo, hi, magic;
};

__device__ __forceinline__ uint32_t vreg_const(uint32_t v) {
    uint32_t r;
    asm("v_mov_b32 %0, %1" : "=v"(r) : "i"(v));
    return r;
}

__device__ __forceinline__ DqConst dq_const() {
    return DqConst{vreg_const(0x000F000Fu), vreg_const(0x00F000F0u), vreg_const(0x64006400u)};
}

// Exact fp16 (code - zero) of the eight codes of a weight word, in k order.
// Pair p (k0+2p, k0+2p+1) sits at bits 4p and 16+4p.  OR-ing 0x6400 onto a
// code in bits 0..3 of a half gives the fp16 value 1024 + q, onto a code in
// bits 4..7 the value 1024 + 16q; the first loses 1024 + z by one packed add,
// the second is brought to q - z by one packed fma with 1/16 (exact: the
// product 64 + q is exact and so is the integer sum).  Nine VALU operations
// per word: one shift, four and-or, four packed f16 ops.
__device__ __forceinline__ f16x8 dequant8(uint32_t w, ZeroOff zo, const DqConst& k) {
    const uint32_t w8 = w >> 8;
    const f16x2 sixteenth = f16x2{(f16)0.0625f, (f16)0.0625f};
    const f16x2 p0 = __builtin_bit_cast(f16x2, (w & k.lo) | k.magic) + zo.even;
    const f16x2 p1 = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, (w & k.hi) | k.magic), sixteenth, zo.odd);
    const f16x2 p2 = __builtin_bit_cast(f16x2, (w8 & k.lo) | k.magic) + zo.even;
    const f16x2 p3 = __builtin_elementwise_fma(__builtin_bit_cast(f16x2, (w8 & k.hi) | k.magic), sixteenth, zo.odd);
    f16x8 r;
    r[0] = p0[0]; r[1] = p0[1]; r[2] = p1[0]; r[3] = p1[1];
    r[4] = p2[0]; r[5] = p2[1]; r[6] = p3[0]; r[7] = p3[1];
    return r;
}


// INT8 fragment (codes of bytes lo[0..3], hi[0..3] in k order) -> the exact
// fp16 values (code - zero): v_perm builds the pairs 0x64 | code = 1024 +
// code, one packed add takes zneg = -(1024 + zero).  Six VALU operations.
__device__ __forceinline__ f16x8 dequant8_u8(uint32_t lo, uint32_t hi, f16x2 zneg) {
    const uint32_t m = 0x64646464u;
    const f16x2 p0 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(m, lo, 0x04010400u)) + zneg;
    const f16x2 p1 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(m, lo, 0x04030402u)) + zneg;
    const f16x2 p2 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(m, hi, 0x04010400u)) + zneg;
    const f16x2 p3 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(m, hi, 0x04030402u)) + zneg;
    f16x8 r;
    r[0] = p0[0]; r[1] = p0[1]; r[2] = p1[0]; r[3] = p1[1];
    r[4] = p2[0]; r[5] = p2[1]; r[6] = p3[0]; r[7] = p3[1];
    return r;
}

// F16 fragment (four words of fp16 pairs, the pairs at k % 8 in {2, 3} and
// {6, 7} held times 16) -> the weights (exact: a power-of-two scaling).
__device__ __forceinline__ f16x8 f16_frag(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
    const f16x2 sixteenth = f16x2{(f16)0.0625f, (f16)0.0625f};
    const f16x2 p0 = __builtin_bit_cast(f16x2, w0), p2 = __builtin_bit_cast(f16x2, w2);
    const f16x2 p1 = __builtin_bit_cast(f16x2, w1) * sixteenth, p3 = __builtin_bit_cast(f16x2, w3) * sixteenth;
    f16x8 r;
    r[0] = p0[0]; r[1] = p0[1]; r[2] = p1[0]; r[3] = p1[1];
    r[4] = p2[0]; r[5] = p2[1]; r[6] = p3[0]; r[7] = p3[1];
    return r;
}

// Reinterpret a 32-bit word as a bf16 pair.  Always pass a scalar: clang
// miscompiles __builtin_bit_cast applied directly to an ext_vector element
// with a loop index (it reads element 0).
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t u) {
    bf16x2 r;
    __builtin_memcpy(&r, &u, 4);
    return r;
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// 2^x on the hardware exponential (v_exp_f32).  The library exp2f adds a
// rescaling step that keeps results below 2^-126 exact as denormals; the
// softmax weights that small add nothing to sums whose largest term is 1.
// exp2_hw(-inf) = 0.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// wave-level reductions (64 lanes): DPP within each row of 16 lanes (swap
// lane pairs, swap pairs of pairs, mirror within 8, mirror within 16), then
// the four row results are read from lanes 0, 16, 32 and 48.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over groups of N (8 or 16) adjacent lanes; every lane of a group ends
// with the group's sum.
template <int N>
__device__ __forceinline__ float row_sum(float v) {
    v += dpp_mov<0xB1>(v);                  // quad_perm [1,0,3,2]
    v += dpp_mov<0x4E>(v);                  // quad_perm [2,3,0,1]
    v += dpp_mov<0x141>(v);                 // row_half_mirror
    if (N == 16) v += dpp_mov<0x140>(v);    // row_mirror
    return v;
}

__device__ __forceinline__ float row_max16(float v) {
    v = fmaxf(v, dpp_mov<0xB1>(v));
    v = fmaxf(v, dpp_mov<0x4E>(v));
    v = fmaxf(v, dpp_mov<0x141>(v));
    v = fmaxf(v, dpp_mov<0x140>(v));
    return v;
}

__device__ __forceinline__ float lane_val(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ float wave_sum(float v) {
    v = row_sum<16>(v);
    return (lane_val(v, 0) + lane_val(v, 16)) + (lane_val(v, 32) + lane_val(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
    v = row_max16(v);
    return fmaxf(fmaxf(lane_val(v, 0), lane_val(v, 16)), fmaxf(lane_val(v, 32), lane_val(v, 48)));
}

// ---------------------------------------------------------------- layouts

// Weight formats of a device linear.  Every format cuts the weight into
// tiles of 64 k x 32 columns, tile (t, kb) at index t * (K_pad / 64) + kb;
// lane l of a wave stands for column 32 t + l % 32 and k half l / 32, and
// its fragment s (0..3) holds the 8 values of k = 64 kb + 16 s + 8 (l / 32)
// + 0..7.
//   WF_INT4: 1 KB tiles, [lane][4 words]: word s = fragment s, codes 0..15
//            in the nibble order of dequant8; groups of 2^lgG along k.
//   WF_INT8: 2 KB tiles, [j][lane][4 words]: half j holds fragments 2 j and
//            2 j + 1, 8 unsigned byte codes each in k order (words 2 (s % 2)
//            and 2 (s % 2) + 1 of the half); one scale and zero point per
//            column, repeated in every group of 128 (symmetric weights hold
//            code + 128 with zero point 128).
//   WF_F16:  4 KB tiles, [s][lane][4 words]: fragment s as 8 fp16 values, k
//            order, those at k % 8 in {2, 3, 6, 7} multiplied by 16 (the
//            GEMV's activations take them divided by 16); scales 1.
enum WeightFormat { WF_INT4 = 0, WF_INT8 = 1, WF_F16 = 2 };

struct DevLinear {
    const uint32_t* qw;      // tiles
    const uint16_t* scales;  // fp16 bits [KG][N_dev]
    const float* ratios;     // [KG][N_dev]
    const uint8_t* zeros;    // [KG][N_dev] or null
    const uint32_t* sz;      // scale bits | zero << 16, [KG][N_dev]; null without zeros
    int K, N;                // logical
    int K_pad, N_dev, KG;    // padded rows, device columns, groups
    int lgG;                 // log2 of the group size (a power of two)
    int wf;                  // WeightFormat
};

// Epilogue kinds shared by the GEMM (prefill) and GEMV (decode).
enum EpiKind { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

// Everything an epilogue needs.
struct EpiArgs {
    // QKV
    uint16_t* q_out;          // bf16 [M][nq][d]
    uint16_t* k_cache;        // bf16 base of the cache
    uint16_t* v_cache;
    long long cache_stride_b; // elements between sequences (decode)
    long long cache_stride_h; // elements between kv heads
    const int32_t* pos;       // [M] position ids
    const int32_t* slot_dev;  // decode: [B] device slots (ctx_lens), or null
    int slot_base;            // with slot_dev null: slot of row 0 (rows are consecutive slots)
    const float* rope_cos;    // [max_seq][d/2]
    const float* rope_sin;
    int nq, nkv, head_dim;
    // RESID
    const float* resid;       // fp32 [M][N]
    float* out_f32;           // fp32 [M][N]
    // SWIGLU
    f16* act_out;             // fp16 [M][F_pad]
    int F_pad;
    int* err;                 // the layer's error flag (W4_FLAG_F16_RANGE)
};
