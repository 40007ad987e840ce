// The two ends of the model around the decoder layers (the runtime loop of
// Sec. 2 and Sec. 4.5): the word-embedding gather and the greedy pick over
// the LM head's logits.  The LM head's matmul runs on the decode GEMV
// (gemv_w4.hip) after the row RMSNorm (misc.hip).
//
// Both kernels are HBM streams with no reuse: the gather reads one table row
// per sequence (2 * hidden bytes) and writes it as fp32; the pick reads the
// logits once (4 * vocab bytes per row) in float4 loads, 8192 logits per
// block so that a 128k vocabulary spreads over 16 blocks per row, and a
// second one-wave launch per row merges the block winners.
#include <climits>

#include "common.h"
#include "lm.h"

namespace {

constexpr int AM_SPAN = 8192;   // logits per block of the first pass

// out[b][:] = table[tokens[b]][:] as fp32 (exact: bf16 is the top half of
// fp32).  One block per row; a token outside [0, V) gives a zero row and
// raises W4_FLAG_TOKEN_ID in *err.
__global__ void __launch_bounds__(256) embed_kernel(const uint16_t* __restrict__ table,
                                                    const int32_t* __restrict__ tokens, int V, int H,
                                                    float* __restrict__ out, int* __restrict__ err) {
    const int b = blockIdx.x;
    const int t = tokens[b];
    const bool ok = t >= 0 && t < V;
    const uint2* src = reinterpret_cast<const uint2*>(table + (size_t)(ok ? t : 0) * H);
    float4* dst = reinterpret_cast<float4*>(out + (size_t)b * H);
    for (int i = threadIdx.x; i < H / 4; i += 256) {
        float4 r{0.f, 0.f, 0.f, 0.f};
        if (ok) {
            const uint2 w = src[i];
            r = float4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                       __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u)};
        }
        dst[i] = r;
    }
    if (!ok && threadIdx.x == 0) atomicOr(err, W4_FLAG_TOKEN_ID);
}

// (bv, bi) becomes (v, i) if v is larger, or equal with a lower index.  A
// NaN compares false both ways and never wins.
__device__ __forceinline__ void am_take(float& bv, int& bi, float v, int i) {
    if (v > bv || (v == bv && i < bi)) {
        bv = v;
        bi = i;
    }
}

__device__ __forceinline__ void am_wave(float& bv, int& bi) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float v = __shfl_xor(bv, off, 64);
        const int i = __shfl_xor(bi, off, 64);
        am_take(bv, bi, v, i);
    }
}

// First pass: block (j, b) reduces logits [j * AM_SPAN, min(V, (j + 1) *
// AM_SPAN)) of row b to one (value, index) pair.  V % 4 == 0.
__global__ void __launch_bounds__(256) argmax_partial_kernel(const float* __restrict__ logits, int V, int nblk,
                                                             float* __restrict__ pv, int* __restrict__ pi) {
    __shared__ float sv[4];
    __shared__ int si[4];
    const int b = blockIdx.y, j = blockIdx.x, tid = threadIdx.x;
    const float* row = logits + (size_t)b * V;
    const int lo = j * AM_SPAN, hi = min(V, lo + AM_SPAN);
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int i = lo + tid * 4; i < hi; i += 256 * 4) {
        const float4 v = *reinterpret_cast<const float4*>(row + i);
        am_take(bv, bi, v.x, i);
        am_take(bv, bi, v.y, i + 1);
        am_take(bv, bi, v.z, i + 2);
        am_take(bv, bi, v.w, i + 3);
    }
    am_wave(bv, bi);
    if ((tid & 63) == 0) {
        sv[tid >> 6] = bv;
        si[tid >> 6] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < 4; w++) am_take(bv, bi, sv[w], si[w]);
        pv[(size_t)b * nblk + j] = bv;
        pi[(size_t)b * nblk + j] = bi;
    }
}

// Second pass: one wave per row merges the nblk block winners.  A row with
// no comparable logit (all NaN) picks token 0.
__global__ void __launch_bounds__(64) argmax_final_kernel(const float* __restrict__ pv, const int* __restrict__ pi,
                                                          int nblk, int32_t* __restrict__ next) {
    const int b = blockIdx.x, l = threadIdx.x;
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int j = l; j < nblk; j += 64) am_take(bv, bi, pv[(size_t)b * nblk + j], pi[(size_t)b * nblk + j]);
    am_wave(bv, bi);
    if (l == 0) next[b] = bi == INT_MAX ? 0 : bi;
}

// The guard after a greedy pick: if any of the error words is non-zero,
// every pick of the step becomes -1.  Lane i reads word i (all in one memory
// round trip) and the wave ORs them.
constexpr int kGuardFlags = 64;
struct FlagList {
    const int* p[kGuardFlags];
    int n;
};

__global__ void __launch_bounds__(64) pick_guard_kernel(FlagList f, int32_t* __restrict__ next, int B) {
    const int lane = threadIdx.x;
    const int v = lane < f.n ? f.p[lane][0] : 0;
    if (__ballot(v != 0) == 0) return;
    for (int b = lane; b < B; b += 64) next[b] = -1;
}

}  // namespace

int launch_embed(const uint16_t* table, const int32_t* tokens, int V, int H, int B, float* out, int* err,
                 hipStream_t stream) {
    if (B < 1 || H % 4 || V < 1) return -1;
    hipLaunchKernelGGL(embed_kernel, dim3(B), dim3(256), 0, stream, table, tokens, V, H, out, err);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int argmax_blocks(int V) { return (V + AM_SPAN - 1) / AM_SPAN; }

int launch_argmax(const float* logits, int B, int V, float* pv, int* pi, int32_t* next, hipStream_t stream) {
    if (B < 1 || V < 4 || V % 4) return -1;
    const int nblk = argmax_blocks(V);
    hipLaunchKernelGGL(argmax_partial_kernel, dim3(nblk, B), dim3(256), 0, stream, logits, V, nblk, pv, pi);
    hipLaunchKernelGGL(argmax_final_kernel, dim3(B), dim3(64), 0, stream, pv, pi, nblk, next);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_pick_guard(const int* const* flags, int n, int32_t* next, int B, hipStream_t stream) {
    for (int i0 = 0; i0 < n; i0 += kGuardFlags) {
        FlagList f{};
        f.n = n - i0 < kGuardFlags ? n - i0 : kGuardFlags;
        for (int i = 0; i < f.n; i++) f.p[i] = flags[i0 + i];
        hipLaunchKernelGGL(pick_guard_kernel, dim3(1), dim3(64), 0, stream, f, next, B);
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
