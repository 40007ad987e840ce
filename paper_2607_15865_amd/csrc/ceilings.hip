// Ceiling kernels (measurement): what the device sustains on the two
// resources the stages are bound by, measured on the box beside the
// published peaks (clocks may be capped under power).
//   * a pure streaming read of a device buffer (16-byte loads, 8 in flight
//     per thread), XOR-folded into one word per thread so that no load is
//     dead;
//   * a pure MFMA loop: the 16x16x32 fp16 MFMA of the layer's GEMV and the
//     32x32x16 fp16 MFMA of its GEMM, on 4 independent accumulators per
//     wave, with operands that change every iteration.
#include "common.h"

namespace {

constexpr int READ_THREADS = 256;
constexpr int READ_UNROLL = 8;

__global__ void __launch_bounds__(READ_THREADS) ceiling_read_kernel(const u32x4* __restrict__ src, size_t n16,
                                                                     uint32_t* __restrict__ sink) {
    const size_t stride = (size_t)gridDim.x * READ_THREADS;
    size_t i = (size_t)blockIdx.x * READ_THREADS + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (READ_UNROLL - 1) * stride < n16; i += READ_UNROLL * stride) {
        u32x4 v[READ_UNROLL];
#pragma unroll
        for (int u = 0; u < READ_UNROLL; u++) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < READ_UNROLL; u++) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < n16; i += stride) {
        const u32x4 v = src[i];
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    sink[(size_t)blockIdx.x * READ_THREADS + threadIdx.x] = acc;
}

template <bool BIG>
__global__ void __launch_bounds__(256) ceiling_mfma_kernel(float* __restrict__ sink, int iters) {
    const int lane = threadIdx.x & 63;
    f16x8 a = {}, b = {};
#pragma unroll
    for (int j = 0; j < 8; j++) {
        a[j] = (f16)(0.001f * (lane + j));
        b[j] = (f16)(0.002f * (lane - j));
    }
    const f16x8 da = a * (f16)0.5f, db = b * (f16)0.25f;
    float out = 0.f;
    if constexpr (BIG) {
        f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
        for (int it = 0; it < iters; it += 2) {     // operands toggle between two values
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(b, a, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, db, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(da, b, c3, 0, 0, 0);
            a += da;
            b += db;
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(b, a, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, db, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(da, b, c3, 0, 0, 0);
            a -= da;
            b -= db;
        }
#pragma unroll
        for (int e = 0; e < 16; e++) out += c0[e] + c1[e] + c2[e] + c3[e];
    } else {
        f32x4 c0 = {}, c1 = {}, c2 = {}, c3 = {};
        for (int it = 0; it < iters; it += 2) {     // operands toggle between two values
            c0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b, a, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, db, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_16x16x32_f16(da, b, c3, 0, 0, 0);
            a += da;
            b += db;
            c0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b, a, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, db, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_16x16x32_f16(da, b, c3, 0, 0, 0);
            a -= da;
            b -= db;
        }
#pragma unroll
        for (int e = 0; e < 4; e++) out += c0[e] + c1[e] + c2[e] + c3[e];
    }
    sink[(size_t)blockIdx.x * 256 + threadIdx.x] = out;
}

}  // namespace

extern "C" int w4_ceiling_read(const void* buf, size_t bytes, uint32_t* sink, int32_t blocks, void* stream) {
    if (!buf || !sink || blocks < 1 || bytes < 16 || (reinterpret_cast<uintptr_t>(buf) & 15)) return W4_EINVAL;
    hipLaunchKernelGGL(ceiling_read_kernel, dim3(blocks), dim3(READ_THREADS), 0, (hipStream_t)stream,
                       reinterpret_cast<const u32x4*>(buf), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? W4_OK : W4_EHIP;
}

extern "C" int w4_ceiling_mfma(float* sink, int32_t blocks, int32_t iters, int32_t big, double* flop, void* stream) {
    if (!sink || !flop || blocks < 1 || iters < 2 || iters % 2) return W4_EINVAL;
    // 4 waves per block, 4 MFMAs per iteration and wave
    const double per = big ? 2.0 * 32 * 32 * 16 : 2.0 * 16 * 16 * 32;
    *flop = per * 4.0 * 4.0 * (double)blocks * (double)iters;
    if (big) hipLaunchKernelGGL(ceiling_mfma_kernel<true>, dim3(blocks), dim3(256), 0, (hipStream_t)stream, sink, iters);
    else hipLaunchKernelGGL(ceiling_mfma_kernel<false>, dim3(blocks), dim3(256), 0, (hipStream_t)stream, sink, iters);
    return hipGetLastError() == hipSuccess ? W4_OK : W4_EHIP;
}
