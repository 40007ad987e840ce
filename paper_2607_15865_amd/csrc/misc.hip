// Row RMSNorm (prefill), the in-place KV append, and the debug dequantiser.
#include "common.h"
#include "launch.h"

namespace {

// top.RMSNorm (Sec. 2.2): y = x / sqrt(mean(x^2) + eps) * gamma over a row,
// rounded to bf16 and held as fp16 (the matmul operand).  One block of 256
// threads per row.  NV: 16-byte chunks of the row per thread (H <= NV * 1024),
// kept in registers between the sum of squares and the output.
template <int NV>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, const uint16_t* __restrict__ gamma,
                                                      float eps, int H, f16* __restrict__ out,
                                                      int* __restrict__ err) {
    __shared__ float part[4];
    const int row = blockIdx.x, tid = threadIdx.x;
    const float* xr = x + (size_t)row * H;
    float4 v[NV];
    uint2 g[NV];
#pragma unroll
    for (int j = 0; j < NV; j++) {
        const int k = (tid + 256 * j) * 4;
        v[j] = k < H ? *reinterpret_cast<const float4*>(xr + k) : float4{0.f, 0.f, 0.f, 0.f};
        g[j] = k < H ? *reinterpret_cast<const uint2*>(gamma + k) : uint2{0u, 0u};
    }
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NV; j++) ss += (v[j].x * v[j].x + v[j].y * v[j].y) + (v[j].z * v[j].z + v[j].w * v[j].w);
    ss = wave_sum(ss);
    if ((tid & 63) == 0) part[tid >> 6] = ss;
    __syncthreads();
    const float tot = part[0] + part[1] + part[2] + part[3];
    const float rinv = 1.0f / sqrtf(tot / (float)H + eps);
    f16* orow = out + (size_t)row * H;
    bool bad = false;
#pragma unroll
    for (int j = 0; j < NV; j++) {
        const int k = (tid + 256 * j) * 4;
        if (k >= H) break;
        f16 o[4];
        o[0] = act_f16(v[j].x * rinv * __uint_as_float(g[j].x << 16), bad);
        o[1] = act_f16(v[j].y * rinv * __uint_as_float(g[j].x & 0xFFFF0000u), bad);
        o[2] = act_f16(v[j].z * rinv * __uint_as_float(g[j].y << 16), bad);
        o[3] = act_f16(v[j].w * rinv * __uint_as_float(g[j].y & 0xFFFF0000u), bad);
        *reinterpret_cast<uint2*>(orow + k) = *reinterpret_cast<const uint2*>(o);
    }
    flag_range(err, bad);
}

struct SlotStarts { int32_t v[64]; };

// Copy new K/V rows [B][T][nkv][d] into cache slots start_b + t.
__global__ void kv_append_kernel(uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                 const uint16_t* __restrict__ kn, const uint16_t* __restrict__ vn,
                                 int B, int T, int nkv, int d, long long sb, long long sh, SlotStarts st) {
    const int segs = d / 8;
    const long long total = (long long)B * T * nkv * segs;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const int seg = (int)(i % segs);
        long long r = i / segs;
        const int g = (int)(r % nkv); r /= nkv;
        const int t = (int)(r % T);
        const int b = (int)(r / T);
        const size_t src = (((size_t)b * T + t) * nkv + g) * d + seg * 8;
        const size_t dst = (size_t)b * sb + (size_t)g * sh + (size_t)(st.v[b] + t) * d + seg * 8;
        *reinterpret_cast<u32x4*>(kc + dst) = *reinterpret_cast<const u32x4*>(kn + src);
        *reinterpret_cast<u32x4*>(vc + dst) = *reinterpret_cast<const u32x4*>(vn + src);
    }
}

// out[k][n] = s * (code - zero) for logical column n (device column
// col_map[n]), read from the tiled layout with the same unpacking as the
// stage kernels.
__global__ void debug_dequant_kernel(DevLinear W, const int32_t* __restrict__ col_map, int K, int N,
                                     float* __restrict__ out) {
    const long long total = (long long)K * N;
    const int KB = W.K_pad / 64;
    for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const int k = (int)(i / N), n = (int)(i % N);
        const int nd = col_map[n];
        const int nt = nd / 32, cc = nd % 32;
        const int kb = k / 64, kr = k % 64;
        const int s = kr / 16, hh = (kr % 16) / 8, j = kr % 8;
        const int lane = hh * 32 + cc;
        const int g = k >> W.lgG;
        const size_t gi = (size_t)g * W.N_dev + nd;
        const size_t tile = ((size_t)nt * KB + kb) * (256u << W.wf);      // words
        f16x8 v8;
        if (W.wf == WF_INT8) {
            const uint32_t* w = W.qw + tile + ((size_t)(s / 2) * 64 + lane) * 4 + 2 * (s % 2);
            const f16 zn = (f16)(-(1024.0f + (float)W.zeros[gi]));
            v8 = dequant8_u8(w[0], w[1], f16x2{zn, zn});
        } else if (W.wf == WF_F16) {
            const uint32_t* w = W.qw + tile + ((size_t)s * 64 + lane) * 4;
            v8 = f16_frag(w[0], w[1], w[2], w[3]);
        } else {
            const uint32_t w = W.qw[tile + (size_t)lane * 4 + s];
            v8 = dequant8(w, zero_off(W.zeros ? (float)W.zeros[gi] : 8.0f), dq_const());
        }
        f16 vals[8];
        __builtin_memcpy(vals, &v8, sizeof vals);
        const float qz = (float)vals[j];
        const float sc = (float)__builtin_bit_cast(f16, W.scales[gi]);
        out[i] = qz * sc;
    }
}

}  // namespace

int launch_rmsnorm(const float* x, const uint16_t* gamma, float eps, int M, int H, f16* out, int* err,
                   hipStream_t stream) {
    if (H % 4 || H > 16 * 1024) return -1;
    const int nv = (H + 1023) / 1024;
    if (nv <= 1) hipLaunchKernelGGL(rmsnorm_kernel<1>, dim3(M), dim3(256), 0, stream, x, gamma, eps, H, out, err);
    else if (nv <= 2) hipLaunchKernelGGL(rmsnorm_kernel<2>, dim3(M), dim3(256), 0, stream, x, gamma, eps, H, out, err);
    else if (nv <= 4) hipLaunchKernelGGL(rmsnorm_kernel<4>, dim3(M), dim3(256), 0, stream, x, gamma, eps, H, out, err);
    else if (nv <= 8) hipLaunchKernelGGL(rmsnorm_kernel<8>, dim3(M), dim3(256), 0, stream, x, gamma, eps, H, out, err);
    else hipLaunchKernelGGL(rmsnorm_kernel<16>, dim3(M), dim3(256), 0, stream, x, gamma, eps, H, out, err);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_kv_append(uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_new, const uint16_t* v_new,
                     int B, int T, int nkv, int d, long long stride_b, long long stride_h,
                     const int32_t* slot_start_host, hipStream_t stream) {
    SlotStarts st;
    for (int b = 0; b < 64; b++) st.v[b] = b < B ? slot_start_host[b] : 0;
    const long long total = (long long)B * T * nkv * (d / 8);
    int blocks = (int)((total + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(kv_append_kernel, dim3(blocks), dim3(256), 0, stream, k_cache, v_cache, k_new, v_new,
                       B, T, nkv, d, stride_b, stride_h, st);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_debug_dequant(const DevLinear& W, const int32_t* col_map, int K, int N, float* out, hipStream_t stream) {
    const long long total = (long long)K * N;
    int blocks = (int)((total + 255) / 256);
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(debug_dequant_kernel, dim3(blocks), dim3(256), 0, stream, W, col_map, K, N, out);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
