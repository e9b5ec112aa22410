// Gate-weighted combine back to token order (paper Sec. 3.2 Eq. (6)):
//   y[t] = sum_j gate[t, j] * expert_out[t*K + j] + lambda * shared[t]
// expert_out is in slot order, so one token's K rows are contiguous. Each
// thread owns 8 consecutive columns of one token, reads each of the K rows
// with one 16-byte load (bf16) and accumulates in fp32 in slot order, then
// adds the shared expert: deterministic, no atomics.
#include "moe_internal.h"

namespace moe {
namespace {

__device__ __forceinline__ void ld8(const bf16_t* p, float* v) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[2 * q] = __uint_as_float(w[q] << 16);
        v[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
}
__device__ __forceinline__ void ld8(const float* p, float* v) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    uint32_t a = __float_as_uint(lo), b = __float_as_uint(hi);
    a += 0x7fffu + ((a >> 16) & 1u);
    b += 0x7fffu + ((b >> 16) & 1u);
    return (a >> 16) | (b & 0xffff0000u);
}
__device__ __forceinline__ void st8(bf16_t* p, const float* v) {
    uint4 u;
    u.x = pack_bf16(v[0], v[1]);
    u.y = pack_bf16(v[2], v[3]);
    u.z = pack_bf16(v[4], v[5]);
    u.w = pack_bf16(v[6], v[7]);
    *reinterpret_cast<uint4*>(p) = u;
}
__device__ __forceinline__ void st8(float* p, const float* v) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

template <typename TE, typename TS>
__global__ __launch_bounds__(256) void k_combine(const TE* __restrict__ eo, const float* __restrict__ gate,
                                                const TS* __restrict__ sh, float lambda,
                                                TE* __restrict__ y, int T, int d, int K) {
    const int per_tok = d / 8;
    const long long item = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const int t = (int)(item / per_tok);
    if (t >= T) return;
    const int c0 = (int)(item - (long long)t * per_tok) * 8;
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.0f;
    for (int j = 0; j < K; ++j) {
        const float g = gate[(size_t)t * K + j];
        float v[8];
        ld8(eo + ((size_t)t * K + j) * d + c0, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] = fmaf(g, v[q], acc[q]);
    }
    if (sh) {
        float v[8];
        ld8(sh + (size_t)t * d + c0, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] = fmaf(lambda, v[q], acc[q]);
    }
    st8(y + (size_t)t * d + c0, acc);
}

}  // namespace

hipError_t launch_combine(const moe_desc_t& d, const void* expert_out, const float* gate,
                          const void* shared, int shared_is_f32, void* y, hipStream_t s) {
    const long long items = (long long)d.T * (d.d / 8);
    const dim3 grid((unsigned)((items + 255) / 256));
    if (d.dtype == MOE_BF16) {
        const bf16_t* eo = static_cast<const bf16_t*>(expert_out);
        if (shared_is_f32)
            hipLaunchKernelGGL((k_combine<bf16_t, float>), grid, dim3(256), 0, s, eo, gate,
                               static_cast<const float*>(shared), d.lambda, static_cast<bf16_t*>(y), d.T,
                               d.d, d.K);
        else
            hipLaunchKernelGGL((k_combine<bf16_t, bf16_t>), grid, dim3(256), 0, s, eo, gate,
                               static_cast<const bf16_t*>(shared), d.lambda, static_cast<bf16_t*>(y), d.T,
                               d.d, d.K);
    } else {
        hipLaunchKernelGGL((k_combine<float, float>), grid, dim3(256), 0, s,
                           static_cast<const float*>(expert_out), gate, static_cast<const float*>(shared),
                           d.lambda, static_cast<float*>(y), d.T, d.d, d.K);
    }
    return hipGetLastError();
}

}  // namespace moe
