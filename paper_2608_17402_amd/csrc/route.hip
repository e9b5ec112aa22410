// Router and gating for gfx950 (paper Sec. 3.1 Eq. (1); Sec. 3.2 Eqs. (4)-(5)
// sigmoid gating with renormalisation; Sec. 3.2 "Load Balancing" Eq. (7):
// the bias b is added to the sigmoid score for selection only).
//
// Routing decides integers, so it is computed reproducibly in fp32:
//   logit  = one fused multiply-add chain over i = 0..d-1, ascending, from +0
//   sigmoid = 1 / (1 + exp(-s)), exp by Cody-Waite reduction and a degree-7
//             Taylor polynomial, using only correctly rounded operations.
// This file is compiled with -ffp-contract=off so the compiler cannot fuse or
// reorder any of these steps.
#include "moe_internal.h"

#include <math.h>

namespace moe {
namespace {

// exp(z) = 2^n * exp(r), n = rint(z / ln 2), r = z - n ln 2 in two steps with
// ln 2 split into a 15-bit head (22713 * 2^-15, so n * head is exact for
// |n| <= 126) and the fp32-rounded remainder.
constexpr float kLog2e = 0x1.715476p+0f;   // fl32(1 / ln 2)
constexpr float kLn2Head = 0x1.62e4p-1f;   // 22713 * 2^-15
constexpr float kLn2Tail = 0x1.7f7d1cp-20f;  // fl32(ln 2 - head)

__device__ __forceinline__ float sigmoid_fp32(float s) {
    // Taylor coefficients 1/k!, each the correctly rounded fp32 quotient.
    const float q2 = 1.0f / 2.0f, q3 = 1.0f / 6.0f, q4 = 1.0f / 24.0f;
    const float q5 = 1.0f / 120.0f, q6 = 1.0f / 720.0f, q7 = 1.0f / 5040.0f;
    float z = -s;
    // Clamp so exp(z) and the quotient stay normal numbers (|z| <= 87).
    z = z > 87.0f ? 87.0f : z;
    z = z < -87.0f ? -87.0f : z;
    const float n = rintf(z * kLog2e);
    float r = fmaf(-n, kLn2Head, z);
    r = fmaf(-n, kLn2Tail, r);
    float p = fmaf(q7, r, q6);
    p = fmaf(p, r, q5);
    p = fmaf(p, r, q4);
    p = fmaf(p, r, q3);
    p = fmaf(p, r, q2);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    const float ez = ldexpf(p, (int)n);
    return 1.0f / (1.0f + ez);
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

// Eight consecutive elements starting at p (16-byte aligned for bf16, two
// 16-byte loads for fp32), widened to fp32.
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[2 * q] = __uint_as_float(w[q] << 16);
        v[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8(const float* p, float* v) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Sigmoid scores of a 64-token x 64-expert tile. Each thread owns 4 tokens
// (ty + 16 r) x 4 experts (tx + 16 c); every accumulator is a sequential FMA
// chain over the model width, fed from fp32 LDS tiles of 32 columns.
constexpr int RT_TOK = 64, RT_EXP = 64, RT_DK = 32, RT_PAD = 4;

template <typename TIn>
__global__ __launch_bounds__(256) void k_router_scores(const TIn* __restrict__ x,
                                                      const TIn* __restrict__ wr,
                                                      float* __restrict__ scores, int T, int d,
                                                      int E) {
    __shared__ __attribute__((aligned(16))) float xs[RT_TOK][RT_DK + RT_PAD];
    __shared__ __attribute__((aligned(16))) float ws[RT_EXP][RT_DK + RT_PAD];
    const int tid = threadIdx.x;
    const int t0 = blockIdx.x * RT_TOK;
    const int e0 = blockIdx.y * RT_EXP;
    const int tx = tid & 15, ty = tid >> 4;
    float acc[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = 0.0f;

    const int lr = tid >> 2, lc = (tid & 3) * 8;  // this thread's 8 loaded columns
    const int xt = t0 + lr, we = e0 + lr;
    for (int k0 = 0; k0 < d; k0 += RT_DK) {
        float v[8];
        if (xt < T) {
            load8(x + (size_t)xt * d + k0 + lc, v);
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) xs[lr][lc + q] = v[q];
        if (we < E) {
            load8(wr + (size_t)we * d + k0 + lc, v);
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) ws[lr][lc + q] = v[q];
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < RT_DK; kk += 4) {
            float4 xv[4], wv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) xv[r] = *reinterpret_cast<const float4*>(&xs[ty + 16 * r][kk]);
#pragma unroll
            for (int c = 0; c < 4; ++c) wv[c] = *reinterpret_cast<const float4*>(&ws[tx + 16 * c][kk]);
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    // ascending column order within the chunk
                    acc[r][c] = fmaf(xv[r].x, wv[c].x, acc[r][c]);
                    acc[r][c] = fmaf(xv[r].y, wv[c].y, acc[r][c]);
                    acc[r][c] = fmaf(xv[r].z, wv[c].z, acc[r][c]);
                    acc[r][c] = fmaf(xv[r].w, wv[c].w, acc[r][c]);
                }
        }
        __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int t = t0 + ty + 16 * r;
        if (t >= T) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int e = e0 + tx + 16 * c;
            if (e < E) scores[(size_t)t * E + e] = sigmoid_fp32(acc[r][c]);
        }
    }
}

// Top-K selection and gates, one wavefront per token. Lane l holds experts
// l, l + 64, ...; each of the K rounds takes the wave-wide best (key
// descending, expert index ascending on equal keys) with a butterfly of
// cross-lane exchanges, then the owner lane marks it taken.
constexpr int kPerLane = kMaxE / kWave;

__global__ __launch_bounds__(256) void k_topk(const float* __restrict__ scores,
                                             const float* __restrict__ bias, int T, int E, int K,
                                             int32_t* __restrict__ topk_idx,
                                             float* __restrict__ topk_gate) {
    const int lane = threadIdx.x & (kWave - 1);
    const int t = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (t >= T) return;  // uniform per wave
    const int per = (E + kWave - 1) / kWave;
    float sig[kPerLane], key[kPerLane];
#pragma unroll
    for (int m = 0; m < kPerLane; ++m) {
        const int e = lane + kWave * m;
        const bool ok = m < per && e < E;
        sig[m] = ok ? scores[(size_t)t * E + e] : 0.0f;
        key[m] = ok ? (bias ? sig[m] + bias[e] : sig[m]) : -INFINITY;
    }
    uint32_t taken = 0;
    float csig[kMaxK];
    int cidx[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        csig[j] = 0.0f;
        cidx[j] = 0;
        if (j >= K) continue;
        float bk = -INFINITY;
        int be = 0x7fffffff;
        float bs = 0.0f;
#pragma unroll
        for (int m = 0; m < kPerLane; ++m) {
            const int e = lane + kWave * m;
            if (m < per && e < E && !((taken >> m) & 1u)) {
                if (key[m] > bk || (key[m] == bk && e < be)) {
                    bk = key[m];
                    be = e;
                    bs = sig[m];
                }
            }
        }
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const float ok = __shfl_xor(bk, off);
            const int oe = __shfl_xor(be, off);
            const float os = __shfl_xor(bs, off);
            if (ok > bk || (ok == bk && oe < be)) {
                bk = ok;
                be = oe;
                bs = os;
            }
        }
        if ((be & (kWave - 1)) == lane) taken |= 1u << (be / kWave);
        csig[j] = bs;
        cidx[j] = be;
    }
    float den = csig[0];
#pragma unroll
    for (int j = 1; j < kMaxK; ++j)
        if (j < K) den = den + csig[j];
    int my_e = 0;
    float my_g = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        if (j == lane && j < K) {
            my_e = cidx[j];
            my_g = csig[j] / den;
        }
    }
    if (lane < K) {
        topk_idx[(size_t)t * K + lane] = my_e;
        topk_gate[(size_t)t * K + lane] = my_g;
    }
}

}  // namespace

hipError_t launch_router_scores(const moe_desc_t& d, const void* x, const void* w_router,
                                float* scores, hipStream_t s) {
    dim3 grid((d.T + RT_TOK - 1) / RT_TOK, (d.E + RT_EXP - 1) / RT_EXP);
    if (d.dtype == MOE_BF16)
        hipLaunchKernelGGL(k_router_scores<bf16_t>, grid, dim3(256), 0, s,
                           static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w_router), scores,
                           d.T, d.d, d.E);
    else
        hipLaunchKernelGGL(k_router_scores<float>, grid, dim3(256), 0, s, static_cast<const float*>(x),
                           static_cast<const float*>(w_router), scores, d.T, d.d, d.E);
    return hipGetLastError();
}

hipError_t launch_topk(const moe_desc_t& d, const float* scores, const float* bias,
                       int32_t* topk_idx, float* topk_gate, hipStream_t s) {
    const int per_block = 256 / kWave;
    dim3 grid((d.T + per_block - 1) / per_block);
    hipLaunchKernelGGL(k_topk, grid, dim3(256), 0, s, scores, bias, d.T, d.E, d.K, topk_idx, topk_gate);
    return hipGetLastError();
}

}  // namespace moe
