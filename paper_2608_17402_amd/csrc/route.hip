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

// ---------------------------------------------------------------- fast path
//
// bf16 layers: the logits are first computed with the bf16 MFMA GEMM (every
// product of two bf16 values is exact in fp32; only the accumulation order
// differs from the FMA chain). For each (token, expert) the difference to the
// chain is bounded by (gamma_d + 4 d u) * ||x_t|| * ||w_e|| (u = 2^-24; the
// chain's own error is at most gamma_d * sum |x_i w_i|, the MFMA's at most
// 4 d u * sum |x_i w_i| under any accumulation order with per-addition error
// of 2u or less, and sum |x_i w_i| <= ||x|| ||w||). Through the sigmoid
// (1/4-Lipschitz, plus the recipe's own few-ulp error) and the bias addition
// this gives an interval around every key. The K-th largest lower end L is a
// lower bound of the true K-th key, so any expert whose upper end is below L
// cannot be selected. The remaining candidates (a dozen or so per token) are
// recomputed with the exact chain and selected exactly as on the exact path:
// indices and gates are identical bit for bit. A token with more than
// kMaxCand candidates is queued and routed by the exact all-experts kernel.

constexpr int kMaxCand = 32;

// Upper bound of the 2-norm of every row of a [rows, d] bf16 matrix (fp32 sum
// of squares, inflated to cover its rounding). One wave per row. Block 0 also
// clears the overflow counter used by the repair kernel.
__global__ __launch_bounds__(256) void k_row_norms(const bf16_t* __restrict__ a, int rows, int d,
                                                   float* __restrict__ out, int32_t* __restrict__ clear) {
    if (clear && blockIdx.x == 0 && threadIdx.x == 0) *clear = 0;
    const int lane = threadIdx.x & (kWave - 1);
    const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (row >= rows) return;
    const bf16_t* p = a + (size_t)row * d;
    float acc = 0.0f;
    for (int i = lane * 8; i < d; i += kWave * 8) {
        float v[8];
        load8(p + i, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc = fmaf(v[q], v[q], acc);
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) out[row] = sqrtf(acc) * 1.001f + 1e-30f;
}

// Candidate selection, exact recomputation of the candidates, exact top-K for
// RB consecutive tokens per block of 512 threads. The router weights stream
// through LDS in chunks of DC columns, double-buffered through registers, so
// each block reads them once; x rows of the block come along in the same
// chunks.
constexpr int kRepairThreads = 512;
constexpr int kRepairWaves = kRepairThreads / kWave;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int RB, int DC, int EMAX, int PER>
__global__ __launch_bounds__(kRepairThreads) void k_router_repair(
    const float* __restrict__ s_fast, const float* __restrict__ xnorm, const float* __restrict__ wnorm,
    const float* __restrict__ bias, const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, int T,
    int d, int E, int K, float cst, int32_t* __restrict__ topk_idx, float* __restrict__ topk_gate,
    int32_t* __restrict__ ovf_count, int32_t* __restrict__ ovf_list) {
    __shared__ uint16_t cand[RB][kMaxCand];
    __shared__ int ncand[RB];
    __shared__ int poff[RB + 1];
    __shared__ uint8_t ptok[RB * kMaxCand];
    __shared__ float sex[RB * kMaxCand];
    __shared__ __attribute__((aligned(16))) bf16_t xs[2][RB][DC];
    __shared__ __attribute__((aligned(16))) bf16_t ws[2][EMAX][DC];

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int t0 = blockIdx.x * RB;

    // Phase A: candidates of each token (a wave per token); lane l holds
    // experts l, l + 64, ... (PER of them).
    for (int tl = wave; tl < RB; tl += kRepairWaves) {
        const int t = t0 + tl;
        if (t >= T) {
            if (lane == 0) ncand[tl] = 0;
            continue;
        }
        const float xn = xnorm[t];
        float lo[PER], hi[PER];
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int e = lane + kWave * m;
            lo[m] = -INFINITY;
            hi[m] = -INFINITY;
            if (e < E) {
                const float b = bias ? bias[e] : 0.0f;
                const float key = sigmoid_fp32(s_fast[(size_t)t * E + e]) + b;
                const float delta = 0.25f * (cst * xn * wnorm[e]) + 2e-6f + 1e-6f * fabsf(b);
                lo[m] = key - delta;
                hi[m] = key + delta;
            }
        }
        // L = K-th largest lower end (a lower bound of the true K-th key).
        uint32_t taken = 0;
        float L = -INFINITY;
        for (int j = 0; j < K; ++j) {
            float bv = -INFINITY;
            int bm = -1;
#pragma unroll
            for (int m = 0; m < PER; ++m)
                if (!((taken >> m) & 1u) && lo[m] > bv) {
                    bv = lo[m];
                    bm = m;
                }
            float wvmax = bv;
#pragma unroll
            for (int off = kWave / 2; off > 0; off >>= 1) wvmax = fmaxf(wvmax, __shfl_xor(wvmax, off));
            const uint64_t holders = __ballot(bm >= 0 && bv == wvmax);
            const int first = __ffsll((unsigned long long)holders) - 1;
            if (lane == first) taken |= 1u << bm;
            L = wvmax;
        }
        // Candidates: upper end >= L, gathered in expert order.
        int nc = 0;
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const bool c = hi[m] >= L;
            const uint64_t bal = __ballot(c);
            if (c) {
                const int pos = nc + __popcll(bal & ((1ull << lane) - 1ull));
                if (pos < kMaxCand) cand[tl][pos] = (uint16_t)(lane + kWave * m);
            }
            nc += __popcll(bal);
        }
        if (nc > kMaxCand) {
            if (lane == 0) {
                const int slot = atomicAdd(ovf_count, 1);
                ovf_list[slot] = t;
            }
            nc = 0;
        }
        if (lane == 0) ncand[tl] = nc;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int tl = 0; tl < RB; ++tl) {
            poff[tl] = run;
            run += ncand[tl];
        }
        poff[RB] = run;
    }
    __syncthreads();
    for (int tl = wave; tl < RB; tl += kRepairWaves)
        for (int j = lane; j < ncand[tl]; j += kWave) ptok[poff[tl] + j] = (uint8_t)tl;
    const int P = poff[RB];

    // Phase B: exact logits of every (token, candidate) pair, one FMA chain per
    // pair over the model width in ascending order.
    constexpr int KP = RB * kMaxCand / kRepairThreads;
    constexpr int CPR = DC / 8;                       // 16-byte chunks per staged row
    constexpr int XQ = (RB * CPR + kRepairThreads - 1) / kRepairThreads;
    constexpr int WQ = (EMAX * CPR + kRepairThreads - 1) / kRepairThreads;
    float acc[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) acc[k] = 0.0f;
    u32x4_t xr[XQ], wrg[WQ];
#define MOE_FETCH(d0)                                                                                      \
    do {                                                                                                   \
        _Pragma("unroll") for (int i = 0; i < XQ; ++i) {                                                   \
            const int q = threadIdx.x + kRepairThreads * i;                                                \
            const int r = q / CPR, c = (q % CPR) * 8;                                                      \
            xr[i] = (u32x4_t){0u, 0u, 0u, 0u};                                                             \
            if (q < RB * CPR && t0 + r < T)                                                                \
                xr[i] = *reinterpret_cast<const u32x4_t*>(x + (size_t)(t0 + r) * d + (d0) + c);            \
        }                                                                                                  \
        _Pragma("unroll") for (int i = 0; i < WQ; ++i) {                                                   \
            const int q = threadIdx.x + kRepairThreads * i;                                                \
            const int r = q / CPR, c = (q % CPR) * 8;                                                      \
            if (r < E) wrg[i] = *reinterpret_cast<const u32x4_t*>(wr + (size_t)r * d + (d0) + c);         \
        }                                                                                                  \
    } while (0)
#define MOE_STASH(b)                                                                                       \
    do {                                                                                                   \
        _Pragma("unroll") for (int i = 0; i < XQ; ++i) {                                                   \
            const int q = threadIdx.x + kRepairThreads * i;                                                \
            if (q < RB * CPR) *reinterpret_cast<u32x4_t*>(&xs[b][q / CPR][(q % CPR) * 8]) = xr[i];         \
        }                                                                                                  \
        _Pragma("unroll") for (int i = 0; i < WQ; ++i) {                                                   \
            const int q = threadIdx.x + kRepairThreads * i;                                                \
            if (q / CPR < E) *reinterpret_cast<u32x4_t*>(&ws[b][q / CPR][(q % CPR) * 8]) = wrg[i];         \
        }                                                                                                  \
    } while (0)
    MOE_FETCH(0);
    MOE_STASH(0);
    __syncthreads();
    int buf = 0;
    for (int d0 = 0; d0 < d; d0 += DC) {
        if (d0 + DC < d) MOE_FETCH(d0 + DC);  // next chunk in flight during this one
#pragma unroll
        for (int k = 0; k < KP; ++k) {
            const int q = threadIdx.x + kRepairThreads * k;
            if (q < P) {
                const int tl = ptok[q];
                const int e = cand[tl][q - poff[tl]];
                float a = acc[k];
#pragma unroll
                for (int i = 0; i < DC; i += 8) {
                    float xv[8], wv[8];
                    load8(&xs[buf][tl][i], xv);
                    load8(&ws[buf][e][i], wv);
#pragma unroll
                    for (int u = 0; u < 8; ++u) a = fmaf(xv[u], wv[u], a);
                }
                acc[k] = a;
            }
        }
        if (d0 + DC < d) MOE_STASH(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }
#undef MOE_FETCH
#undef MOE_STASH
#pragma unroll
    for (int k = 0; k < KP; ++k) {
        const int q = threadIdx.x + kRepairThreads * k;
        if (q < P) sex[q] = sigmoid_fp32(acc[k]);
    }
    __syncthreads();

    // Phase C: exact top-K among the candidates and the gates (a wave per token).
    for (int tl = wave; tl < RB; tl += kRepairWaves) {
        const int t = t0 + tl;
        const int nc = ncand[tl];
        if (t >= T || nc == 0) continue;  // overflow tokens are routed by the exact kernel
        const int e = lane < nc ? (int)cand[tl][lane] : 0x7fffffff;
        const float sg = lane < nc ? sex[poff[tl] + lane] : 0.0f;
        const float key = lane < nc ? (bias ? sg + bias[e] : sg) : -INFINITY;
        bool taken = false;
        float csig[kMaxK];
        int cidx[kMaxK];
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            csig[j] = 0.0f;
            cidx[j] = 0;
            if (j >= K) continue;
            float bk = taken ? -INFINITY : key;
            int be = taken ? 0x7fffffff : e;
            float bs = sg;
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
            if (be == e && lane < nc) taken = true;
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
        for (int j = 0; j < kMaxK; ++j)
            if (j == lane && j < K) {
                my_e = cidx[j];
                my_g = csig[j] / den;
            }
        if (lane < K) {
            topk_idx[(size_t)t * K + lane] = my_e;
            topk_gate[(size_t)t * K + lane] = my_g;
        }
    }
}

// Exact routing of the queued tokens: all E logits by the FMA chain, then
// the same top-K. Persistent blocks walk the queue; every block exits once
// the queue (fixed by the time this kernel starts) is exhausted.
__global__ __launch_bounds__(256) void k_router_exact_list(const bf16_t* __restrict__ x,
                                                          const bf16_t* __restrict__ wr,
                                                          const float* __restrict__ bias, int d, int E, int K,
                                                          const int32_t* __restrict__ ovf_count,
                                                          const int32_t* __restrict__ ovf_list,
                                                          int32_t* __restrict__ topk_idx,
                                                          float* __restrict__ topk_gate) {
    __shared__ float sig[kMaxE];
    const int n = *ovf_count;
    const int lane = threadIdx.x & (kWave - 1);
    for (int it = blockIdx.x; it < n; it += gridDim.x) {
        const int t = ovf_list[it];
        const bf16_t* xt = x + (size_t)t * d;
        for (int e = threadIdx.x; e < E; e += blockDim.x) {
            const bf16_t* we = wr + (size_t)e * d;
            float a = 0.0f;
            for (int i = 0; i < d; i += 8) {
                float xv[8], wv[8];
                load8(xt + i, xv);
                load8(we + i, wv);
#pragma unroll
                for (int u = 0; u < 8; ++u) a = fmaf(xv[u], wv[u], a);
            }
            sig[e] = sigmoid_fp32(a);
        }
        __syncthreads();
        if (threadIdx.x < kWave) {
            const int per = (E + kWave - 1) / kWave;
            float sg[kPerLane], key[kPerLane];
#pragma unroll
            for (int m = 0; m < kPerLane; ++m) {
                const int e = lane + kWave * m;
                const bool ok = m < per && e < E;
                sg[m] = ok ? sig[e] : 0.0f;
                key[m] = ok ? (bias ? sg[m] + bias[e] : sg[m]) : -INFINITY;
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
                    if (m < per && e < E && !((taken >> m) & 1u) && (key[m] > bk || (key[m] == bk && e < be))) {
                        bk = key[m];
                        be = e;
                        bs = sg[m];
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
            for (int j = 0; j < kMaxK; ++j)
                if (j == lane && j < K) {
                    my_e = cidx[j];
                    my_g = csig[j] / den;
                }
            if (lane < K) {
                topk_idx[(size_t)t * K + lane] = my_e;
                topk_gate[(size_t)t * K + lane] = my_g;
            }
        }
        __syncthreads();
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

namespace moe {

float router_fast_bound_constant(int d) {
    const double u = 1.0 / 16777216.0;
    const double gamma = d * u / (1.0 - d * u);
    return (float)((gamma + 4.0 * d * u) * 1.01);
}

hipError_t launch_router_fast_finish(const moe_desc_t& d, const float* s_fast, const void* x,
                                     const void* w_router, const float* bias, float* xnorm, float* wnorm,
                                     int32_t* ovf_count, int32_t* ovf_list, int32_t* topk_idx,
                                     float* topk_gate, hipStream_t s) {
    const bf16_t* xb = static_cast<const bf16_t*>(x);
    const bf16_t* wb = static_cast<const bf16_t*>(w_router);
    hipLaunchKernelGGL(k_row_norms, dim3((d.T + 3) / 4), dim3(256), 0, s, xb, d.T, d.d, xnorm, ovf_count);
    hipLaunchKernelGGL(k_row_norms, dim3((d.E + 3) / 4), dim3(256), 0, s, wb, d.E, d.d, wnorm, nullptr);
    const float cst = router_fast_bound_constant(d.d);
    // Blocks of 128 tokens for large batches (router weights streamed once per
    // block), 32 for small ones (enough blocks to fill the GPU). Router weight
    // chunks of 32 columns while E <= 256, else 16.
#define MOE_REPAIR(RBv, DCv, EMv, PERv)                                                                    \
    hipLaunchKernelGGL((k_router_repair<RBv, DCv, EMv, PERv>), dim3((d.T + RBv - 1) / RBv), dim3(kRepairThreads), \
                       0, s, s_fast, xnorm, wnorm, bias, xb, wb, d.T, d.d, d.E, d.K, cst, topk_idx, topk_gate,  \
                       ovf_count, ovf_list)
    const bool big = d.T >= 16384;
    const int per = (d.E + kWave - 1) / kWave;
    if (per <= 1) { if (big) MOE_REPAIR(128, 32, 256, 1); else MOE_REPAIR(32, 32, 256, 1); }
    else if (per <= 2) { if (big) MOE_REPAIR(128, 32, 256, 2); else MOE_REPAIR(32, 32, 256, 2); }
    else if (per <= 4) { if (big) MOE_REPAIR(128, 32, 256, 4); else MOE_REPAIR(32, 32, 256, 4); }
    else if (per <= 8) { if (big) MOE_REPAIR(128, 16, 512, 8); else MOE_REPAIR(32, 16, 512, 8); }
    else { if (big) MOE_REPAIR(128, 16, 1024, 16); else MOE_REPAIR(32, 16, 1024, 16); }
#undef MOE_REPAIR
    hipLaunchKernelGGL(k_router_exact_list, dim3(64), dim3(256), 0, s, xb, wb, bias, d.d, d.E, d.K, ovf_count,
                       ovf_list, topk_idx, topk_gate);
    return hipGetLastError();
}

}  // namespace moe
