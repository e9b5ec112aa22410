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
#include "gemm_device.h"
#include "moe_internal.h"

#include <math.h>

#include <type_traits>
#include <utility>

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
// indices and gates are identical bit for bit. A token with more candidates
// than its slots (16, or 32 when K > 8) is queued and routed by the exact
// all-experts kernel.
//
// The interval test itself uses a cheap sigmoid (hardware exp2 and
// reciprocal, absolute error below 1e-6 for every input, covered by extra
// slack in the half-width); only the candidates go through recipe S.

__device__ __forceinline__ float sigmoid_fast(float s) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-s * kLog2e));
}

// Upper bound of the 2-norm of every row of a [rows, d] bf16 matrix (fp32 sum
// of squares, inflated to cover its rounding). One wave per row. Block 0 also
// clears the overflow counter used by the repair kernel.
__global__ __launch_bounds__(256) void k_row_norms(const bf16_t* __restrict__ a, int rows_a,
                                                   float* __restrict__ out_a, const bf16_t* __restrict__ b,
                                                   int rows_b, float* __restrict__ out_b, int d,
                                                   int32_t* __restrict__ clear, float* __restrict__ a32) {
    if (clear && blockIdx.x == 0 && threadIdx.x == 0) *clear = 0;
    const int lane = threadIdx.x & (kWave - 1);
    // One wave per row: the rows of a, then (from the next block on) those of b.
    const int wpb = blockDim.x / kWave;
    const int blocks_a = (rows_a + wpb - 1) / wpb;
    const bool second = (int)blockIdx.x >= blocks_a;
    const int row = ((int)blockIdx.x - (second ? blocks_a : 0)) * wpb + threadIdx.x / kWave;
    if (row >= (second ? rows_b : rows_a)) return;
    const bf16_t* p = (second ? b : a) + (size_t)row * d;
    float* out = second ? out_b : out_a;
    float acc = 0.0f;
    // a32 (optional): the rows of a widened to fp32 (exact), for the
    // small-batch chain kernel.
    float* const r32 = (a32 && !second) ? a32 + (size_t)row * d : nullptr;
    for (int i = lane * 8; i < d; i += kWave * 8) {
        float v[8];
        load8(p + i, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc = fmaf(v[q], v[q], acc);
        if (r32) {
            *reinterpret_cast<float4*>(r32 + i) = make_float4(v[0], v[1], v[2], v[3]);
            *reinterpret_cast<float4*>(r32 + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
        }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) out[row] = sqrtf(acc) * 1.001f + 1e-30f;
}

// Maximum over each aligned group of 16 lanes (a DPP row), in every lane of
// the group: swaps inside quads (xor 1, xor 2), then the mirror inside each
// half row and the mirror of the whole row.
template <int CTRL>
__device__ __forceinline__ float dpp_max(float a) {
    return fmaxf(a, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), CTRL, 0xF, 0xF, false)));
}
__device__ __forceinline__ float row16_max(float v) {
    v = dpp_max<0xB1>(v);   // quad_perm [1, 0, 3, 2]
    v = dpp_max<0x4E>(v);   // quad_perm [2, 3, 0, 1]
    v = dpp_max<0x141>(v);  // row_half_mirror
    v = dpp_max<0x140>(v);  // row_mirror
    return v;
}

// Maximum over each aligned group of LPA lanes (16 or 64).
template <int LPA>
__device__ __forceinline__ float group_max(float v) {
    static_assert(LPA == 16 || LPA == 64, "groups of 16 or 64 lanes");
    v = row16_max(v);
    if constexpr (LPA == 64) {
        v = fmaxf(v, __shfl_xor(v, 16));
        v = fmaxf(v, __shfl_xor(v, 32));
    }
    return v;
}

// PER consecutive floats from a 16-byte aligned address.
template <int PER>
__device__ __forceinline__ void load_row(const float* p, float (&v)[PER]) {
#pragma unroll
    for (int i = 0; i < PER / 4; ++i) {
        const float4 q = *reinterpret_cast<const float4*>(p + 4 * i);
        v[4 * i] = q.x;
        v[4 * i + 1] = q.y;
        v[4 * i + 2] = q.z;
        v[4 * i + 3] = q.w;
    }
}

// Candidates of each token: LPA lanes per token, lane g holding experts
// g PER .. g PER + PER - 1 (contiguous, so that its logits are PER / 4
// 16-byte loads); the MFMA logits have rows of ld >= E (a multiple of 64), in
// nsplit partial arrays (split K) sstride floats apart. L = the K-th largest
// lower end of the key intervals; the candidates are the experts whose upper
// end reaches L, written to cand[t][0 .. NS) (in no particular order) with
// their count in ncand[t]. A token with more than NS candidates gets
// ncand = -1 and is appended to the overflow queue.
template <int LPA, int PER, int NS, bool SPLIT>
__global__ __launch_bounds__(256) void k_router_cand(const float* __restrict__ s_fast,
                                                    const bf16_t* __restrict__ x,
                                                    const float* __restrict__ xnorm2, int d,
                                                    const float* __restrict__ wnorm,
                                                    const float* __restrict__ bias, int T, int E, int ld,
                                                    int K, float cst, uint16_t* __restrict__ cand,
                                                    int32_t* __restrict__ ncand, int32_t* __restrict__ ovf_count,
                                                    int32_t* __restrict__ ovf_list, int nsplit, size_t sstride) {
    static_assert(LPA <= kWave && kWave % LPA == 0, "token groups inside a wave");
    static_assert(PER % 4 == 0 && 64 % PER == 0, "whole 16-byte loads inside a row of a multiple of 64");
    const int lane = threadIdx.x & (kWave - 1);
    const int g = lane % LPA;
    const int t = blockIdx.x * (blockDim.x / LPA) + threadIdx.x / LPA;
    const bool live = t < T;  // uniform within the group: dead groups compute on -inf
    const uint64_t grp = (LPA == kWave ? ~0ull : ((1ull << LPA) - 1ull)) << (lane - g);

    // Selection biases and weight-row norms of all experts, in LDS.
    static_assert(LPA * PER <= kMaxE, "the lanes' experts inside the arrays");
    __shared__ __attribute__((aligned(16))) float sb[kMaxE];
    __shared__ __attribute__((aligned(16))) float swn[kMaxE];
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        sb[e] = bias ? bias[e] : 0.0f;
        swn[e] = wnorm[e];
    }

    // ||x_t||, raised by 0.1 % as k_row_norms does for the weight rows (an
    // upper bound is all the interval needs; the rounding of the sum of
    // squares, in any order, is far inside that margin). The sum of squares
    // comes from the logits GEMM (xnorm2) or, without it, from the token's
    // LPA lanes reading its row in 16-byte pieces and adding their partial
    // sums.
    float ss = 0.0f;
    if (xnorm2) {
        ss = live ? xnorm2[t] : 0.0f;
    } else {
        if (live) {
            // Four pieces per round, all loaded before the adds.
            const bf16_t* xr = x + (size_t)t * d;
            for (int i = g * 8; i < d; i += 4 * LPA * 8) {
                float v[4][8];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (i + u * LPA * 8 < d) load8(xr + i + u * LPA * 8, v[u]);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (i + u * LPA * 8 < d)
#pragma unroll
                        for (int q = 0; q < 8; ++q) ss = fmaf(v[u][q], v[u][q], ss);
            }
        }
#pragma unroll
        for (int off = LPA / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    }
    const float xn = live ? sqrtf(ss) * 1.001f + 1e-30f : 0.0f;

    // Fast logits of the lane's experts. Split-K logits (SPLIT, up to 8
    // parts): the partial sums in part order (any order of the d products is
    // covered by the bound), with every part's loads issued before the first
    // add (parts past nsplit re-read part 0 and are not added).
    // Dead tokens read row 0 and lanes past the logit row column 0 (neither
    // is used), so the loads need no branch.
    const int e0 = g * PER;
    float sf[PER];
    {
        const float* row = s_fast + (size_t)(live ? t : 0) * ld + (e0 < ld ? e0 : 0);
        if constexpr (SPLIT) {
            float pv[8][PER];
#pragma unroll
            for (int q = 0; q < 8; ++q) load_row<PER>(row + (q < nsplit ? q * sstride : 0), pv[q]);
#pragma unroll
            for (int m = 0; m < PER; ++m) sf[m] = pv[0][m];
#pragma unroll
            for (int q = 1; q < 8; ++q)
#pragma unroll
                for (int m = 0; m < PER; ++m) sf[m] = q < nsplit ? sf[m] + pv[q][m] : sf[m];
        } else {
            load_row<PER>(row, sf);
        }
    }
    __syncthreads();
    // The lane's biases and norms in 16-byte LDS reads (entries past E are
    // read but not used), then every interval without a branch.
    float bv[PER], wn[PER];
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
        const float4 b4 = *reinterpret_cast<const float4*>(sb + e0 + 4 * q);
        const float4 n4 = *reinterpret_cast<const float4*>(swn + e0 + 4 * q);
        bv[4 * q] = b4.x, bv[4 * q + 1] = b4.y, bv[4 * q + 2] = b4.z, bv[4 * q + 3] = b4.w;
        wn[4 * q] = n4.x, wn[4 * q + 1] = n4.y, wn[4 * q + 2] = n4.z, wn[4 * q + 3] = n4.w;
    }
    float lo[PER], hi[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const bool ok = live && e0 + m < E;
        const float key = sigmoid_fast(sf[m]) + bv[m];
        const float delta = 0.25f * (cst * xn * wn[m]) + 4e-6f + 1e-6f * fabsf(bv[m]);
        lo[m] = ok ? key - delta : -INFINITY;
        hi[m] = ok ? key + delta : -INFINITY;
    }
    // L: the K-th largest of the lanes' three largest lower ends. These are a
    // subset of all lower ends, so L is at most the K-th largest lower end and
    // still a lower bound of the true K-th key; it equals it unless one lane
    // holds four or more of the K largest.
    float t1 = -INFINITY, t2 = -INFINITY, t3 = -INFINITY;
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const float v = lo[m];
        t3 = fmaxf(t3, fminf(t2, v));
        t2 = fmaxf(t2, fminf(t1, v));
        t1 = fmaxf(t1, v);
    }
    float L = -INFINITY;
    int used = 0;  // how many of t1, t2, t3 (in that order) have been taken
    for (int j = 0; j < K; ++j) {
        const float mine = used == 0 ? t1 : (used == 1 ? t2 : (used == 2 ? t3 : -INFINITY));
        const float gmax = group_max<LPA>(mine);
        const uint64_t holders = __ballot(used < 3 && mine == gmax) & grp;
        if (holders && lane == __ffsll((unsigned long long)holders) - 1) ++used;
        L = gmax;
    }
    int nc = 0;
    if constexpr (LPA == 16) {
        // Lane g's candidates in expert order after those of lanes 0 .. g - 1
        // (an inclusive scan of the lanes' counts along the 16-lane DPP row).
        uint32_t cbits = 0;
#pragma unroll
        for (int m = 0; m < PER; ++m) cbits |= (live && hi[m] >= L) ? (1u << m) : 0u;
        const int cnt = __popc(cbits);
        int incl = cnt;
        incl += __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xF, 0xF, false);  // row_shr:1
        incl += __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xF, 0xF, false);  // row_shr:2
        incl += __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xF, 0xF, false);  // row_shr:4
        incl += __builtin_amdgcn_update_dpp(0, incl, 0x118, 0xF, 0xF, false);  // row_shr:8
        nc = __builtin_amdgcn_update_dpp(0, incl, 0x15F, 0xF, 0xF, false);     // row_newbcast:15
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int pos = incl - cnt + __popc(cbits & ((1u << m) - 1u));
            if (((cbits >> m) & 1u) && pos < NS) cand[(size_t)t * NS + pos] = (uint16_t)(e0 + m);
        }
    } else {
        const uint64_t below = grp & ((1ull << lane) - 1ull);
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const bool c = live && hi[m] >= L;
            const uint64_t bal = __ballot(c) & grp;
            if (c) {
                const int pos = nc + __popcll(bal & below);
                if (pos < NS) cand[(size_t)t * NS + pos] = (uint16_t)(e0 + m);
            }
            nc += __popcll(bal);
        }
    }
    if (live && g == 0) {
        if (nc > NS) {
            const int slot = atomicAdd(ovf_count, 1);
            ovf_list[slot] = t;
            nc = -1;
        }
        ncand[t] = nc;
    }
}

// Exact top-K of a token's candidates and their gates, for the chain kernels
// (TPB tokens of LPT lanes, CPL chains per lane; candidate slot g + LPT c of
// token tl holds expert ec[c] with exact logit acc[c]). Every candidate's key
// (sigmoid plus selection bias), sigmoid and expert go to LDS; each lane
// ranks its own candidates among the token's in (key descending, expert
// ascending) order, the order of taking the K largest keys one by one; ranks
// below K are the slots. Then every lane of the token forms the gate
// denominator in slot order and writes its slots. Called by every thread of
// the block once its chains are done; lds holds at least
// TPB (12 LPT CPL + 8 kMaxK) bytes and is no longer read by the chains.
template <int TPB, int LPT, int CPL>
__device__ __forceinline__ void chain_select(uint8_t* lds, int tl, int g, int t, int T, int nc, int K,
                                             const bool (&on)[CPL], const int (&ec)[CPL], const float (&acc)[CPL],
                                             const float (&bc)[CPL], bool has_bias, int32_t* __restrict__ topk_idx,
                                             float* __restrict__ topk_gate) {
    constexpr int NS = LPT * CPL;
    float* skey = reinterpret_cast<float*>(lds);
    float* ssig = skey + TPB * NS;
    int* sexp = reinterpret_cast<int*>(ssig + TPB * NS);
    float* osig = reinterpret_cast<float*>(sexp + TPB * NS);
    int* oexp = reinterpret_cast<int*>(osig + TPB * kMaxK);
    float kc[CPL], sc[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int j = g + LPT * c;
        sc[c] = 0.0f;
        kc[c] = 0.0f;
        if (on[c]) {
            sc[c] = sigmoid_fp32(acc[c]);
            kc[c] = has_bias ? sc[c] + bc[c] : sc[c];
            skey[tl * NS + j] = kc[c];
            ssig[tl * NS + j] = sc[c];
            sexp[tl * NS + j] = ec[c];
        }
    }
    __syncthreads();
    // The token's NS keys and experts in 16-byte reads (slots from nc on are
    // read but not counted).
    static_assert(NS % 4 == 0, "whole 16-byte reads");
    float kq[NS];
    int eq[NS];
#pragma unroll
    for (int q = 0; q < NS; q += 4) {
        const float4 k4 = *reinterpret_cast<const float4*>(skey + tl * NS + q);
        const int4 e4 = *reinterpret_cast<const int4*>(sexp + tl * NS + q);
        kq[q] = k4.x, kq[q + 1] = k4.y, kq[q + 2] = k4.z, kq[q + 3] = k4.w;
        eq[q] = e4.x, eq[q + 1] = e4.y, eq[q + 2] = e4.z, eq[q + 3] = e4.w;
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        if (!on[c]) continue;
        int rank = 0;  // the candidate itself compares neither greater nor lower
#pragma unroll
        for (int q = 0; q < NS; ++q)
            rank += (q < nc && (kq[q] > kc[c] || (kq[q] == kc[c] && eq[q] < ec[c]))) ? 1 : 0;
        if (rank < K) {
            osig[tl * kMaxK + rank] = sc[c];
            oexp[tl * kMaxK + rank] = ec[c];
        }
    }
    __syncthreads();
    if (t >= T || nc == 0) return;
    // Gate denominator in slot order 0 .. K - 1.
    float os[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; j += 4) {
        const float4 o4 = *reinterpret_cast<const float4*>(osig + tl * kMaxK + j);
        os[j] = o4.x, os[j + 1] = o4.y, os[j + 2] = o4.z, os[j + 3] = o4.w;
    }
    float den = os[0];
#pragma unroll
    for (int j = 1; j < kMaxK; ++j) den = j < K ? den + os[j] : den;
    for (int j = g; j < K; j += LPT) {
        topk_idx[(size_t)t * K + j] = oexp[tl * kMaxK + j];
        topk_gate[(size_t)t * K + j] = osig[tl * kMaxK + j] / den;
    }
}

// Exact top-K of token t from its E sigmoids (sig, in LDS) and gates, by one
// wave: each of the K rounds takes the wave-wide best key (descending, lower
// expert index first on equal keys) with a butterfly of cross-lane exchanges.
__device__ __forceinline__ void exact_select_wave(const float* sig, const float* __restrict__ bias, int E, int K,
                                                  int t, int lane, int32_t* __restrict__ topk_idx,
                                                  float* __restrict__ topk_gate) {
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

// Exact routing of the queued tokens: all E logits by the FMA chain, then
// the same top-K. Blocks first, first + stride, ... walk the queue (fixed by
// the time this runs); every block exits once it is exhausted. Any block
// size that is a multiple of the wave works (the selection uses wave 0).
__device__ __forceinline__ void exact_list_run(const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr,
                               const float* __restrict__ bias, int d, int E, int K,
                               const int32_t* __restrict__ ovf_count, const int32_t* __restrict__ ovf_list,
                               int32_t* __restrict__ topk_idx, float* __restrict__ topk_gate, int first,
                               int stride) {
    __shared__ float sig[kMaxE];
    const int n = *ovf_count;
    const int lane = threadIdx.x & (kWave - 1);
    for (int it = first; it < n; it += stride) {
        const int t = ovf_list[it];
        const bf16_t* xt = x + (size_t)t * d;
        for (int e = threadIdx.x; e < E; e += blockDim.x) {
            const bf16_t* we = wr + (size_t)e * d;
            // The same fma sequence over i = 0..d-1; the loads of 32 columns
            // are issued before their multiply-adds (d is a multiple of 64).
            float a = 0.0f;
            for (int i = 0; i < d; i += 32) {
                float xv[4][8], wv[4][8];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    load8(xt + i + 8 * q, xv[q]);
                    load8(we + i + 8 * q, wv[q]);
                }
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int u = 0; u < 8; ++u) a = fmaf(xv[q][u], wv[q][u], a);
            }
            sig[e] = sigmoid_fp32(a);
        }
        __syncthreads();
        if (threadIdx.x < kWave) exact_select_wave(sig, bias, E, K, t, lane, topk_idx, topk_gate);
        __syncthreads();
    }
}

// Exact logits of the candidates, recipe S, exact top-K and gates. LPT lanes
// per token, each running CPL candidate chains (slots g, g + LPT, ...) side by
// side: one fused multiply-add chain per candidate over the model width, in
// ascending order. The block's tokens stream their x rows from global memory;
// the router weights of every expert stream through LDS in chunks of DC
// columns (bf16, rows padded by 16 bytes against bank conflicts, widened to
// fp32 in registers), double-buffered with one barrier per chunk; DC must
// divide d. Tokens queued by the candidate kernel are skipped.
template <int TPB, int LPT, int CPL, int EMAX, int DC>
__global__ __launch_bounds__(TPB* LPT) void k_router_chain(const bf16_t* __restrict__ x,
                                                         const bf16_t* __restrict__ wr,
                                                         const float* __restrict__ bias,
                                                         const uint16_t* __restrict__ cand,
                                                         const int32_t* __restrict__ ncand, int T, int d, int E,
                                                         int K, int32_t* __restrict__ topk_idx,
                                                         float* __restrict__ topk_gate, int chain_blocks,
                                                         const int32_t* __restrict__ ovf_count,
                                                         const int32_t* __restrict__ ovf_list) {
    // Blocks from chain_blocks on route the tokens of the overflow queue (all
    // of it is written: the candidate kernel has finished); with an empty
    // queue they exit at once.
    if ((int)blockIdx.x >= chain_blocks) {
        exact_list_run(x, wr, bias, d, E, K, ovf_count, ovf_list, topk_idx, topk_gate,
                       (int)blockIdx.x - chain_blocks, (int)gridDim.x - chain_blocks);
        return;
    }
    constexpr int NT = TPB * LPT;
    constexpr int NS = LPT * CPL;
    constexpr int ROW = DC + 8;             // bf16 per LDS row (16 bytes of padding)
    constexpr int XQ = DC / 8;              // 16-byte x pieces per chunk
    constexpr int WP = EMAX * DC / 8;        // 16-byte router-weight pieces per chunk
    constexpr int WQ = (WP + NT - 1) / NT;   // per thread
    static_assert(NS <= 32, "at most 32 candidate slots");
    constexpr int RING = 2 * EMAX * ROW * 2, SEL = TPB * (NS * 12 + kMaxK * 8);
    __shared__ __attribute__((aligned(16))) uint8_t lds[RING > SEL ? RING : SEL];
    auto wsh = reinterpret_cast<bf16_t(*)[EMAX][ROW]>(lds);

    const int tid = threadIdx.x;
    const int g = tid % LPT;
    const int tl = tid / LPT;

    // Token slots grouped by the chains per lane each token needs (0..CPL).
    // A wave runs as many chains per lane as its busiest token; in token
    // order nearly every wave holds some token with a few extra candidates,
    // grouped most waves run only the chains of a token with K candidates.
    // The order is ascending token within a group; a token's results do not
    // depend on the lanes that compute it.
    static_assert(TPB % kWave == 0 && NT >= TPB, "token slots fill whole waves");
    constexpr int TW = TPB / kWave;
    __shared__ int32_t sperm[TPB];
    __shared__ int32_t sgrp[TW][CPL + 1];
    {
        const int lane = tid & (kWave - 1), wv = tid / kWave;
        int key = 0;
        uint64_t same = 0;
        if (tid < TPB) {  // whole waves
            const int u = blockIdx.x * TPB + tid;
            const int n = u < T ? ncand[u] : 0;
            key = n <= 0 ? 0 : min((n + LPT - 1) / LPT, CPL);
#pragma unroll
            for (int k = 0; k <= CPL; ++k) {
                const uint64_t m = __ballot(key == k);
                if (k == key) same = m;
                if (lane == 0) sgrp[wv][k] = __popcll(m);
            }
        }
        __syncthreads();
        if (tid < TPB) {
            int pos = __popcll(same & ((1ull << lane) - 1ull));
            for (int k = 0; k < key; ++k)
                for (int w = 0; w < TW; ++w) pos += sgrp[w][k];
            for (int w = 0; w < wv; ++w) pos += sgrp[w][key];
            sperm[pos] = tid;
        }
        __syncthreads();
    }
    const int t = blockIdx.x * TPB + sperm[tl];
    int nc = t < T ? ncand[t] : 0;
    nc = nc < 0 ? 0 : nc;  // queued tokens are routed by the exact-list kernel
    int ec[CPL];
    bool on[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int j = g + LPT * c;
        on[c] = j < nc;
        ec[c] = on[c] ? (int)cand[(size_t)t * NS + j] : 0;
    }
    const bf16_t* xt = x + (size_t)(t < T ? t : 0) * d;
    float bc[CPL];  // selection bias of each chain's expert, read while the chains run
#pragma unroll
    for (int c = 0; c < CPL; ++c) bc[c] = (bias && on[c]) ? bias[ec[c]] : 0.0f;

    u32x4_t xr[XQ], wrg[WQ];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < XQ; ++i) xr[i] = *reinterpret_cast<const u32x4_t*>(xt + k0 + 8 * i);
#pragma unroll
        for (int i = 0; i < WQ; ++i) {
            const int q = (tid + NT * i) * 8;  // element of the EMAX x DC chunk
            const int e = q / DC, c = q % DC;
            wrg[i] = (u32x4_t){0u, 0u, 0u, 0u};
            if (tid + NT * i < WP && e < E) wrg[i] = *reinterpret_cast<const u32x4_t*>(wr + (size_t)e * d + k0 + c);
        }
    };
    auto stash = [&](int b) {
#pragma unroll
        for (int i = 0; i < WQ; ++i) {
            if (tid + NT * i >= WP) continue;
            const int q = (tid + NT * i) * 8;
            *reinterpret_cast<u32x4_t*>(&wsh[b][q / DC][q % DC]) = wrg[i];
        }
    };

    float acc[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[c] = 0.0f;

    // One chunk: for every 8 columns, widen x once and advance each of the
    // first NC chains by 8 fused multiply-adds (ascending columns).
    auto chunk = [&](auto NCC, int b) {
        constexpr int NC = decltype(NCC)::value;
#pragma unroll
        for (int i = 0; i < XQ; ++i) {
            const u32x4_t u = xr[i];
            const float x0 = __uint_as_float(u.x << 16), x1 = __uint_as_float(u.x & 0xffff0000u);
            const float x2 = __uint_as_float(u.y << 16), x3 = __uint_as_float(u.y & 0xffff0000u);
            const float x4 = __uint_as_float(u.z << 16), x5 = __uint_as_float(u.z & 0xffff0000u);
            const float x6 = __uint_as_float(u.w << 16), x7 = __uint_as_float(u.w & 0xffff0000u);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const u32x4_t w = *reinterpret_cast<const u32x4_t*>(&wsh[b][ec[c]][8 * i]);
                float a = acc[c];
                a = fmaf(x0, __uint_as_float(w.x << 16), a);
                a = fmaf(x1, __uint_as_float(w.x & 0xffff0000u), a);
                a = fmaf(x2, __uint_as_float(w.y << 16), a);
                a = fmaf(x3, __uint_as_float(w.y & 0xffff0000u), a);
                a = fmaf(x4, __uint_as_float(w.z << 16), a);
                a = fmaf(x5, __uint_as_float(w.z & 0xffff0000u), a);
                a = fmaf(x6, __uint_as_float(w.w << 16), a);
                a = fmaf(x7, __uint_as_float(w.w & 0xffff0000u), a);
                acc[c] = a;
            }
            // Keep the compiler from hoisting every fragment read of the chunk
            // (registers, not latency, bound this kernel's occupancy).
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    int nmax = 0;  // chains any lane of this wave runs (uniform)
#pragma unroll
    for (int c = 0; c < CPL; ++c) nmax += __ballot(on[c]) != 0 ? 1 : 0;

    u32x4_t xn[XQ];
    fetch(0);
    stash(0);
    __syncthreads();
    int buf = 0;
    const int nch = d / DC;
    for (int ch = 0; ch < nch; ++ch) {
        // Next chunk in flight during this one: its x into xn, its weights
        // into registers (stored to the other buffer after the chains).
        if (ch + 1 < nch) {
            const int k1 = (ch + 1) * DC;
#pragma unroll
            for (int i = 0; i < XQ; ++i) xn[i] = *reinterpret_cast<const u32x4_t*>(xt + k1 + 8 * i);
#pragma unroll
            for (int i = 0; i < WQ; ++i) {
                const int q = (tid + NT * i) * 8;
                const int e = q / DC, c = q % DC;
                wrg[i] = (u32x4_t){0u, 0u, 0u, 0u};
                if (tid + NT * i < WP && e < E) wrg[i] = *reinterpret_cast<const u32x4_t*>(wr + (size_t)e * d + k1 + c);
            }
        }
        // The wave's chain count (uniform) picks an unrolled chunk.
        static_for<CPL>([&](auto IC) {
            constexpr int n = decltype(IC)::value + 1;
            if (nmax == n) chunk(std::integral_constant<int, n>{}, buf);
        });
        if (ch + 1 < nch) {
            stash(buf ^ 1);
#pragma unroll
            for (int i = 0; i < XQ; ++i) xr[i] = xn[i];
        }
        __syncthreads();
        buf ^= 1;
    }

    // Selection (the ring is free after the last barrier).
    chain_select<TPB, LPT, CPL>(lds, tl, g, t, T, nc, K, on, ec, acc, bc, bias != nullptr, topk_idx, topk_gate);
}

// Exact logits for small batches, where streaming every expert's weights
// through LDS per block of tokens costs more than the candidates need: one
// 64-lane wave per TPB = 64 / LPT tokens, one candidate chain per lane (LPT =
// the candidate slots). The block's x rows are staged in LDS widened to fp32;
// each lane reads its candidate's router-weight row, widened to fp32 by the
// norm kernel (wr32), straight from global memory in groups of 32 columns,
// two groups ahead of the multiply-adds. A multiply-add then costs one FMA
// plus a quarter of an LDS and of a global read, against three VALU
// operations with bf16 operands (both widenings); at a few waves per CU the
// kernel is bound by each wave's issue and latency, not by bandwidth. The
// chain is the same fused multiply-add sequence over i = 0..d-1, from +0, on
// the same (exactly widened) values as in k_router_chain.
//
// Blocks from chain_blocks on route the tokens of the overflow queue instead
// (exact_list_run), so that no separate launch is needed; the chain blocks
// skip queued tokens and write nothing for them. Dynamic LDS: max(TPB d fp32,
// the selection's arrays). d is a multiple of 64.
template <int LPT>
__global__ __launch_bounds__(kWave) void k_router_chain_direct(const bf16_t* __restrict__ x,
                                                             const float* __restrict__ wr32,
                                                             const bf16_t* __restrict__ wr,
                                                             const float* __restrict__ bias,
                                                             const uint16_t* __restrict__ cand,
                                                             const int32_t* __restrict__ ncand, int T, int d, int E,
                                                             int K, int32_t* __restrict__ topk_idx,
                                                             float* __restrict__ topk_gate, int chain_blocks,
                                                             const int32_t* __restrict__ ovf_count,
                                                             const int32_t* __restrict__ ovf_list) {
    if ((int)blockIdx.x >= chain_blocks) {
        exact_list_run(x, wr, bias, d, E, K, ovf_count, ovf_list, topk_idx, topk_gate,
                       (int)blockIdx.x - chain_blocks, (int)gridDim.x - chain_blocks);
        return;
    }
    constexpr int TPB = kWave / LPT;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_dyn[];
    const int tid = threadIdx.x;
    const int g = tid % LPT;
    const int tl = tid / LPT;
    const int t = blockIdx.x * TPB + tl;
    int nc = t < T ? ncand[t] : 0;
    nc = nc < 0 ? 0 : nc;  // queued tokens are routed by the queue blocks
    const bool on[1] = {g < nc};
    const int ec[1] = {on[0] ? (int)cand[(size_t)t * LPT + g] : 0};
    const float bc[1] = {(bias && on[0]) ? bias[ec[0]] : 0.0f};

    // x rows of the block's tokens, widened to fp32 (tokens past T copy row
    // T - 1; their chains are off).
    float* xs = reinterpret_cast<float*>(lds_dyn);
    // Four 16-byte pieces per lane and round, all loaded before the writes.
    const bf16_t* xt = x + (size_t)(t < T ? t : T - 1) * d;
    for (int i0 = g * 8; i0 < d; i0 += 4 * LPT * 8) {
        u32x4_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u * LPT * 8 < d) v[u] = *reinterpret_cast<const u32x4_t*>(xt + i0 + u * LPT * 8);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + u * LPT * 8;
            if (i < d) {
                *reinterpret_cast<float4*>(xs + tl * d + i) =
                    make_float4(__uint_as_float(v[u].x << 16), __uint_as_float(v[u].x & 0xffff0000u),
                                __uint_as_float(v[u].y << 16), __uint_as_float(v[u].y & 0xffff0000u));
                *reinterpret_cast<float4*>(xs + tl * d + i + 4) =
                    make_float4(__uint_as_float(v[u].z << 16), __uint_as_float(v[u].z & 0xffff0000u),
                                __uint_as_float(v[u].w << 16), __uint_as_float(v[u].w & 0xffff0000u));
            }
        }
    }
    __syncthreads();

    float acc[1] = {0.0f};
    if (__ballot(on[0]) != 0) {
        const float* we = wr32 + (size_t)ec[0] * d;
        const float* xr = xs + tl * d;
        const int ng = d / 32;  // even, >= 2
        // Ring of RB groups of 32 columns of weights in registers, RB - 1
        // groups ahead of the multiply-adds, and the x values of the next
        // group read from LDS while the current group's multiply-adds run: at
        // a wave or two per SIMD nothing else hides either latency.
        constexpr int RB = 4;
        float4 w[RB][8], xv[2][8];
        auto load = [&](int b, int grp) {
#pragma unroll
            for (int u = 0; u < 8; ++u) w[b][u] = *reinterpret_cast<const float4*>(we + grp * 32 + 4 * u);
        };
        auto read_x = [&](int b, int grp) {
#pragma unroll
            for (int u = 0; u < 8; ++u) xv[b][u] = *reinterpret_cast<const float4*>(xr + grp * 32 + 4 * u);
        };
        float a = 0.0f;
#pragma unroll
        for (int b = 0; b < RB - 1; ++b)
            if (b < ng) load(b, b);
        read_x(0, 0);
        for (int n = 0; n < ng; n += RB) {
            static_for<RB>([&](auto BC) {
                constexpr int b = decltype(BC)::value;
                if (n + b < ng) {
                    if (n + b + RB - 1 < ng) load((b + RB - 1) % RB, n + b + RB - 1);
                    if (n + b + 1 < ng) read_x((b + 1) & 1, n + b + 1);
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        a = fmaf(xv[b & 1][u].x, w[b][u].x, a);
                        a = fmaf(xv[b & 1][u].y, w[b][u].y, a);
                        a = fmaf(xv[b & 1][u].z, w[b][u].z, a);
                        a = fmaf(xv[b & 1][u].w, w[b][u].w, a);
                    }
                }
            });
        }
        acc[0] = a;
    }
    __syncthreads();  // the selection reuses the x rows' LDS
    chain_select<TPB, LPT, 1>(lds_dyn, tl, g, t, T, nc, K, on, ec, acc, bc, bias != nullptr, topk_idx, topk_gate);
}

// Small batches with K <= 8, at most 256 experts and d <= 4096: the whole
// repair in one launch. A one-wave block takes 4 tokens, 16 lanes each (lane
// g holding experts g PER .. g PER + PER - 1, as in the candidate kernel):
//  - the weight-row norms come from the logits GEMM's per-part sums of
//    squares (wsq [nsplit][ld]), the token norms from the token's x row,
//    which the block stages in LDS widened to fp32 for the chains anyway;
//  - the interval test of the candidate kernel, the candidate list in LDS;
//  - lane g runs the exact chain of the token's candidate g (slot 16 tl + g).
//    The weight rows of the block's 64 slots stream through LDS in chunks of
//    128 columns, three buffers deep, by direct-to-LDS copies of 1 KB that
//    each carry 256 contiguous bytes of four slots' rows (8 cache lines per
//    copy, where a row per lane would touch 64). The chain is a run of
//    dependent multiply-adds; the bf16 weights of the next 16 columns are
//    widened between them, so that the adds never wait on the widening;
//  - then the chain kernels' selection;
//  - a token with more candidates than its 16 slots is routed by the block
//    itself: every E logit by the same chain, recipe S and the exact top-K,
//    so no queue crosses blocks.
// Every multiply-add chain and selection is the same as on the other paths,
// so indices and gates are identical bit for bit.
constexpr int kSmallTpb = 4;      // tokens per one-wave block
constexpr int kSmallChunk = 128;  // weight columns per LDS chunk
constexpr int kSmallBufs = 3;     // chunk buffers (two chunks in flight)
// One copy: 16-byte piece j (columns 8j .. 8j + 7 of the chunk) of slot
// 4i + q at byte 16 (4 j + q); 64 bytes of padding after each copy put the 16
// slots that a quarter wave reads at once on distinct LDS banks.
constexpr int kSmallCopyBytes = kWave * 16 + 64;
constexpr int kSmallBufBytes = (kWave / 4) * kSmallCopyBytes;
constexpr int kSmallSelBytes = kSmallTpb * (16 * 12 + kMaxK * 8);
static_assert(kSmallSelBytes + 256 * 4 <= kSmallBufs * kSmallBufBytes, "selection arrays fit the buffers");

// 16 bytes from LDS at addr + OFF (inline assembly: the compiler neither sees
// the read nor waits for it; the caller waits with lgkmcnt and pins the
// result with tie()).
template <int OFF>
__device__ __forceinline__ u32x4_t lds_read16u_off(uint32_t addr) {
    u32x4_t r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}

// Element j (0..15) of 16 bf16 held in two 16-byte registers, widened.
__device__ __forceinline__ float bf16_elem(const u32x4_t (&w)[2], int j) {
    const uint32_t bits = w[j / 8][(j / 2) % 4];
    return __uint_as_float((j & 1) ? (bits & 0xffff0000u) : (bits << 16));
}

// Dynamic LDS of k_router_small: the 4 x rows (d + 4 floats each: the pad
// spreads the 4 tokens' reads over the banks) and the chunk buffers, which
// the selection's arrays and the overflow path's sigmoids reuse afterwards.
// At d = 1536 this and the static arrays stay under half the LDS, so two
// blocks share a CU (one image's 257 blocks all run at once).
size_t router_small_lds_bytes(int d) {
    return (size_t)kSmallTpb * (d + 4) * 4 + (size_t)kSmallBufs * kSmallBufBytes;
}

template <int PER>
__global__ __launch_bounds__(kWave) void k_router_small(const float* __restrict__ s_fast, int nsplit,
                                                      size_t sstride, int ld, const float* __restrict__ wsq,
                                                      const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr,
                                                      const float* __restrict__ bias, int T, int d, int E, int K,
                                                      float cst, int32_t* __restrict__ topk_idx,
                                                      float* __restrict__ topk_gate) {
    constexpr int LPA = 16, NS = 16, TPB = kSmallTpb, EM = LPA * PER;
    static_assert(TPB * LPA == kWave, "one wave of 4 tokens");
    static_assert(PER % 4 == 0 && 64 % PER == 0, "whole 16-byte loads inside a row of a multiple of 64");
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_dyn[];
    __shared__ __attribute__((aligned(16))) float sb[EM];
    __shared__ __attribute__((aligned(16))) float swn[EM];
    __shared__ uint16_t scand[TPB][NS];
    __shared__ int snc[TPB];  // candidates per token (more than NS: the block routes it in full)
    const int lane = threadIdx.x;
    const int g = lane % LPA, tl = lane / LPA;
    const int t = blockIdx.x * TPB + tl;
    const bool live = t < T;  // uniform within the token's lanes
    const uint64_t grp = ((1ull << LPA) - 1ull) << (lane - g);
    const int XS = d + 4;  // x row stride in LDS (floats)
    float* xs = reinterpret_cast<float*>(lds_dyn);
    uint8_t* wbuf = lds_dyn + (size_t)TPB * XS * 4;
    uint8_t* sel = wbuf;                                        // after the chains
    float* ssig = reinterpret_cast<float*>(wbuf + kSmallSelBytes);  // overflow path

    // Every global load of the token phase is issued before the first use:
    // the partial logits of the lane's experts, the parts' sums of squares of
    // the weight rows and the x pieces (tokens past T read row T - 1, lanes
    // past the logit row read column 0; neither is used).
    const int e0 = g * PER;
    float pv[8][PER];
    {
        const float* row = s_fast + (size_t)(live ? t : T - 1) * ld + (e0 < ld ? e0 : 0);
#pragma unroll
        for (int q = 0; q < 8; ++q) load_row<PER>(row + (q < nsplit ? q * sstride : 0), pv[q]);
    }
    constexpr int EPL = EM / kWave > 0 ? EM / kWave : 1;
    float part[EPL][8];
#pragma unroll
    for (int m = 0; m < EPL; ++m) {
        const int e = lane + kWave * m;
        const int ec = e < E ? e : 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) part[m][q] = wsq[(size_t)(q < nsplit ? q : 0) * ld + ec];
    }
    // x: sixteen 16-byte pieces per lane and round (2048 columns), the last
    // round's pieces past d re-reading the row's last piece.
    const bf16_t* xt = x + (size_t)(live ? t : T - 1) * d;
    constexpr int XU = 16;
    u32x4_t xr16[XU];
#pragma unroll
    for (int u = 0; u < XU; ++u) {
        const int i = g * 8 + u * LPA * 8;
        xr16[u] = *reinterpret_cast<const u32x4_t*>(xt + (i < d ? i : d - 8));
    }

    // Selection biases and weight-row norms: the parts' sums of squares added
    // in part order and raised by 0.1 % as the norm kernel does (an upper
    // bound is all the interval needs).
#pragma unroll
    for (int m = 0; m < EPL; ++m) {
        const int e = lane + kWave * m;
        float ss = part[m][0];
#pragma unroll
        for (int q = 1; q < 8; ++q) ss = q < nsplit ? ss + part[m][q] : ss;
        if (e < E) {
            swn[e] = sqrtf(ss) * 1.001f + 1e-30f;
            sb[e] = bias ? bias[e] : 0.0f;
        }
    }

    // x rows widened to fp32 in LDS, and the token's sum of squares from the
    // same values.
    float ssq[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // four partial sums: no long dependent run
    for (int i0 = g * 8; i0 < d; i0 += XU * LPA * 8) {
        if (i0 != g * 8) {  // rounds past the first (d > 2048)
#pragma unroll
            for (int u = 0; u < XU; ++u) {
                const int i = i0 + u * LPA * 8;
                xr16[u] = *reinterpret_cast<const u32x4_t*>(xt + (i < d ? i : d - 8));
            }
        }
#pragma unroll
        for (int u = 0; u < XU; ++u) {
            const int i = i0 + u * LPA * 8;
            if (i < d) {
                const u32x4_t v = xr16[u];
                const float f[8] = {__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                                    __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u),
                                    __uint_as_float(v.z << 16), __uint_as_float(v.z & 0xffff0000u),
                                    __uint_as_float(v.w << 16), __uint_as_float(v.w & 0xffff0000u)};
                *reinterpret_cast<float4*>(xs + tl * XS + i) = make_float4(f[0], f[1], f[2], f[3]);
                *reinterpret_cast<float4*>(xs + tl * XS + i + 4) = make_float4(f[4], f[5], f[6], f[7]);
#pragma unroll
                for (int q = 0; q < 8; ++q) ssq[q % 4] = fmaf(f[q], f[q], ssq[q % 4]);
            }
        }
    }
    float ssx = (ssq[0] + ssq[1]) + (ssq[2] + ssq[3]);
#pragma unroll
    for (int off = LPA / 2; off > 0; off >>= 1) ssx += __shfl_xor(ssx, off);
    const float xn = live ? sqrtf(ssx) * 1.001f + 1e-30f : 0.0f;

    // Fast logits of the lane's experts: the K parts added in part order.
    float sf[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) sf[m] = pv[0][m];
#pragma unroll
    for (int q = 1; q < 8; ++q)
#pragma unroll
        for (int m = 0; m < PER; ++m) sf[m] = q < nsplit ? sf[m] + pv[q][m] : sf[m];
    __syncthreads();
    // The interval test, as in the candidate kernel.
    // The lane's biases and norms in 16-byte LDS reads (entries past E are
    // read but not used), then every interval without a branch.
    float bv[PER], wn[PER];
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
        const float4 b4 = *reinterpret_cast<const float4*>(sb + e0 + 4 * q);
        const float4 n4 = *reinterpret_cast<const float4*>(swn + e0 + 4 * q);
        bv[4 * q] = b4.x, bv[4 * q + 1] = b4.y, bv[4 * q + 2] = b4.z, bv[4 * q + 3] = b4.w;
        wn[4 * q] = n4.x, wn[4 * q + 1] = n4.y, wn[4 * q + 2] = n4.z, wn[4 * q + 3] = n4.w;
    }
    float lo[PER], hi[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const bool ok = live && e0 + m < E;
        const float key = sigmoid_fast(sf[m]) + bv[m];
        const float delta = 0.25f * (cst * xn * wn[m]) + 4e-6f + 1e-6f * fabsf(bv[m]);
        lo[m] = ok ? key - delta : -INFINITY;
        hi[m] = ok ? key + delta : -INFINITY;
    }
    float t1 = -INFINITY, t2 = -INFINITY, t3 = -INFINITY;
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const float v = lo[m];
        t3 = fmaxf(t3, fminf(t2, v));
        t2 = fmaxf(t2, fminf(t1, v));
        t1 = fmaxf(t1, v);
    }
    float L = -INFINITY;
    int used = 0;
    for (int j = 0; j < K; ++j) {
        const float mine = used == 0 ? t1 : (used == 1 ? t2 : (used == 2 ? t3 : -INFINITY));
        const float gmax = group_max<LPA>(mine);
        const uint64_t holders = __ballot(used < 3 && mine == gmax) & grp;
        if (holders && lane == __ffsll((unsigned long long)holders) - 1) ++used;
        L = gmax;
    }
    // Candidates: lane g's in expert order after those of lanes 0 .. g - 1
    // (an inclusive scan of the lanes' counts along the 16-lane DPP row).
    uint32_t cbits = 0;
#pragma unroll
    for (int m = 0; m < PER; ++m) cbits |= (live && hi[m] >= L) ? (1u << m) : 0u;
    const int cnt = __popc(cbits);
    int incl = cnt;
    incl += __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xF, 0xF, false);  // row_shr:1
    incl += __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xF, 0xF, false);  // row_shr:2
    incl += __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xF, 0xF, false);  // row_shr:4
    incl += __builtin_amdgcn_update_dpp(0, incl, 0x118, 0xF, 0xF, false);  // row_shr:8
    const int nc = __builtin_amdgcn_update_dpp(0, incl, 0x15F, 0xF, 0xF, false);  // row_newbcast:15
#pragma unroll
    for (int m = 0; m < PER; ++m) {
        const int pos = incl - cnt + __popc(cbits & ((1u << m) - 1u));
        if (((cbits >> m) & 1u) && pos < NS) scand[tl][pos] = (uint16_t)(e0 + m);
    }
    if (g == 0) snc[tl] = nc;
    __syncthreads();

    // Exact chain of candidate g (slot 16 tl + g).
    const int ncx = nc > NS ? 0 : nc;  // an overflowing token is routed below
    const bool on[1] = {g < ncx};
    const int ec[1] = {on[0] ? (int)scand[tl][g] : 0};
    const float bc[1] = {(bias && on[0]) ? sb[ec[0]] : 0.0f};
    float acc[1] = {0.0f};
    if (__ballot(on[0]) != 0) {
        // Copy sources: in copy i this lane carries 16 bytes of slot
        // 4i + lane % 4, piece lane / 4 of the chunk's 256 bytes of that
        // slot's row. Free slots copy row 0 (in bounds, never read); the rest
        // of a ragged last chunk is never read either.
        int ncs[TPB];
#pragma unroll
        for (int u = 0; u < TPB; ++u) ncs[u] = snc[u] > NS ? 0 : snc[u];
        uint32_t roff[kWave / 4];
#pragma unroll
        for (int i = 0; i < kWave / 4; ++i) {
            const int slot = 4 * i + (lane & 3);
            const int su = slot / NS, sg = slot % NS;
            const int e = sg < ncs[su] ? (int)scand[su][sg] : 0;
            roff[i] = (uint32_t)e * (uint32_t)d * 2u + (uint32_t)(lane >> 2) * 16u;
        }
        const __amdgpu_buffer_rsrc_t rw = make_rsrc(wr, (uint32_t)((size_t)E * d * 2));
        auto copy_chunk = [&](int c) {
            uint8_t* dst = wbuf + (size_t)(c % kSmallBufs) * kSmallBufBytes;
#pragma unroll
            for (int i = 0; i < kWave / 4; ++i)
                copy16_to_lds(rw, roff[i], (uint32_t)c * (kSmallChunk * 2), dst + i * kSmallCopyBytes);
        };
        // This lane's slot in buffer 0 (piece j at + 64 j) and its token's x row.
        const uint32_t wa0 = lds_address(wbuf) + (uint32_t)(lane >> 2) * kSmallCopyBytes + (uint32_t)(lane & 3) * 16u;
        const uint32_t xa0 = lds_address(reinterpret_cast<uint8_t*>(xs + tl * XS));
        const int nch = (d + kSmallChunk - 1) / kSmallChunk;
        float a = 0.0f;
        // Register sets of three units in rotation (raw 16-byte reads) and the
        // widened weights of two units.
        u32x4_t wv[3][2] = {}, xv[3][4] = {};
        float wf[2][16];
        copy_chunk(0);
        if (nch > 1) copy_chunk(1);
        for (int c = 0; c < nch; ++c) {
            // Chunk c is in LDS once at most one chunk's copies are in flight
            // (a single wave: its own copies).
            if (c + 1 < nch) wait_vmcnt<kWave / 4>(); else wait_vmcnt<0>();
            // Chunk c - 1's buffer is free: every LDS read of it was awaited.
            if (c + 2 < nch) copy_chunk(c + 2);
            const uint32_t wa = wa0 + (uint32_t)(c % kSmallBufs) * kSmallBufBytes;
            const uint32_t xa = xa0 + (uint32_t)c * (kSmallChunk * 4);
            const int left = (d - c * kSmallChunk) / 16;
            const int nu = left < kSmallChunk / 16 ? left : kSmallChunk / 16;  // units of 16 columns
            auto issue = [&](auto KC) {
                constexpr int k = decltype(KC)::value;
                constexpr int r = k % 3;
                wv[r][0] = lds_read16u_off<k * 128>(wa);
                wv[r][1] = lds_read16u_off<k * 128 + 64>(wa);
                xv[r][0] = lds_read16u_off<k * 64>(xa);
                xv[r][1] = lds_read16u_off<k * 64 + 16>(xa);
                xv[r][2] = lds_read16u_off<k * 64 + 32>(xa);
                xv[r][3] = lds_read16u_off<k * 64 + 48>(xa);
            };
            auto settle = [&](int r) {
                tie(wv[r][0]);
                tie(wv[r][1]);
#pragma unroll
                for (int q = 0; q < 4; ++q) tie(xv[r][q]);
            };
            issue(std::integral_constant<int, 0>{});
            if (nu > 1) issue(std::integral_constant<int, 1>{});
            if (nu > 1) wait_lgkmcnt<6>(); else wait_lgkmcnt<0>();
            settle(0);
#pragma unroll
            for (int j = 0; j < 16; ++j) wf[0][j] = bf16_elem(wv[0], j);
            static_for<kSmallChunk / 16>([&](auto KC) {
                constexpr int k = decltype(KC)::value;
                constexpr int r = k % 3, r1 = (k + 1) % 3;
                if (k < nu) {
                    wait_lgkmcnt<0>();  // unit k + 1's reads (the last ones issued)
                    settle(r1);
                    if constexpr (k + 2 < kSmallChunk / 16)
                        if (k + 2 < nu) issue(std::integral_constant<int, k + 2>{});
                    // Unit k's 16 multiply-adds in column order, unit k + 1's
                    // weights widened in between.
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        a = fmaf(__uint_as_float(xv[r][j / 4][j % 4]), wf[k % 2][j], a);
                        wf[(k + 1) % 2][j] = bf16_elem(wv[r1], j);
                    }
                }
            });
        }
        acc[0] = a;
    }
    // The selection's arrays reuse the chunk buffers (no copy is in flight).
    chain_select<TPB, LPA, 1>(sel, tl, g, t, T, ncx, K, on, ec, acc, bc, bias != nullptr, topk_idx, topk_gate);

    // Overflowing tokens, one at a time: lane l runs the chains of experts
    // l, l + 64, ... side by side (at most 4 for E <= 256), each the same fma
    // sequence over i = 0..d-1 from +0, then recipe S and the exact top-K.
    for (int u = 0; u < TPB; ++u) {
        if (snc[u] <= NS) continue;  // uniform: one LDS value for the whole wave
        const int tu = blockIdx.x * TPB + u;
        const float* xr = xs + u * XS;
        constexpr int EPL = EM / kWave > 0 ? EM / kWave : 1;
        float av[EPL];
        const bf16_t* we[EPL];
#pragma unroll
        for (int m = 0; m < EPL; ++m) {
            av[m] = 0.0f;
            const int e = lane + kWave * m;
            we[m] = wr + (size_t)(e < E ? e : 0) * d;
        }
        for (int i = 0; i < d; i += 8) {
            const float4 x0 = *reinterpret_cast<const float4*>(xr + i);
            const float4 x1 = *reinterpret_cast<const float4*>(xr + i + 4);
            const float xv8[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            u32x4_t wq4[EPL];
#pragma unroll
            for (int m = 0; m < EPL; ++m) wq4[m] = *reinterpret_cast<const u32x4_t*>(we[m] + i);
#pragma unroll
            for (int m = 0; m < EPL; ++m) {
                const uint32_t wq[4] = {wq4[m].x, wq4[m].y, wq4[m].z, wq4[m].w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    av[m] = fmaf(xv8[2 * q], __uint_as_float(wq[q] << 16), av[m]);
                    av[m] = fmaf(xv8[2 * q + 1], __uint_as_float(wq[q] & 0xffff0000u), av[m]);
                }
            }
        }
#pragma unroll
        for (int m = 0; m < EPL; ++m) {
            const int e = lane + kWave * m;
            if (e < E) ssig[e] = sigmoid_fp32(av[m]);
        }
        __syncthreads();
        exact_select_wave(ssig, bias, E, K, tu, lane, topk_idx, topk_gate);
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

int router_cand_slots(int K) { return K <= 8 ? 16 : 32; }

float router_fast_bound_constant(int d) {
    const double u = 1.0 / 16777216.0;
    const double gamma = d * u / (1.0 - d * u);
    return (float)((gamma + 4.0 * d * u) * 1.01);
}

bool router_small_batch(const moe_desc_t& d) { return d.T < 256 * 64; }

bool router_small_fused(const moe_desc_t& d) {
    return router_small_batch(d) && d.K <= 8 && d.E <= 256 && d.d <= 4096;
}

hipError_t launch_router_fast_finish(const moe_desc_t& d, const float* s_fast, int ld, int nsplit, const void* x,
                                     const float* xnorm2, const void* w_router, const float* bias, float* wnorm,
                                     float* wr32, const float* wsq,
                                     uint16_t* cand, int32_t* ncand, int32_t* ovf_count, int32_t* ovf_list,
                                     int32_t* topk_idx, float* topk_gate, hipStream_t s) {
    const bf16_t* xb = static_cast<const bf16_t*>(x);
    const bf16_t* wb = static_cast<const bf16_t*>(w_router);
    if (nsplit < 1 || nsplit > 8) return hipErrorInvalidValue;  // the candidate kernels add at most 8 parts
    if (wsq) {  // one launch: norms, candidates, chains, selection and overflow
        if (!router_small_fused(d)) return hipErrorInvalidValue;
        const size_t shm = router_small_lds_bytes(d.d);
        auto launch = [&](auto kern) -> hipError_t {
            if (shm > 65536) {
                const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL(kern, dim3((d.T + 3) / 4), dim3(kWave), shm, s, s_fast, nsplit, (size_t)d.T * ld, ld,
                               wsq, xb, wb, bias, d.T, d.d, d.E, d.K, router_fast_bound_constant(d.d), topk_idx,
                               topk_gate);
            return hipGetLastError();
        };
        if (d.E <= 64) return launch(k_router_small<4>);
        if (d.E <= 128) return launch(k_router_small<8>);
        return launch(k_router_small<16>);
    }
    const bool small = router_small_batch(d);
    // Weight-row norms (the token norms are formed in the candidate kernel);
    // for small batches also the fp32 copy of the weights the chains read.
    hipLaunchKernelGGL(k_row_norms, dim3((d.E + 3) / 4), dim3(256), 0, s, wb, d.E, wnorm, nullptr, 0, nullptr, d.d,
                       ovf_count, small ? wr32 : nullptr);
    const size_t sstride = (size_t)d.T * ld;
    const float cst = router_fast_bound_constant(d.d);
    const int ns = router_cand_slots(d.K);
    // Candidates: 16 lanes per token (64 for more than 256 experts); blocks
    // of one wave for small batches, so that every CU gets work.
    const int cand_threads = d.T >= 16384 ? 256 : kWave;
#define MOE_CAND(LPAv, PERv, NSv)                                                                           \
    hipLaunchKernelGGL((nsplit > 1 ? k_router_cand<LPAv, PERv, NSv, true> : k_router_cand<LPAv, PERv, NSv, false>), \
                       dim3((d.T + cand_threads / LPAv - 1) / (cand_threads / LPAv)), dim3(cand_threads), 0, s, \
                       s_fast, xb, xnorm2, d.d, wnorm, bias, d.T, d.E, ld, d.K, cst, cand, ncand, ovf_count,    \
                       ovf_list, nsplit, sstride)
    // E / LPA experts per lane (at least 4), so that every lane of a token
    // holds experts and L is taken over all of them.
    if (d.E <= 64) { if (ns == 16) MOE_CAND(16, 4, 16); else MOE_CAND(16, 4, 32); }
    else if (d.E <= 128) { if (ns == 16) MOE_CAND(16, 8, 16); else MOE_CAND(16, 8, 32); }
    else if (d.E <= 256) { if (ns == 16) MOE_CAND(16, 16, 16); else MOE_CAND(16, 16, 32); }
    else if (d.E <= 512) { if (ns == 16) MOE_CAND(64, 8, 16); else MOE_CAND(64, 8, 32); }
    else { if (ns == 16) MOE_CAND(64, 16, 16); else MOE_CAND(64, 16, 32); }
#undef MOE_CAND
    // Exact chains: 256 (or 128) tokens per block of 1024 threads while that
    // still gives a block per CU, then 64 tokens per block, then (small
    // batches) one wave per 4 (or 2) tokens reading weights directly.
#define MOE_CHAIN(TPBv, LPTv, CPLv, EMv, DCv)                                                               \
    hipLaunchKernelGGL((k_router_chain<TPBv, LPTv, CPLv, EMv, DCv>), dim3((d.T + TPBv - 1) / TPBv + 64),     \
                       dim3(TPBv * LPTv), 0, s, xb, wb, bias, cand, ncand, d.T, d.d, d.E, d.K, topk_idx, topk_gate, \
                       (d.T + TPBv - 1) / TPBv, ovf_count, ovf_list)
#define MOE_CHAIN_E(TPBv, LPTv, CPLv, DCv)                                                                     \
    do {                                                                                                    \
        if (d.E <= 64) MOE_CHAIN(TPBv, LPTv, CPLv, 64, DCv);                                                \
        else if (d.E <= 256) MOE_CHAIN(TPBv, LPTv, CPLv, 256, DCv);                                         \
        else MOE_CHAIN(TPBv, LPTv, CPLv, 1024, 16);                                                         \
    } while (0)
    const int big_tpb = ns == 16 ? 256 : 128;
    if (d.T >= 256 * big_tpb) {
        if (ns == 16) MOE_CHAIN_E(256, 4, 4, 64); else MOE_CHAIN_E(128, 8, 4, 64);
    } else if (d.T >= 256 * 64) {
        if (ns == 16) MOE_CHAIN_E(64, 4, 4, 64); else MOE_CHAIN_E(64, 8, 4, 64);
    } else {
        // One wave per 64 / ns tokens, fp32 weights straight from global
        // memory; 64 more one-wave blocks route the overflow queue.
        const int tpb = kWave / ns;
        const size_t sel = (size_t)tpb * (ns * 12 + kMaxK * 8);
        const size_t xs = (size_t)tpb * d.d * 4;
        const size_t shm = xs > sel ? xs : sel;
        const int chain_blocks = (d.T + tpb - 1) / tpb;
        const dim3 grid(chain_blocks + 64);
        auto launch = [&](auto kern) -> hipError_t {
            if (shm > 65536) {  // x rows of d > 4096 in LDS
                const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL(kern, grid, dim3(kWave), shm, s, xb, wr32, wb, bias, cand, ncand, d.T, d.d, d.E, d.K,
                               topk_idx, topk_gate, chain_blocks, ovf_count, ovf_list);
            return hipGetLastError();
        };
        return ns == 16 ? launch(k_router_chain_direct<16>) : launch(k_router_chain_direct<32>);
    }
#undef MOE_CHAIN_E
#undef MOE_CHAIN
    return hipGetLastError();
}

}  // namespace moe
