// Loss-free load balancing: the update of the selection bias from one
// iteration's per-expert token counts (paper Sec. 3.2 "Load Balancing":
// Eq. (8) sign rule, Eq. (9) z-score rule).
//
// The counts are what the permutation produces (tokens routed to each
// expert). The sign rule decides sign(t_e - mean) exactly on integers
// (E t_e against the sum) and moves b_e by one fp32 add of -alpha or +alpha.
// The z-score rule uses the population standard deviation over the E experts
// in double precision, in a fixed order (mean by one division; variance as a
// sum over ascending e of separately rounded squares; correctly rounded
// square root; z by one division; b - alpha z; one rounding to fp32), so the
// result is reproducible bit for bit. A zero deviation (all counts equal)
// leaves the bias unchanged. Built without multiply-add contraction.
#include "moe_internal.h"

#include <math.h>

namespace moe {
namespace {

__global__ __launch_bounds__(1024) void k_bias_update(const int32_t* __restrict__ counts, float* __restrict__ bias,
                                                      int E, float alpha, int rule) {
    __shared__ int32_t cnt[kMaxE];
    __shared__ long long s_total;
    __shared__ double s_mean, s_dev;
    for (int e = threadIdx.x; e < E; e += blockDim.x) cnt[e] = counts[e];
    __syncthreads();
    if (threadIdx.x == 0) {
        // One thread, ascending e: the order the rule's rounding is defined in
        // (E <= 1024 terms, from LDS).
        long long total = 0;
        for (int e = 0; e < E; ++e) total += cnt[e];
        double mean = 0.0, dev = 0.0;
        if (rule == MOE_BIAS_ZSCORE) {
            mean = (double)total / (double)E;
            double var = 0.0;
            for (int e = 0; e < E; ++e) {
                const double diff = (double)cnt[e] - mean;
                const double sq = diff * diff;
                var = var + sq;
            }
            var = var / (double)E;
            dev = sqrt(var);
        }
        s_total = total;
        s_mean = mean;
        s_dev = dev;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        if (rule == MOE_BIAS_SIGN) {
            const long long scaled = (long long)E * cnt[e];
            if (scaled > s_total) bias[e] = bias[e] - alpha;
            else if (scaled < s_total) bias[e] = bias[e] + alpha;
        } else if (s_dev != 0.0) {
            const double z = ((double)cnt[e] - s_mean) / s_dev;
            const double step = (double)alpha * z;
            bias[e] = (float)((double)bias[e] - step);
        }
    }
}

}  // namespace

hipError_t launch_bias_update(int32_t E, const int32_t* counts, float* bias, float alpha, int32_t rule,
                              hipStream_t s) {
    hipLaunchKernelGGL(k_bias_update, dim3(1), dim3(1024), 0, s, counts, bias, (int)E, alpha, (int)rule);
    return hipGetLastError();
}

}  // namespace moe
