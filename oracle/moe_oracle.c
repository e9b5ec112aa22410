/*
 * Plain CPU oracle of one fine-grained Mixture-of-Experts MLP layer, as the
 * MoE-ViE paper states it.
 *
 *   TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU
 *   baseline leg of the benchmark may load this library. The GPU path never
 *   calls it, shares no code with it, and fails loudly when its own HIP
 *   library is missing instead of falling back to this.
 *
 * What it computes (paper references are to sections and equations):
 *   router logits        s = W_r x                            Sec. 3.1, Eq. (1)
 *   sigmoid gating       g = top-k(Sigmoid(s)), renormalised   Sec. 3.2, Eqs. (4)-(5)
 *   selection bias       select by top-k(Sigmoid(s) + b)       Sec. 3.2 "Load Balancing", Eq. (7)
 *   layer output         y = sum_T g'_e E_e(x) + lambda * shared(x)   Eq. (6)
 *   permutation          sort slots by expert, bincount, cumsum       App. "MoE Kernel", Algorithm 1 Phase 1
 *   expert MLP           E(x) = W2 GELU(W1 x), no linear biases
 *   SwiGLU expert MLP    E(x) = W2 (SiLU(W1 x) * (W3 x))   App. "MoE Kernel", Algorithm 1 Phase 2
 *   bias update          b_e -= alpha sign(t_e - mu)  or  alpha (t_e - mu) / sigma
 *                                                       Sec. 3.2 "Load Balancing", Eqs. (8)-(9)
 *   expert backward      dx, dW1, dW2 of the expert MLP given the gradient of
 *                        its output (the grouped training GEMMs with the
 *                        activation as a separate step, App. "MoE Kernel",
 *                        the paragraph after Algorithm 1): the chain rule
 *
 * Precision. Everything that is a plain definition (expert MLPs, combine) is
 * evaluated in double precision. Routing decides integers (which experts a
 * token uses), so it is evaluated in the kernel's precision, fp32, following
 * two fixed recipes that the GPU path implements independently:
 *   recipe R  logit = fp32 sequential fused multiply-add chain over the model
 *             width in ascending index order, starting from +0;
 *   recipe S  sigmoid(s) = 1 / (1 + exp(-s)) with exp evaluated by Cody-Waite
 *             range reduction (Cody & Waite, 1980) and a degree-7 Taylor
 *             polynomial, from correctly rounded fp32 operations only.
 * Gates are then fp32 as well, so indices and gates are comparable bit for bit.
 *
 * Readings of points the paper leaves open:
 *   - the bias b only selects experts; gate values use the unbiased sigmoid
 *     renormalised over the chosen K;
 *   - ties in the selection key go to the lower expert index; the K slots of a
 *     token are ordered by descending key;
 *   - the shared expert is a separate always-on MLP of its own width, weight
 *     lambda, no gate;
 *   - in a bf16 layer the expert activation GELU(W1 x) is materialised in bf16
 *     (round to nearest even) before fc2, as the paper's kernel writes its
 *     activation tile to a buffer; nothing else is rounded here.
 *   - backward: the same rounding points as the forward for the activation
 *     (bf16 layers round act(W1 x) to bf16, which dW2 then uses), and in a
 *     bf16 layer the gradient of the pre-activation (GELU: dH; SwiGLU: dG and
 *     dU) is rounded to bf16, the operand of the dx and dW1 products. Weight
 *     gradients are sums over the expert's rows; nothing else is rounded.
 *   - bias update: t_e is the number of tokens routed to expert e (the
 *     permutation's counts), mu their mean over the E experts, sigma their
 *     standard deviation over the E experts (the whole population: divided
 *     by E); sign(0) = 0; when sigma = 0 (all counts equal) the z-score
 *     update changes nothing. The sign decision is exact (E t_e against the
 *     integer sum); the sign update is one fp32 add of -alpha, +alpha or
 *     nothing. The z-score update is evaluated in double precision in a fixed
 *     order (mean by one division, variance summed over e ascending with a
 *     separate multiply and add, correctly rounded square root) and rounded
 *     to fp32 once, so an implementation following the same order agrees
 *     bit for bit.
 *
 * Build: gcc -O2 -mfma -ffp-contract=off -fopenmp -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_VERSION 1

int oracle_version(void) { return ORACLE_VERSION; }

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---------------------------------------------------------------- recipe S */

/* Constants of recipe S, each derived from its definition:
 *   LOG2E      = fl32(1 / ln 2)
 *   LN2_HI     = ln 2 rounded to 15 significant bits (22713 * 2^-15), so
 *                n * LN2_HI is exact for |n| <= 126
 *   LN2_LO     = fl32(ln 2 - LN2_HI)
 *   C_k        = fl32(1 / k!) for k = 0..7                                   */
static const float S_LOG2E = 0x1.715476p+0f;
static const float S_LN2_HI = 0x1.62e4p-1f;
static const float S_LN2_LO = 0x1.7f7d1cp-20f;

float oracle_sigmoid(float s) {
    const float c2 = 1.0f / 2.0f, c3 = 1.0f / 6.0f, c4 = 1.0f / 24.0f;
    const float c5 = 1.0f / 120.0f, c6 = 1.0f / 720.0f, c7 = 1.0f / 5040.0f;
    /* exp(z) with z = -s, clamped so that exp(z) and the result stay normal. */
    float z = -s;
    if (z > 87.0f) z = 87.0f;
    if (z < -87.0f) z = -87.0f;
    float zl = z * S_LOG2E;
    float n = rintf(zl);
    float r = fmaf(-n, S_LN2_HI, z);
    r = fmaf(-n, S_LN2_LO, r);
    /* Taylor polynomial of exp(r), Horner form, highest degree first. */
    float p = c7;
    p = fmaf(p, r, c6);
    p = fmaf(p, r, c5);
    p = fmaf(p, r, c4);
    p = fmaf(p, r, c3);
    p = fmaf(p, r, c2);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    float e = ldexpf(p, (int)n);
    float den = 1.0f + e;
    return 1.0f / den;
}

/* ---------------------------------------------------------------- recipe R */

/* Router logit s_e = sum_i x_i W_r[e, i] (Eq. (1)), fp32 sequential FMA chain. */
static float logit_r(const float *x, const float *w, int d) {
    float s = 0.0f;
    for (int i = 0; i < d; ++i) s = fmaf(x[i], w[i], s);
    return s;
}

void oracle_logits(int T, int d, int E, const float *x, const float *wr, float *logits) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t)
        for (int e = 0; e < E; ++e)
            logits[(size_t)t * E + e] = logit_r(x + (size_t)t * d, wr + (size_t)e * d, d);
}

/* Sigmoid scores of every expert for every token (recipes R and S). */
void oracle_scores(int T, int d, int E, const float *x, const float *wr, float *scores) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t)
        for (int e = 0; e < E; ++e)
            scores[(size_t)t * E + e] =
                oracle_sigmoid(logit_r(x + (size_t)t * d, wr + (size_t)e * d, d));
}

/* ------------------------------------------------------------------ route */

/* Top-K of one token from its sigmoid scores sig[E] and the selection bias
 * (Eq. (7)); gates renormalise the unbiased scores of the chosen experts
 * (Eq. (5)). Key a beats key b when a > b, or a == b and a's index is lower. */
static void select_topk(int E, int K, const float *sig, const float *bias,
                        int32_t *idx, float *gate, unsigned char *taken) {
    memset(taken, 0, (size_t)E);
    for (int j = 0; j < K; ++j) {
        int best = -1;
        float best_key = 0.0f;
        for (int e = 0; e < E; ++e) {
            if (taken[e]) continue;
            float key = bias ? sig[e] + bias[e] : sig[e];
            if (best < 0 || key > best_key) { best = e; best_key = key; }
        }
        taken[best] = 1;
        idx[j] = best;
    }
    float den = sig[idx[0]];
    for (int j = 1; j < K; ++j) den = den + sig[idx[j]];
    for (int j = 0; j < K; ++j) gate[j] = sig[idx[j]] / den;
}

/* Routing of T tokens: topk_idx[T, K] (int32) and topk_gate[T, K] (fp32).
 * bias may be NULL (no selection bias). */
void oracle_route(int T, int d, int E, int K, const float *x, const float *wr,
                  const float *bias, int32_t *topk_idx, float *topk_gate) {
#pragma omp parallel
    {
        float *sig = (float *)malloc(sizeof(float) * (size_t)E);
        unsigned char *taken = (unsigned char *)malloc((size_t)E);
#pragma omp for schedule(static)
        for (int t = 0; t < T; ++t) {
            for (int e = 0; e < E; ++e)
                sig[e] = oracle_sigmoid(logit_r(x + (size_t)t * d, wr + (size_t)e * d, d));
            select_topk(E, K, sig, bias, topk_idx + (size_t)t * K, topk_gate + (size_t)t * K, taken);
        }
        free(sig);
        free(taken);
    }
}

/* Top-K from precomputed scores (used to study a bias vector without
 * recomputing logits). Same rules as oracle_route. */
void oracle_topk_from_scores(int T, int E, int K, const float *scores, const float *bias,
                             int32_t *topk_idx, float *topk_gate) {
#pragma omp parallel
    {
        unsigned char *taken = (unsigned char *)malloc((size_t)E);
#pragma omp for schedule(static)
        for (int t = 0; t < T; ++t)
            select_topk(E, K, scores + (size_t)t * E, bias, topk_idx + (size_t)t * K,
                        topk_gate + (size_t)t * K, taken);
        free(taken);
    }
}

/* ---------------------------------------------------------------- permute */

/* Algorithm 1, Phase 1: group the T*K slots (slot n = t*K + j) by expert.
 *   counts[e]            BinCount of the flattened expert ids
 *   offsets[0..E]        exclusive cumulative sum of counts
 *   sorted_slots[...]    slot ids in stable sorted-by-expert order: within an
 *                        expert, ascending slot id                          */
void oracle_permute(int T, int E, int K, const int32_t *topk_idx, int32_t *counts,
                    int32_t *offsets, int32_t *sorted_slots) {
    size_t n_slots = (size_t)T * K;
    for (int e = 0; e < E; ++e) counts[e] = 0;
    for (size_t n = 0; n < n_slots; ++n) counts[topk_idx[n]] += 1;
    offsets[0] = 0;
    for (int e = 0; e < E; ++e) offsets[e + 1] = offsets[e] + counts[e];
    int32_t *fill = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
    for (int e = 0; e < E; ++e) fill[e] = offsets[e];
    for (size_t n = 0; n < n_slots; ++n) sorted_slots[fill[topk_idx[n]]++] = (int32_t)n;
    free(fill);
}

/* ------------------------------------------------------------ expert MLP */

/* GELU with the exact Gaussian CDF: v * Phi(v) = 0.5 v (1 + erf(v / sqrt 2)). */
double oracle_gelu(double v) { return 0.5 * v * (1.0 + erf(v * 0.70710678118654752440)); }

/* Nearest bf16 value (ties to even) of a finite double in the normal bf16 range. */
double oracle_round_bf16(double v) {
    if (v == 0.0) return v;
    int ex;
    double m = frexp(v, &ex);          /* v = m * 2^ex, 0.5 <= |m| < 1 */
    double q = nearbyint(ldexp(m, 8)); /* 8 significant bits, ties to even */
    return ldexp(q, ex - 8);
}

/* SiLU (swish): v * Sigmoid(v) = v / (1 + exp(-v)). */
double oracle_silu(double v) { return v / (1.0 + exp(-v)); }

/* One expert MLP applied to one input row: out = W2 act(W1 x), with
 *   GELU experts (swiglu = 0):   act(W1 x) = GELU(W1 x), w1[h, d];
 *   SwiGLU experts (swiglu = 1): act = SiLU(W1 x) * (W3 x) elementwise, w1 holds
 *                                W1 (gate) rows 0..h-1 then W3 (up) rows h..2h-1.
 *   x[d], w2[d, h], hid[h] scratch; row k of W1 / W3 is hidden unit k. */
static void expert_row(int d, int h, int swiglu, const float *x, const float *w1, const float *w2,
                       int act_bf16, double *hid, double *out) {
    for (int k = 0; k < h; ++k) {
        const float *w = w1 + (size_t)k * d;
        double a = 0.0;
        for (int i = 0; i < d; ++i) a += (double)w[i] * (double)x[i];
        if (swiglu) {
            const float *wu = w1 + ((size_t)h + k) * d;
            double up = 0.0;
            for (int i = 0; i < d; ++i) up += (double)wu[i] * (double)x[i];
            a = oracle_silu(a) * up;
        } else {
            a = oracle_gelu(a);
        }
        hid[k] = act_bf16 ? oracle_round_bf16(a) : a;
    }
    for (int c = 0; c < d; ++c) {
        const float *w = w2 + (size_t)c * h;
        double o = 0.0;
        for (int k = 0; k < h; ++k) o += (double)w[k] * hid[k];
        out[c] = o;
    }
}

static void expert_rows(int n, int d, int h, int swiglu, const float *rows, const float *w1,
                        const float *w2, int act_bf16, double *out) {
#pragma omp parallel
    {
        double *hid = (double *)malloc(sizeof(double) * (size_t)h);
#pragma omp for schedule(static)
        for (int r = 0; r < n; ++r)
            expert_row(d, h, swiglu, rows + (size_t)r * d, w1, w2, act_bf16, hid, out + (size_t)r * d);
        free(hid);
    }
}

/* out[n, :] = W2 act(W1 rows[n, :]) for n rows through one expert's weights. */
void oracle_expert_rows(int n, int d, int h, const float *rows, const float *w1,
                        const float *w2, int act_bf16, double *out) {
    expert_rows(n, d, h, 0, rows, w1, w2, act_bf16, out);
}

/* The same with a SwiGLU expert: w13[2h, d] (gate rows, then up rows). */
void oracle_expert_rows_swiglu(int n, int d, int h, const float *rows, const float *w13,
                               const float *w2, int act_bf16, double *out) {
    expert_rows(n, d, h, 1, rows, w13, w2, act_bf16, out);
}

/* ------------------------------------------------------- expert backward */

/* d/dv GELU(v) = Phi(v) + v phi(v), Phi the standard normal CDF and phi its
 * density. */
double oracle_gelu_grad(double v) {
    return 0.5 * (1.0 + erf(v * 0.70710678118654752440)) + v * exp(-0.5 * v * v) * 0.39894228040143267794;
}

/* d/dv SiLU(v) = s (1 + v (1 - s)) with s = Sigmoid(v) = 1 / (1 + exp(-v)). */
double oracle_silu_grad(double v) {
    const double sg = 1.0 / (1.0 + exp(-v));
    return sg * (1.0 + v * (1.0 - sg));
}

/* Backward of one expert MLP over n rows (the chain rule, term by term).
 * Forward per row r (x = rows[r], out = W2 a):
 *   GELU experts:   p = W1 x, a = GELU(p)
 *   SwiGLU experts: p = W1 x (gate), q = W3 x (up), a = SiLU(p) * q
 * Given G = go[r] = dL/d out:
 *   da    = W2^T G
 *   GELU:   dp = da * GELU'(p)
 *   SwiGLU: dp = da * q * SiLU'(p),  dq = da * SiLU(p)
 *   dx[r] = W1^T dp (+ W3^T dq)
 *   dW2  += G a^T,  dW1 += dp x^T  (dW3 += dq x^T)
 * act_bf16: a, dp and dq are rounded to bf16 where they are formed.
 * Shapes: rows, go, dx [n, d]; w1 and dw1 [h, d] (SwiGLU [2h, d]: gate rows,
 * then up rows); w2 and dw2 [d, h]. dw1 and dw2 are overwritten with the sums
 * over the n rows, taken in ascending row order. */
static void expert_backward(int n, int d, int h, int swiglu, const float *rows, const float *w1,
                            const float *w2, const float *go, int act_bf16, double *dx, double *dw1,
                            double *dw2) {
    const int hr = swiglu ? 2 * h : h;              /* rows of w1 and dw1 */
    double *act = (double *)malloc(sizeof(double) * (size_t)n * h);
    double *dpre = (double *)malloc(sizeof(double) * (size_t)n * hr); /* dp rows, then dq rows */
#pragma omp parallel
    {
        double *da = (double *)malloc(sizeof(double) * (size_t)h);
#pragma omp for schedule(static)
        for (int r = 0; r < n; ++r) {
            const float *x = rows + (size_t)r * d;
            const float *g = go + (size_t)r * d;
            for (int k = 0; k < h; ++k) {
                double acc = 0.0;
                for (int c = 0; c < d; ++c) acc += (double)w2[(size_t)c * h + k] * (double)g[c];
                da[k] = acc;
            }
            for (int k = 0; k < h; ++k) {
                const float *wg = w1 + (size_t)k * d;
                double p = 0.0;
                for (int i = 0; i < d; ++i) p += (double)wg[i] * (double)x[i];
                double a, dp, dq = 0.0;
                if (swiglu) {
                    const float *wu = w1 + ((size_t)h + k) * d;
                    double q = 0.0;
                    for (int i = 0; i < d; ++i) q += (double)wu[i] * (double)x[i];
                    a = oracle_silu(p) * q;
                    dp = da[k] * q * oracle_silu_grad(p);
                    dq = da[k] * oracle_silu(p);
                } else {
                    a = oracle_gelu(p);
                    dp = da[k] * oracle_gelu_grad(p);
                }
                act[(size_t)r * h + k] = act_bf16 ? oracle_round_bf16(a) : a;
                dpre[(size_t)r * hr + k] = act_bf16 ? oracle_round_bf16(dp) : dp;
                if (swiglu) dpre[(size_t)r * hr + h + k] = act_bf16 ? oracle_round_bf16(dq) : dq;
            }
            for (int i = 0; i < d; ++i) {
                double acc = 0.0;
                for (int k = 0; k < hr; ++k) acc += (double)w1[(size_t)k * d + i] * dpre[(size_t)r * hr + k];
                dx[(size_t)r * d + i] = acc;
            }
        }
        free(da);
    }
#pragma omp parallel for schedule(static)
    for (int c = 0; c < d; ++c)
        for (int k = 0; k < h; ++k) {
            double acc = 0.0;
            for (int r = 0; r < n; ++r) acc += (double)go[(size_t)r * d + c] * act[(size_t)r * h + k];
            dw2[(size_t)c * h + k] = acc;
        }
#pragma omp parallel for schedule(static)
    for (int k = 0; k < hr; ++k)
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int r = 0; r < n; ++r) acc += dpre[(size_t)r * hr + k] * (double)rows[(size_t)r * d + i];
            dw1[(size_t)k * d + i] = acc;
        }
    free(act);
    free(dpre);
}

void oracle_expert_backward(int n, int d, int h, const float *rows, const float *w1, const float *w2,
                            const float *go, int act_bf16, double *dx, double *dw1, double *dw2) {
    expert_backward(n, d, h, 0, rows, w1, w2, go, act_bf16, dx, dw1, dw2);
}

void oracle_expert_backward_swiglu(int n, int d, int h, const float *rows, const float *w13, const float *w2,
                                   const float *go, int act_bf16, double *dx, double *dw13, double *dw2) {
    expert_backward(n, d, h, 1, rows, w13, w2, go, act_bf16, dx, dw13, dw2);
}

/* --------------------------------------------------------------- combine */

/* Eq. (6): y[t] = sum_j g[t, j] * O[t*K + j] + lambda * S[t].
 * expert_out is in slot order [T*K, d]; shared may be NULL. */
void oracle_combine(int T, int d, int K, const double *expert_out, const float *gate,
                    const double *shared, double lambda, double *y) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int j = 0; j < K; ++j)
                acc += (double)gate[(size_t)t * K + j] * expert_out[((size_t)t * K + j) * d + c];
            if (shared) acc += lambda * shared[(size_t)t * d + c];
            y[(size_t)t * d + c] = acc;
        }
    }
}

/* ----------------------------------------------------------------- layer */

/* The whole layer for a set of tokens, straight from the per-token definition
 * (Eqs. (1), (4)-(7)): route the token, run its K chosen experts and the shared
 * expert, mix. tok lists n_tok token ids (NULL means tokens 0..n_tok-1); the
 * outputs are indexed by position in that list:
 *   idx_out[n_tok, K], gate_out[n_tok, K] (either may be NULL), y_out[n_tok, d].
 * Shapes: x[T, d], wr[E, d], bias[E] or NULL, w1[E, h, d], w2[E, d, h],
 * w1s[hs, d], w2s[d, hs] (hs == 0: no shared expert, w1s/w2s ignored). */
static void layer(int n_tok, const int32_t *tok, int d, int E, int K, int h, int hs, int swiglu,
                  float lambda, int act_bf16, const float *x, const float *wr, const float *bias,
                  const float *w1, const float *w2, const float *w1s, const float *w2s,
                  int32_t *idx_out, float *gate_out, double *y_out) {
    const size_t w1_rows = swiglu ? 2 * (size_t)h : (size_t)h; /* rows of one expert's W1 (and W3) */
#pragma omp parallel
    {
        int hmax = h > hs ? h : hs;
        float *sig = (float *)malloc(sizeof(float) * (size_t)E);
        unsigned char *taken = (unsigned char *)malloc((size_t)E);
        double *hid = (double *)malloc(sizeof(double) * (size_t)(hmax > 0 ? hmax : 1));
        double *o = (double *)malloc(sizeof(double) * (size_t)d);
        int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)K);
        float *g = (float *)malloc(sizeof(float) * (size_t)K);
#pragma omp for schedule(dynamic, 1)
        for (int p = 0; p < n_tok; ++p) {
            int t = tok ? tok[p] : p;
            const float *xt = x + (size_t)t * d;
            for (int e = 0; e < E; ++e) sig[e] = oracle_sigmoid(logit_r(xt, wr + (size_t)e * d, d));
            select_topk(E, K, sig, bias, idx, g, taken);
            double *y = y_out + (size_t)p * d;
            for (int c = 0; c < d; ++c) y[c] = 0.0;
            for (int j = 0; j < K; ++j) {
                int e = idx[j];
                expert_row(d, h, swiglu, xt, w1 + (size_t)e * w1_rows * d, w2 + (size_t)e * d * h, act_bf16,
                           hid, o);
                for (int c = 0; c < d; ++c) y[c] += (double)g[j] * o[c];
            }
            if (hs > 0) {
                expert_row(d, hs, swiglu, xt, w1s, w2s, act_bf16, hid, o);
                for (int c = 0; c < d; ++c) y[c] += (double)lambda * o[c];
            }
            if (idx_out) memcpy(idx_out + (size_t)p * K, idx, sizeof(int32_t) * (size_t)K);
            if (gate_out) memcpy(gate_out + (size_t)p * K, g, sizeof(float) * (size_t)K);
        }
        free(sig);
        free(taken);
        free(hid);
        free(o);
        free(idx);
        free(g);
    }
}

void oracle_layer(int n_tok, const int32_t *tok, int T, int d, int E, int K, int h, int hs,
                  float lambda, int act_bf16, const float *x, const float *wr, const float *bias,
                  const float *w1, const float *w2, const float *w1s, const float *w2s,
                  int32_t *idx_out, float *gate_out, double *y_out) {
    (void)T;
    layer(n_tok, tok, d, E, K, h, hs, 0, lambda, act_bf16, x, wr, bias, w1, w2, w1s, w2s, idx_out, gate_out,
          y_out);
}

/* The layer with SwiGLU experts (routed and shared): w13[E, 2h, d] and
 * w13s[2hs, d] hold the gate rows then the up rows of each expert. */
void oracle_layer_swiglu(int n_tok, const int32_t *tok, int T, int d, int E, int K, int h, int hs,
                         float lambda, int act_bf16, const float *x, const float *wr, const float *bias,
                         const float *w13, const float *w2, const float *w13s, const float *w2s,
                         int32_t *idx_out, float *gate_out, double *y_out) {
    (void)T;
    layer(n_tok, tok, d, E, K, h, hs, 1, lambda, act_bf16, x, wr, bias, w13, w2, w13s, w2s, idx_out, gate_out,
          y_out);
}

/* Loss-free balancing bias update (Sec. 3.2 "Load Balancing"): rule 0 is the
 * sign update of Eq. (8), rule 1 the z-score update of Eq. (9). counts[E]
 * are the tokens routed to each expert in this iteration; bias[E] is updated
 * in place with step alpha. */
void oracle_bias_update(int E, const int32_t *counts, float *bias, float alpha, int rule) {
    long long total = 0;
    for (int e = 0; e < E; ++e) total += counts[e];
    if (rule == 0) {
        for (int e = 0; e < E; ++e) {
            long long scaled = (long long)E * counts[e]; /* compare t_e with total / E exactly */
            if (scaled > total) bias[e] = bias[e] - alpha;
            else if (scaled < total) bias[e] = bias[e] + alpha;
        }
        return;
    }
    double mu = (double)total / (double)E;
    double var = 0.0;
    for (int e = 0; e < E; ++e) {
        double dev = (double)counts[e] - mu;
        double sq = dev * dev;
        var = var + sq;
    }
    var = var / (double)E;
    double sigma = sqrt(var);
    if (sigma == 0.0) return;
    for (int e = 0; e < E; ++e) {
        double z = ((double)counts[e] - mu) / sigma;
        double step = (double)alpha * z;
        bias[e] = (float)((double)bias[e] - step);
    }
}
