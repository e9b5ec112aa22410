// Host side of the C ABI declared in include/moe_vie.h: argument validation
// (before anything is enqueued), the workspace layout, and the stream-ordered
// kernel sequence of each entry point. No host synchronisation anywhere.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>

#include "moe_internal.h"

#define MOE_API extern "C" __attribute__((visibility("default")))

namespace moe {

int32_t permute_blocks(int64_t n_slots, int32_t E);

namespace {

thread_local char g_err[512];

moe_status_t vfail(moe_status_t st, const char* fmt, va_list ap) {
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    return st;
}

moe_status_t fail(moe_status_t st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vfail(st, fmt, ap);
    va_end(ap);
    return st;
}

moe_status_t ok() {
    g_err[0] = 0;
    return MOE_OK;
}

}  // namespace

moe_status_t set_last_error(moe_status_t st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vfail(st, fmt, ap);
    va_end(ap);
    return st;
}

namespace {

moe_status_t hip_fail(hipError_t e, const char* where) {
    return fail(MOE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool dim_ok(int32_t v, int32_t lo) { return v >= lo && v <= 8192; }

moe_status_t check_desc(const moe_desc_t* d) {
    if (!d) return fail(MOE_ERR_INVALID_ARG, "desc is NULL");
    if (d->dtype != MOE_F32 && d->dtype != MOE_BF16)
        return fail(MOE_ERR_UNSUPPORTED, "dtype %d is not MOE_F32 or MOE_BF16", d->dtype);
    if (d->flags & ~(MOE_FLAG_EXACT_ROUTER | MOE_FLAG_SWIGLU))
        return fail(MOE_ERR_INVALID_ARG, "unknown flags 0x%x", d->flags);
    const bool swiglu = d->flags & MOE_FLAG_SWIGLU;
    if (swiglu && d->dtype != MOE_BF16) return fail(MOE_ERR_UNSUPPORTED, "SwiGLU experts need a bf16 layer");
    if (d->T < 1) return fail(MOE_ERR_INVALID_ARG, "T = %d must be >= 1", d->T);
    if (d->K < 1 || d->K > kMaxK) return fail(MOE_ERR_INVALID_ARG, "K = %d must be in [1, %d]", d->K, kMaxK);
    if (d->E < d->K || d->E > kMaxE)
        return fail(MOE_ERR_INVALID_ARG, "E = %d must be in [K = %d, %d]", d->E, d->K, kMaxE);
    if ((int64_t)d->T * d->K >= ((int64_t)1 << 31))
        return fail(MOE_ERR_INVALID_ARG, "T*K = %lld must be < 2^31", (long long)d->T * d->K);
    const int32_t hmin = swiglu ? 1 : 64;
    if (!dim_ok(d->d, 64) || !dim_ok(d->h, hmin) || (d->h_shared != 0 && !dim_ok(d->h_shared, hmin)))
        return fail(MOE_ERR_INVALID_ARG, "d = %d, h = %d, h_shared = %d out of range [%d, 8192]", d->d, d->h,
                    d->h_shared, hmin);
    if (d->d % 64) return fail(MOE_ERR_UNSUPPORTED, "d = %d must be a multiple of 64", d->d);
    if (!swiglu && (d->h % 64 || d->h_shared % 64))
        return fail(MOE_ERR_UNSUPPORTED, "h = %d, h_shared = %d must be multiples of 64 (GELU experts)", d->h,
                    d->h_shared);
    if (!std::isfinite(d->lambda)) return fail(MOE_ERR_INVALID_ARG, "lambda is not finite");
    // GEMM operands are addressed through 32-bit buffer offsets.
    const uint64_t es = d->dtype == MOE_BF16 ? 2 : 4, lim = (uint64_t)1 << 32;
    if ((uint64_t)d->T * d->d * es >= lim || (uint64_t)d->T * d->K * act_stride(*d, d->h) * es >= lim ||
        (uint64_t)d->T * act_stride(*d, d->h_shared) * es >= lim)
        return fail(MOE_ERR_UNSUPPORTED, "x, the expert activations or the shared activations exceed 4 GiB");
    return MOE_OK;
}

// The backward supports bf16 layers (GELU or SwiGLU experts); its transposed
// operands and slot gradients are addressed through 32-bit buffer offsets.
moe_status_t check_backward_desc(const moe_desc_t* d) {
    const moe_status_t st = check_desc(d);
    if (st != MOE_OK) return st;
    if (d->dtype != MOE_BF16) return fail(MOE_ERR_UNSUPPORTED, "the backward needs a bf16 layer");
    const uint64_t lim = (uint64_t)1 << 32, TK = (uint64_t)d->T * d->K;
    const uint64_t ld = TK + 128 * (uint64_t)d->E + 64;
    const uint64_t hw = (uint64_t)act_stride(*d, d->h) * ((d->flags & MOE_FLAG_SWIGLU) ? 2 : 1);
    if (TK * d->d * 2 >= lim || TK * hw * 2 >= lim || (uint64_t)(d->d > hw ? d->d : hw) * ld * 2 >= lim)
        return fail(MOE_ERR_UNSUPPORTED, "the backward's slot or transposed operands exceed 4 GiB");
    return MOE_OK;
}

moe_status_t check_ptr(const void* p, const char* name, bool nullable = false) {
    if (!p) {
        if (nullable) return MOE_OK;
        return fail(MOE_ERR_INVALID_ARG, "%s is NULL", name);
    }
    if (reinterpret_cast<uintptr_t>(p) & 15u) return fail(MOE_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return MOE_OK;
}

#define CHECK(expr)                         \
    do {                                    \
        const moe_status_t _st = (expr);    \
        if (_st != MOE_OK) return _st;      \
    } while (0)

#define HIP_CHECK(expr, where)                      \
    do {                                            \
        const hipError_t _e = (expr);               \
        if (_e != hipSuccess) return hip_fail(_e, where); \
    } while (0)

size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

moe_status_t check_ws(const moe_desc_t& d, const void* ws, size_t bytes, WorkspacePlan* plan) {
    *plan = plan_workspace(d);
    if (!ws) return fail(MOE_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", plan->total);
    if (reinterpret_cast<uintptr_t>(ws) & 255u)
        return fail(MOE_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
    if (bytes < plan->total)
        return fail(MOE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, plan->total);
    return MOE_OK;
}

template <typename T>
T* region(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<uint8_t*>(ws) + off);
}

}  // namespace

size_t elem_size(int32_t dtype) { return dtype == MOE_BF16 ? 2 : 4; }

// Row stride of the router scores: E rounded up to 64, the column-tile width
// of the MFMA logits GEMM (columns past E are computed from zero weight rows).
static int32_t router_ld(const moe_desc_t& d) { return (d.E + 63) / 64 * 64; }

static bool fast_router(const moe_desc_t& d) { return d.dtype == MOE_BF16 && !(d.flags & MOE_FLAG_EXACT_ROUTER); }

// Rows of the router logits GEMM's M-tiles (256 once the batch gives each CU
// tiles of 256 rows, else 64).
static int router_bm(const moe_desc_t& d) { return (int64_t)d.T * router_ld(d) >= (int64_t)200 * 65536 ? 256 : 64; }

// K split of the fast router's logits GEMM. Small batches have too few
// 64-row tiles to occupy the chip (17 x 2 for one image against 256 CUs), so
// the d / 64 K slabs are split over up to 4 parts of at least two slabs, each
// writing its own partial logits; the candidate kernel adds them in order.
// (8 parts: one image's route 29 -> 31 us, the repair reading twice the
// partial logits.)
static int32_t router_splits(const moe_desc_t& d) {
    if (!fast_router(d) || router_bm(d) != 64 || d.T >= 8192) return 1;
    const int nk = d.d / 64;
    for (int p = 4; p >= 2; p /= 2)
        if (nk % p == 0 && nk / p >= 2) return p;
    return 1;
}

// Width of the router logits GEMM on the persistent kernel: the logit row
// rounded up to its 256-column tile.
static int32_t router_n256(const moe_desc_t& d) { return (router_ld(d) + 255) / 256 * 256; }

// Whether the router's logits GEMM runs on the persistent kernel and also
// forms the tokens' sums of squares: large batches (the 256-row tiles of at
// least 128 logit columns, rounded up to 256, give every CU a tile), no K
// split. The candidate kernel then reads T floats instead of x again (201 MB
// at ViT-G widths, 134 MB at ViT-L's). Rounding 128 columns up to 256 doubles
// that small GEMM's MFMA work, which costs less than the second read of x.
static bool router_norms_in_gemm(const moe_desc_t& d) {
    return fast_router(d) && router_ld(d) >= 128 && (int64_t)d.T * router_n256(d) >= (int64_t)200 * 65536 &&
           d.d >= 128 && router_splits(d) == 1;
}

WorkspacePlan plan_workspace(const moe_desc_t& d) {
    WorkspacePlan p;
    const size_t es = elem_size(d.dtype);
    const size_t TK = (size_t)d.T * d.K;
    p.n_hist_blocks = permute_blocks((int64_t)TK, d.E);
    p.tile_bm = gemm_tile_bm(d.dtype, (int64_t)TK / d.E);
    // The SwiGLU first layer runs on 256-row tiles only with two or more K slabs.
    if ((d.flags & MOE_FLAG_SWIGLU) && d.d < 128) p.tile_bm = 64;
    const size_t busy = TK < (size_t)d.E ? TK : (size_t)d.E;  // experts that can hold a slot
    p.max_tiles = (int32_t)((TK + busy * (p.tile_bm - 1)) / p.tile_bm);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes);
        return o;
    };
    p.idx = take(TK * 4);
    p.gate = take(TK * 4);
    p.router_splits = router_splits(d);
    p.scores = take((size_t)p.router_splits * d.T * router_ld(d) * 4);
    p.wnorm = take((size_t)d.E * 4);
    const bool small_fused = fast_router(d) && router_small_fused(d);
    p.wr32 = take(fast_router(d) && router_small_batch(d) && !small_fused ? (size_t)d.E * d.d * 4 : 0);
    p.wsq = take(small_fused ? (size_t)p.router_splits * router_ld(d) * 4 : 0);
    p.xnorm2 = take(router_norms_in_gemm(d) ? (size_t)d.T * 4 : 0);
    p.ovf = take((size_t)(d.T + 1) * 4);
    p.cand = take((size_t)d.T * router_cand_slots(d.K) * 2);
    p.ncand = take((size_t)d.T * 4);
    p.counts = take((size_t)d.E * 4);
    p.offsets = take((size_t)(d.E + 1) * 4);
    p.slots = take(TK * 4);
    p.blockhist = take((size_t)p.n_hist_blocks * d.E * 4);
    p.tiles = take((size_t)p.max_tiles * sizeof(TileDesc));
    p.ntiles = take(16);
    p.act = take(TK * act_stride(d, d.h) * es);
    p.eout = take(TK * d.d * es);
    p.sact = take((size_t)d.T * act_stride(d, d.h_shared) * es);
    p.sout = take(d.h_shared ? (size_t)d.T * d.d * 4 : 0);
    p.total = off;
    return p;
}

BackwardPlan plan_backward(const moe_desc_t& d) {
    BackwardPlan b;
    b.fwd = plan_workspace(d);
    const size_t TK = (size_t)d.T * d.K;
    b.ld = (int32_t)((TK + 128 * (size_t)d.E + 63) / 64 * 64);  // windows: >= 2 slabs, rounded up to one
    size_t off = b.fwd.total;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes);
        return o;
    };
    const bool sw = d.flags & MOE_FLAG_SWIGLU;
    b.hh = act_stride(d, d.h);
    b.hw = sw ? 2 * b.hh : b.hh;
    const size_t hh = b.hh, hw = b.hw;
    b.pre = take(TK * hw * 4);
    b.w1t = take((size_t)d.E * d.d * hw * 2);
    b.w2t = take((size_t)d.E * hh * d.d * 2);
    b.dh = take(TK * hw * 2);
    b.dxs = take(TK * d.d * 4);
    b.koff = take(((size_t)d.E + 1) * 4);
    b.gt = take((size_t)d.d * b.ld * 2);
    b.at = take(hh * b.ld * 2);
    b.dht = take(hw * b.ld * 2);
    b.xt = take((size_t)d.d * b.ld * 2);
    b.items_max = d.E + (int32_t)(((size_t)b.ld / 64 + kWgradSlabs - 1) / kWgradSlabs);
    b.items = take((size_t)b.items_max * sizeof(TileDesc));
    b.rlist = take((size_t)d.E * sizeof(TileDesc));
    b.wcount = take(16);
    b.partials = take((size_t)b.items_max * d.d * hw * 4);
    b.dw1p = (sw && b.hh != d.h) ? take((size_t)d.E * hw * d.d * 4) : 0;
    b.total = off;
    return b;
}

// Router and gating: exact chain for every logit, or MFMA logits plus exact
// repair of the candidates (same result).
static moe_status_t enqueue_route(const moe_desc_t& d, const WorkspacePlan& p, void* ws, const void* x,
                                  const void* w_router, const float* bias, int32_t* idx, float* gate,
                                  hipStream_t s) {
    float* scores = region<float>(ws, p.scores);
    if (!fast_router(d)) {
        HIP_CHECK(launch_router_scores(d, x, w_router, scores, s), "router scores");
        HIP_CHECK(launch_topk(d, scores, bias, idx, gate, s), "top-k");
        return MOE_OK;
    }
    GemmArgs g{};
    g.A = x;
    g.B = w_router;
    g.C = scores;
    g.dense_rows = d.T;
    g.N = router_ld(d);
    g.b_rows = d.E;
    g.Kdim = d.d;
    g.route_k = 1;
    g.row_mode = ROWS_IDENTITY;
    const int bm = router_bm(d);
    g.max_tiles = (d.T + bm - 1) / bm;
    g.a_bytes = (uint32_t)((size_t)d.T * d.d * 2);
    g.k_splits = p.router_splits;
    const bool norms = router_norms_in_gemm(d);
    float* xnorm2 = norms ? region<float>(ws, p.xnorm2) : nullptr;
    if (norms) {  // 256-column tiles; the columns past the logit row are not stored
        g.N = router_n256(d);
        g.ldc = router_ld(d);
        g.max_tiles = (d.T + 255) / 256;
        g.C2 = xnorm2;
    }
    // Small batches: the logits GEMM (64-row tiles) also forms the weight
    // rows' sums of squares per K part, and the repair is one launch.
    float* wsq = router_small_fused(d) ? region<float>(ws, p.wsq) : nullptr;
    if (wsq) g.C2 = wsq;
    HIP_CHECK(launch_gemm(d, norms ? EPI_ROUTER_F32 : EPI_STORE_F32, norms ? 256 : bm, g, s), "router logits gemm");
    int32_t* ovf = region<int32_t>(ws, p.ovf);
    HIP_CHECK(launch_router_fast_finish(d, scores, router_ld(d), p.router_splits, x, xnorm2, w_router, bias,
                                        region<float>(ws, p.wnorm),
                                        region<float>(ws, p.wr32), wsq, region<uint16_t>(ws, p.cand),
                                        region<int32_t>(ws, p.ncand), ovf, ovf + 1, idx, gate, s),
              "router repair");
    return MOE_OK;
}

// Routed experts: fc1 + GELU into the activation buffer (sorted order), then
// fc2 scattered to slot order.
static moe_status_t enqueue_routed_mlp(const moe_desc_t& d, const WorkspacePlan& p, void* ws, const void* x,
                                       const int32_t* sorted_slots, const int32_t* offsets, const void* w1,
                                       const void* w2, void* expert_out, hipStream_t s,
                                       void* const* events = nullptr, bool tiles_built = false) {
    TileDesc* tiles = region<TileDesc>(ws, p.tiles);
    int32_t* ntiles = region<int32_t>(ws, p.ntiles);
    if (!tiles_built)
        HIP_CHECK(launch_build_tiles(d.E, p.tile_bm, p.max_tiles, offsets, tiles, ntiles, s), "build_tiles");
    if (events) HIP_CHECK(hipEventRecord(static_cast<hipEvent_t>(events[0]), s), "event record");
    GemmArgs g{};
    g.A = x;
    g.B = w1;
    g.C = region<void>(ws, p.act);
    g.row_map = sorted_slots;
    g.tiles = tiles;
    g.n_tiles = ntiles;
    const bool swiglu = d.flags & MOE_FLAG_SWIGLU;
    const int32_t ldh = act_stride(d, d.h);
    g.N = d.h;
    g.Kdim = d.d;
    g.route_k = d.K;
    g.row_mode = ROWS_GATHER_TOKENS;
    g.max_tiles = p.max_tiles;
    g.b_group_stride = (int64_t)(swiglu ? 2 : 1) * d.h * d.d;
    g.a_bytes = (uint32_t)((size_t)d.T * d.d * elem_size(d.dtype));
    g.act_n = d.h;
    g.act_ld = ldh;
    // Weight-read-bound (one 64-row M-tile per expert on average): each expert's
    // weights are read once, non-temporally, so that they do not evict the
    // gathered token rows and the activation rows, which are read again.
    g.b_nt = p.tile_bm == 64 && (int64_t)d.T * d.K <= (int64_t)64 * d.E;
    HIP_CHECK(launch_gemm(d, swiglu ? EPI_SWIGLU_STORE : EPI_GELU_STORE, p.tile_bm, g, s), "fc1 grouped gemm");
    if (events && events[1]) HIP_CHECK(hipEventRecord(static_cast<hipEvent_t>(events[1]), s), "event record");
    GemmArgs g2 = g;
    g2.A = region<void>(ws, p.act);
    g2.B = w2;
    g2.C = expert_out;
    g2.N = d.d;
    g2.Kdim = ldh;
    g2.row_mode = ROWS_IDENTITY;
    g2.b_group_stride = (int64_t)d.d * ldh;
    g2.a_bytes = (uint32_t)((size_t)d.T * d.K * ldh * elem_size(d.dtype));
    HIP_CHECK(launch_gemm(d, EPI_SCATTER_SLOT, p.tile_bm, g2, s), "fc2 grouped gemm");
    if (events) HIP_CHECK(hipEventRecord(static_cast<hipEvent_t>(events[2]), s), "event record");
    return MOE_OK;
}

// Shared expert over all T tokens in token order, fp32 output for the combine.
// With `fuse` (expert outputs, gates and y given) and a shape the fused
// epilogue supports, fc2 also performs the combine and writes y; *fused tells
// whether it did (the separate combine is then skipped).
struct CombineArgs {
    const void* expert_out;
    const float* gate;
    void* y;
};
static moe_status_t enqueue_shared_mlp(const moe_desc_t& d, const WorkspacePlan& p, void* ws, const void* x,
                                       const void* w1s, const void* w2s, float* sout, hipStream_t s,
                                       const CombineArgs* fuse = nullptr, bool* fused = nullptr) {
    if (fused) *fused = false;
    const bool swiglu = d.flags & MOE_FLAG_SWIGLU;
    const int32_t ldh = act_stride(d, d.h_shared);
    int bm = gemm_dense_bm(d.dtype, d.T, ldh < d.d ? ldh : d.d);
    if (swiglu && d.d < 128) bm = 64;  // 256-row SwiGLU tiles need two or more K slabs
    GemmArgs g{};
    g.A = x;
    g.B = w1s;
    g.C = region<void>(ws, p.sact);
    g.dense_rows = d.T;
    g.N = d.h_shared;
    g.Kdim = d.d;
    g.route_k = 1;
    g.row_mode = ROWS_IDENTITY;
    g.max_tiles = (d.T + bm - 1) / bm;
    g.a_bytes = (uint32_t)((size_t)d.T * d.d * elem_size(d.dtype));
    g.act_n = d.h_shared;
    g.act_ld = ldh;
    HIP_CHECK(launch_gemm(d, swiglu ? EPI_SWIGLU_STORE : EPI_GELU_STORE, bm, g, s), "shared fc1 gemm");
    GemmArgs g2 = g;
    g2.A = region<void>(ws, p.sact);
    g2.B = w2s;
    g2.C = sout;
    g2.N = d.d;
    g2.Kdim = ldh;
    g2.a_bytes = (uint32_t)((size_t)d.T * ldh * elem_size(d.dtype));
    if (fuse && fused && gemm_combine_fusable(d, bm, g2.N, g2.Kdim)) {
        g2.C = fuse->y;
        g2.gate = fuse->gate;
        g2.eo = fuse->expert_out;
        g2.lambda = d.lambda;
        g2.route_k = d.K;
        HIP_CHECK(launch_gemm(d, EPI_COMBINE, bm, g2, s), "shared fc2 gemm with the combine");
        *fused = true;
        return MOE_OK;
    }
    HIP_CHECK(launch_gemm(d, EPI_STORE_F32, bm, g2, s), "shared fc2 gemm");
    return MOE_OK;
}

// Backward of the routed experts (bf16). fc1 again keeps the fp32
// pre-activations P (SwiGLU: gate G and up U, stacked); dH is (Gout W2) times
// GELU'(P) (SwiGLU: dG and dU from G and U), formed in that product's epilogue
// with Gout the output gradients gathered by slot; the slot gradients of x are
// dH W1 (fp32, slot order) summed per token; the weight gradients are
// K-windowed products of slab-major transposed operands.
static moe_status_t enqueue_backward(const moe_desc_t& d, const BackwardPlan& b, void* ws, const void* x,
                                     const int32_t* sorted_slots, const int32_t* offsets, const void* w1,
                                     const void* w2, const void* gout, void* dx, float* dw1, float* dw2,
                                     hipStream_t s) {
    const WorkspacePlan& p = b.fwd;
    const bool sw = d.flags & MOE_FLAG_SWIGLU;
    const size_t TK = (size_t)d.T * d.K;
    const int hh = b.hh, hw = b.hw;
    TileDesc* tiles = region<TileDesc>(ws, p.tiles);
    int32_t* ntiles = region<int32_t>(ws, p.ntiles);
    void* act = region<void>(ws, p.act);
    float* pre = region<float>(ws, b.pre);
    void* w1t = region<void>(ws, b.w1t);
    void* w2t = region<void>(ws, b.w2t);
    void* dh = region<void>(ws, b.dh);
    float* dxs = region<float>(ws, b.dxs);
    int32_t* koff = region<int32_t>(ws, b.koff);
    HIP_CHECK(launch_build_tiles(d.E, p.tile_bm, p.max_tiles, offsets, tiles, ntiles, s), "build_tiles");
    // Weight-gradient windows first: on the persistent kernel the recompute
    // and dA products write the transposed activation and dH into them.
    void* gt = region<void>(ws, b.gt);
    void* at = region<void>(ws, b.at);
    void* dht = region<void>(ws, b.dht);
    void* xt = region<void>(ws, b.xt);
    TileDesc* items = region<TileDesc>(ws, b.items);
    TileDesc* rlist = region<TileDesc>(ws, b.rlist);
    int32_t* wcount = region<int32_t>(ws, b.wcount);
    float* partials = region<float>(ws, b.partials);
    HIP_CHECK(launch_wgrad_plan(offsets, d.E, koff, items, rlist, wcount, s), "weight-gradient plan");
    const bool direct_t = gemm_backward_transposed(d, p.tile_bm);
    if (sw) HIP_CHECK(launch_transpose_w13(w1, d.E, d.h, hh, d.d, w1t, s), "transpose w13");
    else HIP_CHECK(launch_transpose_w(w1, d.E, d.h, d.d, w1t, s), "transpose w1");
    HIP_CHECK(launch_transpose_w(w2, d.E, d.d, hh, w2t, s), "transpose w2");

    GemmArgs g{};  // fc1 again: the activation (bf16) and the pre-activations (fp32)
    g.A = x;
    g.B = w1;
    g.C = act;
    g.C2 = pre;
    g.row_map = sorted_slots;
    g.tiles = tiles;
    g.n_tiles = ntiles;
    g.N = d.h;
    g.Kdim = d.d;
    g.route_k = d.K;
    g.row_mode = ROWS_GATHER_TOKENS;
    g.max_tiles = p.max_tiles;
    g.b_group_stride = (int64_t)(sw ? 2 : 1) * d.h * d.d;
    g.a_bytes = (uint32_t)((size_t)d.T * d.d * 2);
    g.act_n = d.h;
    g.act_ld = hh;
    if (direct_t) {
        g.CT = at;
        g.ct_cols = hh;
        g.koff = koff;
        g.goff = offsets;
    }
    HIP_CHECK(launch_gemm(d, sw ? EPI_SWIGLU_BWD : EPI_GELU_BWD, p.tile_bm, g, s), "backward fc1");

    GemmArgs ga = g;  // dH from Gout W2 and the pre-activations
    ga.A = gout;
    ga.B = w2t;
    ga.C = dh;
    ga.C2 = nullptr;
    ga.aux = pre;
    ga.N = hh;
    ga.b_group_stride = (int64_t)hh * d.d;
    ga.row_mode = ROWS_GATHER_SLOTS;
    ga.a_bytes = (uint32_t)(TK * d.d * 2);
    // SwiGLU dA keeps its row output only: its epilogue already carries the
    // fp32 gate and up reads, and a second, transposed output costs more
    // there than the separate gather of dH.
    const bool direct_dh = direct_t && !sw;
    ga.CT = direct_dh ? dht : nullptr;
    ga.ct_cols = hw;
    HIP_CHECK(launch_gemm(d, sw ? EPI_DSWIGLU : EPI_DGELU, p.tile_bm, ga, s), "backward dA");

    GemmArgs gx = g;  // slot gradients of x: dH W1, fp32 to slot order
    gx.A = dh;
    gx.B = w1t;
    gx.C = dxs;
    gx.C2 = nullptr;
    gx.N = d.d;
    gx.Kdim = hw;
    gx.b_group_stride = (int64_t)d.d * hw;
    gx.row_mode = ROWS_IDENTITY;
    gx.a_bytes = (uint32_t)(TK * hw * 2);
    gx.CT = nullptr;
    HIP_CHECK(launch_gemm(d, EPI_SCATTER_SLOT_F32, p.tile_bm, gx, s), "backward dx");
    HIP_CHECK(launch_slot_sum(dxs, d.T, d.K, d.d, dx, s), "slot sum");

    // Weight gradients: transposed operands in per-expert K windows (the
    // activation and dH ones written above when the products ran persistent).
    HIP_CHECK(launch_transpose_window(gout, d.d, SRC_SLOT, sorted_slots, d.K, offsets, koff, d.E, gt, b.ld, s),
              "transpose G");
    if (direct_t)
        HIP_CHECK(launch_zero_empty_windows(at, hh, offsets, koff, d.E, s), "empty windows");
    else
        HIP_CHECK(launch_transpose_window(act, hh, SRC_SORTED, sorted_slots, d.K, offsets, koff, d.E, at, b.ld, s),
                  "transpose A");
    if (direct_dh)
        HIP_CHECK(launch_zero_empty_windows(dht, hw, offsets, koff, d.E, s), "empty windows");
    else
        HIP_CHECK(launch_transpose_window(dh, hw, SRC_SORTED, sorted_slots, d.K, offsets, koff, d.E, dht, b.ld, s),
                  "transpose dH");
    HIP_CHECK(launch_transpose_window(x, d.d, SRC_TOKEN, sorted_slots, d.K, offsets, koff, d.E, xt, b.ld, s),
              "transpose x");
    auto wgrad = [&](const void* pa, int m, const void* pb, int n, float* out, const char* what) -> moe_status_t {
        GemmArgs w{};
        w.A = pa;
        w.B = pb;
        w.C = out;
        w.dense_rows = m;
        w.N = n;
        w.Kdim = b.ld;
        w.route_k = 1;
        w.row_mode = ROWS_IDENTITY;
        w.tiles = items;
        w.n_tiles = wcount;
        w.C2 = partials;
        const int bm = m % 256 == 0 ? 256 : 64;
        w.max_tiles = b.items_max * (m / bm);
        w.a_bytes = (uint32_t)((size_t)m * b.ld * 2);
        HIP_CHECK(launch_gemm(d, EPI_WGRAD_F32, bm, w, s), what);
        HIP_CHECK(launch_wgrad_reduce(partials, rlist, wcount, d.E, (size_t)m * n, out, s), what);
        return MOE_OK;
    };
    CHECK(wgrad(gt, d.d, at, hh, dw2, "dW2"));
    if (b.dw1p) {  // SwiGLU with padded halves: compute padded, then drop the padding rows
        float* dw1p = region<float>(ws, b.dw1p);
        CHECK(wgrad(dht, hw, xt, d.d, dw1p, "dW13"));
        HIP_CHECK(launch_compact_rows(dw1p, d.E, d.h, hh, d.d, dw1, s), "dW13 rows");
    } else {
        CHECK(wgrad(dht, hw, xt, d.d, dw1, "dW1"));
    }
    return MOE_OK;
}

}  // namespace moe

using namespace moe;

MOE_API const char* moe_status_string(moe_status_t st) {
    switch (st) {
        case MOE_OK: return "MOE_OK";
        case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
        case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
        case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
        case MOE_ERR_HIP: return "MOE_ERR_HIP";
    }
    return "MOE_ERR_UNKNOWN";
}

MOE_API const char* moe_last_error(void) { return g_err; }

MOE_API moe_status_t moe_workspace_size(const moe_desc_t* desc, size_t* bytes) {
    CHECK(check_desc(desc));
    if (!bytes) return fail(MOE_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = plan_workspace(*desc).total;
    return ok();
}

MOE_API moe_status_t moe_route(const moe_desc_t* desc, const void* x, const void* w_router, const float* bias,
                               int32_t* topk_idx, float* topk_gate, void* workspace, size_t workspace_bytes,
                               void* stream) {
    CHECK(check_desc(desc));
    CHECK(check_ptr(x, "x"));
    CHECK(check_ptr(w_router, "w_router"));
    CHECK(check_ptr(bias, "bias", true));
    CHECK(check_ptr(topk_idx, "topk_idx"));
    CHECK(check_ptr(topk_gate, "topk_gate"));
    WorkspacePlan p;
    CHECK(check_ws(*desc, workspace, workspace_bytes, &p));
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    CHECK(enqueue_route(*desc, p, workspace, x, w_router, bias, topk_idx, topk_gate, s));
    return ok();
}

MOE_API moe_status_t moe_permute(const moe_desc_t* desc, const int32_t* topk_idx, int32_t* counts,
                                 int32_t* offsets, int32_t* sorted_slots, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    CHECK(check_desc(desc));
    CHECK(check_ptr(topk_idx, "topk_idx"));
    CHECK(check_ptr(counts, "counts"));
    CHECK(check_ptr(offsets, "offsets"));
    CHECK(check_ptr(sorted_slots, "sorted_slots"));
    WorkspacePlan p;
    CHECK(check_ws(*desc, workspace, workspace_bytes, &p));
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    HIP_CHECK(launch_permute(*desc, topk_idx, counts, offsets, sorted_slots, region<int32_t>(workspace, p.blockhist),
                             p.n_hist_blocks, s),
              "permute");
    return ok();
}

MOE_API moe_status_t moe_grouped_mlp(const moe_desc_t* desc, const void* x, const int32_t* sorted_slots,
                                     const int32_t* offsets, const void* w1, const void* w2, void* expert_out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
    CHECK(check_desc(desc));
    CHECK(check_ptr(x, "x"));
    CHECK(check_ptr(sorted_slots, "sorted_slots"));
    CHECK(check_ptr(offsets, "offsets"));
    CHECK(check_ptr(w1, "w1"));
    CHECK(check_ptr(w2, "w2"));
    CHECK(check_ptr(expert_out, "expert_out"));
    WorkspacePlan p;
    CHECK(check_ws(*desc, workspace, workspace_bytes, &p));
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    CHECK(enqueue_routed_mlp(*desc, p, workspace, x, sorted_slots, offsets, w1, w2, expert_out, s));
    return ok();
}

MOE_API moe_status_t moe_combine(const moe_desc_t* desc, const void* expert_out, const float* topk_gate,
                                 const void* shared_out, void* y, void* stream) {
    CHECK(check_desc(desc));
    CHECK(check_ptr(expert_out, "expert_out"));
    CHECK(check_ptr(topk_gate, "topk_gate"));
    CHECK(check_ptr(shared_out, "shared_out", true));
    CHECK(check_ptr(y, "y"));
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    HIP_CHECK(launch_combine(*desc, expert_out, topk_gate, shared_out, desc->dtype == MOE_F32, y, s), "combine");
    return ok();
}

MOE_API moe_status_t moe_layer_forward(const moe_desc_t* desc, const void* x, const void* w_router,
                                       const float* bias, const void* w1, const void* w2, const void* w1s,
                                       const void* w2s, void* y, int32_t* topk_idx_out, float* topk_gate_out,
                                       void* workspace, size_t workspace_bytes, void* const* events,
                                       void* stream) {
    CHECK(check_desc(desc));
    const moe_desc_t& d = *desc;
    CHECK(check_ptr(x, "x"));
    CHECK(check_ptr(w_router, "w_router"));
    CHECK(check_ptr(bias, "bias", true));
    CHECK(check_ptr(w1, "w1"));
    CHECK(check_ptr(w2, "w2"));
    if (d.h_shared > 0) {
        CHECK(check_ptr(w1s, "w1s"));
        CHECK(check_ptr(w2s, "w2s"));
    }
    CHECK(check_ptr(y, "y"));
    CHECK(check_ptr(topk_idx_out, "topk_idx_out", true));
    CHECK(check_ptr(topk_gate_out, "topk_gate_out", true));
    if (events && (!events[0] || !events[2]))
        return fail(MOE_ERR_INVALID_ARG, "events must hold three event slots, the first and the last non-NULL");
    WorkspacePlan p;
    CHECK(check_ws(d, workspace, workspace_bytes, &p));
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();

    int32_t* idx = topk_idx_out ? topk_idx_out : region<int32_t>(workspace, p.idx);
    float* gate = topk_gate_out ? topk_gate_out : region<float>(workspace, p.gate);
    int32_t* counts = region<int32_t>(workspace, p.counts);
    int32_t* offsets = region<int32_t>(workspace, p.offsets);
    int32_t* slots = region<int32_t>(workspace, p.slots);
    void* eout = region<void>(workspace, p.eout);
    float* sout = d.h_shared ? region<float>(workspace, p.sout) : nullptr;

    CHECK(enqueue_route(d, p, workspace, x, w_router, bias, idx, gate, s));
    // The permute's scan also builds the routed experts' tile table.
    HIP_CHECK(launch_permute(d, idx, counts, offsets, slots, region<int32_t>(workspace, p.blockhist),
                             p.n_hist_blocks, s, p.tile_bm, p.max_tiles, region<TileDesc>(workspace, p.tiles),
                             region<int32_t>(workspace, p.ntiles)),
              "permute");
    CHECK(enqueue_routed_mlp(d, p, workspace, x, slots, offsets, w1, w2, eout, s, events, true));
    bool fused = false;
    if (d.h_shared) {
        const CombineArgs c{eout, gate, y};
        CHECK(enqueue_shared_mlp(d, p, workspace, x, w1s, w2s, sout, s, &c, &fused));
    }
    if (!fused) HIP_CHECK(launch_combine(d, eout, gate, sout, 1, y, s), "combine");
    return ok();
}

MOE_API moe_status_t moe_backward_workspace_size(const moe_desc_t* desc, size_t* bytes) {
    CHECK(check_backward_desc(desc));
    if (!bytes) return fail(MOE_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = plan_backward(*desc).total;
    return ok();
}

MOE_API moe_status_t moe_grouped_mlp_backward(const moe_desc_t* desc, const void* x, const int32_t* sorted_slots,
                                              const int32_t* offsets, const void* w1, const void* w2,
                                              const void* grad_expert_out, void* dx, float* dw1, float* dw2,
                                              void* workspace, size_t workspace_bytes, void* stream) {
    CHECK(check_backward_desc(desc));
    CHECK(check_ptr(x, "x"));
    CHECK(check_ptr(sorted_slots, "sorted_slots"));
    CHECK(check_ptr(offsets, "offsets"));
    CHECK(check_ptr(w1, "w1"));
    CHECK(check_ptr(w2, "w2"));
    CHECK(check_ptr(grad_expert_out, "grad_expert_out"));
    CHECK(check_ptr(dx, "dx"));
    CHECK(check_ptr(dw1, "dw1"));
    CHECK(check_ptr(dw2, "dw2"));
    const BackwardPlan b = plan_backward(*desc);
    if (!workspace) return fail(MOE_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", b.total);
    if (reinterpret_cast<uintptr_t>(workspace) & 255u)
        return fail(MOE_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
    if (workspace_bytes < b.total)
        return fail(MOE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, b.total);
    (void)hipGetLastError();
    CHECK(enqueue_backward(*desc, b, workspace, x, sorted_slots, offsets, w1, w2, grad_expert_out, dx, dw1, dw2,
                           static_cast<hipStream_t>(stream)));
    return ok();
}

MOE_API moe_status_t moe_bias_update(const moe_desc_t* desc, const int32_t* counts, float* bias, float alpha,
                                     int32_t rule, void* stream) {
    CHECK(check_desc(desc));
    CHECK(check_ptr(counts, "counts"));
    CHECK(check_ptr(bias, "bias"));
    if (!(alpha >= 0.0f) || !(alpha <= 3.402823466e38f))
        return fail(MOE_ERR_INVALID_ARG, "alpha must be finite and >= 0");
    if (rule != MOE_BIAS_SIGN && rule != MOE_BIAS_ZSCORE)
        return fail(MOE_ERR_INVALID_ARG, "rule must be MOE_BIAS_SIGN or MOE_BIAS_ZSCORE");
    (void)hipGetLastError();
    HIP_CHECK(launch_bias_update(desc->E, counts, bias, alpha, rule, static_cast<hipStream_t>(stream)),
              "bias update");
    return ok();
}
