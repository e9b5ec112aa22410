// Internal declarations shared by the HIP translation units of the MoE-layer
// library: element types, the workspace plan, tile tables and the kernel
// launchers. Nothing here is part of the public C ABI (include/moe_vie.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "moe_vie.h"

namespace moe {

// bf16 is carried as raw 16-bit patterns in memory.
typedef uint16_t bf16_t;

constexpr int kWave = 64;          // CDNA wavefront width
// MI355X: 8 accelerator complex dies, 32 CUs each, workgroups dispatched
// round-robin over them. A performance assumption only: the XCD-aware tile
// orders built on it are bijections over the grid, so which tiles run, and
// every result, is the same on a part with another XCD count or dispatch.
constexpr int kNumXcd = 8;
constexpr int kMaxE = 1024;
constexpr int kMaxCombineK = 8;  // routed slots per token the fused combine epilogues take
constexpr int kMaxK = 16;

// One M-tile of a grouped GEMM: `rows` rows (<= BM) of expert `e`, starting
// at sorted position `row0` (rows of one expert are contiguous).
struct TileDesc {
    int32_t e;
    int32_t row0;
    int32_t rows;
    int32_t pad;
};

// How the GEMM kernels find the A rows and where the output rows go.
enum GemmRowMode : int {
    ROWS_GATHER_TOKENS = 0,  // A row of sorted position p is x[sorted_slots[p] / K]
    ROWS_IDENTITY = 1,       // A row of position p is row p
    ROWS_GATHER_SLOTS = 2,   // A row of sorted position p is row sorted_slots[p] (slot order)
};

enum GemmEpilogue : int {
    EPI_GELU_STORE = 0,     // C[p, :] = act(GELU(acc)) at the sorted position p
    EPI_SCATTER_SLOT = 1,   // C[sorted_slots[p], :] = acc  (expert_out in slot order)
    EPI_STORE_F32 = 2,      // C[p, :] = acc as fp32 (shared expert output)
    EPI_COMBINE = 3,        // C[p, :] = y_p = out(sum_j gate[p, j] eo[p K + j, :] + lambda acc): the
                            // gate-weighted combine fused into the shared expert's fc2 (dense only)
    EPI_SWIGLU_STORE = 4,   // C[p, c] = act(SiLU(G[p, c]) * U[p, c]) for c < act_n, 0 for act_n <= c <
                            // act_ld (C's row stride): B holds per group the act_n gate rows, then
                            // the act_n up rows. The launcher sets N: a tile of BN columns computes
                            // BN / 2 activation columns from the matching gate and up rows
    // Backward of GELU experts (tiled kernel only):
    EPI_GELU_BWD = 5,       // C[p, :] = bf16(GELU(acc)) and C2[p, :] = acc (fp32), sorted order
    EPI_DGELU = 6,          // C[p, :] = bf16(acc * GELU'(aux[p, :])) (aux fp32 [rows, N]), sorted order
    EPI_SCATTER_SLOT_F32 = 7,  // C[sorted_slots[p], :] = acc as fp32
    EPI_WGRAD_F32 = 8,      // weight gradients (fp32): A [dense_rows, Kdim] and B [N, Kdim], stored
                            // slab-major ([Kdim / 64][rows][64]), are shared by all experts; work item
                            // i = tiles[i] = {e, k0, klen, dest} sums K columns
                            // k0 .. k0 + klen (multiples of 64) of rows m into C[e][m, :] (dest < 0) or into
                            // the partial block C2[dest] [dense_rows, N]; *n_tiles items
    // Backward of SwiGLU experts (tiled kernel only):
    EPI_SWIGLU_BWD = 9,     // EPI_SWIGLU_STORE, and the fp32 gate and up pre-activations into C2
                            // [rows, 2 act_ld]: G at column c, U at column act_ld + c
    EPI_DSWIGLU = 10,       // dA = acc (N = act_ld columns); with G, U from aux [rows, 2 act_ld] (fp32):
                            // C[p, c] = bf16(dA U SiLU'(G)), C[p, act_ld + c] = bf16(dA SiLU(G)) for
                            // c < act_n, 0 for act_n <= c < act_ld
    // Router logits (dense, persistent kernel only):
    EPI_ROUTER_F32 = 11,    // EPI_STORE_F32, and C2[p] = sum over k of A[p, k]^2 (fp32, any order): the
                            // token norms of the router's interval test, formed from the fragments the
                            // K loop already holds
};

struct GemmArgs {
    const void* A;             // rows of length Kdim (layer dtype)
    const void* B;             // weights [groups][N][Kdim] (layer dtype)
    void* C;                   // output rows of length N
    const int32_t* row_map;    // sorted_slots (gather / scatter), may be null for identity
    const TileDesc* tiles;     // grouped mode: tile table
    const int32_t* n_tiles;    // grouped mode: device-side tile count
    int32_t dense_rows;        // dense mode (tiles == null): M rows in one group
    int32_t N;
    int32_t Kdim;
    int32_t route_k;           // K of the routing (slot -> token = slot / route_k)
    int32_t row_mode;          // GemmRowMode
    int32_t max_tiles;         // upper bound on the number of M-tiles (grid sizing)
    int64_t b_group_stride;    // elements between consecutive experts' weights
    int32_t b_rows;            // dense bf16 only: rows of B that exist (0 = N); rows past them read as zeros
    uint32_t a_bytes;          // bytes of the A operand buffer (bounds of its buffer resource)
    void* C2;                  // EPI_GELU_BWD: second output (fp32); EPI_WGRAD_F32: partial blocks;
                               // EPI_ROUTER_F32: the rows' sums of squares [dense_rows] (fp32);
                               // tiled dense EPI_STORE_F32: the sums of squares of B's rows over each K
                               // part, [k_splits][N] (fp32), or null
    // Backward, persistent kernel: the bf16 output (the activation, or dH) also
    // written transposed into the weight-gradient K windows, slab-major
    // [windows / 64][ct_cols][64]: sorted position p of expert e goes to window
    // position koff[e] + p - goff[e]; padding positions of the window get 0.
    // EPI_GELU_BWD / EPI_SWIGLU_BWD then skip the row-major activation.
    void* CT;
    int32_t ct_cols;
    const int32_t* koff;       // [E + 1] window starts
    const int32_t* goff;       // [E + 1] group offsets (sorted positions)
    const void* aux;           // EPI_DGELU: the pre-activation (fp32, rows of N); EPI_DSWIGLU: G, U
    int32_t ldc;               // persistent kernel, EPI_WGRAD_F32 / EPI_DSWIGLU: the real column count when N
                               // is rounded up to the tile width (0 = N); columns past it are not stored
    int32_t act_n;             // EPI_SWIGLU_STORE: activation width h (valid columns)
    int32_t act_ld;            // EPI_SWIGLU_STORE: activation row stride (h rounded up to 128)
    const float* gate;         // EPI_COMBINE: gates [rows, route_k]
    const void* eo;            // EPI_COMBINE: expert outputs [rows * route_k, N] in slot order
    float lambda;              // EPI_COMBINE: shared-expert weight
    int32_t k_splits;          // tiled kernel, dense EPI_STORE_F32 only: K split into this many parts (0 or
                               // 1 = none), part p writing its partial sums to C + p * dense_rows * N
    int32_t b_nt;              // tiled kernel: B is read once by the launch (one M-tile per group on
                               // average), so its copies carry the non-temporal hint
};

// Offsets (bytes) of every workspace region for one descriptor.
struct WorkspacePlan {
    size_t idx, gate, scores, counts, offsets, slots, blockhist, tiles, ntiles;
    size_t wnorm, ovf, cand, ncand, wr32, xnorm2, wsq;
    int32_t router_splits;   // split-K parts of the fast router's logits GEMM
    size_t act, eout, sact, sout;
    size_t total;
    int32_t n_hist_blocks;   // blocks of the permute histogram / scatter
    int32_t tile_bm;         // M-tile height of the routed grouped GEMM
    int32_t max_tiles;       // upper bound on routed M-tiles
};

size_t elem_size(int32_t dtype);
// Records the message of a failing call (read back by moe_last_error) and
// returns `st`.
moe_status_t set_last_error(moe_status_t st, const char* fmt, ...);
WorkspacePlan plan_workspace(const moe_desc_t& d);

// Workspace of the expert-MLP backward: the forward plan (tile table,
// activation), then the backward's own regions.
struct BackwardPlan {
    WorkspacePlan fwd;
    // hh = activation row stride (h, or ldh for SwiGLU); hw = pre-activation
    // width (hh, or 2 ldh for SwiGLU: gate columns then up columns).
    size_t pre;              // pre-activations [T*K, hw] fp32, sorted order
    size_t w1t, w2t;         // transposed weights [E, d, hw] and [E, hh, d]
    size_t dh;               // pre-activation gradient [T*K, hw] bf16, sorted order
    size_t dxs;              // slot gradients of x [T*K, d] fp32, slot order
    size_t koff;             // [E + 1] K-window starts
    size_t gt, at, dht, xt;  // transposed operands [d | hh | hw, ld] bf16
    size_t items, rlist;     // weight-gradient work items and split experts (TileDesc each)
    size_t wcount;           // [4] int32: item count, split-expert count
    size_t partials;         // [items_max, d, hw] fp32 partial sums of split experts
    size_t dw1p;             // SwiGLU with h < ldh: padded [E, hw, d] fp32 first-layer gradient, else 0
    int32_t hh, hw;
    int32_t ld;              // row length of the transposed operands: T*K + 128 E, rounded up to 64
    int32_t items_max;       // bound on the work items (and on the partial blocks)
    size_t total;
};
BackwardPlan plan_backward(const moe_desc_t& d);
// M-tile height of the grouped GEMM for groups of `avg_rows` rows on average.
int gemm_tile_bm(int32_t dtype, int64_t avg_rows);
// Row stride of an expert activation of hidden width h: h itself for GELU
// experts, h rounded up to a multiple of 64 for SwiGLU experts (the padding
// columns hold zeros, and the second layer's weights have the same stride).
inline int32_t act_stride(const moe_desc_t& d, int32_t h) {
    return (d.flags & MOE_FLAG_SWIGLU) ? (h + 63) / 64 * 64 : h;
}
// M-tile height of a dense GEMM of `rows` rows and `n` output columns.
int gemm_dense_bm(int32_t dtype, int64_t rows, int32_t n);

// ---- launchers (each returns the first HIP error, hipSuccess otherwise)
hipError_t launch_router_scores(const moe_desc_t& d, const void* x, const void* w_router,
                                float* scores, hipStream_t s);
hipError_t launch_topk(const moe_desc_t& d, const float* scores, const float* bias,
                       int32_t* topk_idx, float* topk_gate, hipStream_t s);
// Fast-router tail: norms, candidate repair with exact recomputation, and the
// exact fallback for tokens with too many candidates. s_fast = MFMA logits,
// rows of ld >= E floats.
// cand [T][router_cand_slots(K)] and ncand [T] are scratch of the candidate
// pass.
// The logits come in nsplit partial arrays of T x ld (split K), summed in
// order. Small batches (router_small_batch) read the weights as fp32 from
// wr32 [E, d], which the norm kernel writes; larger ones ignore it. xnorm2
// [T]: the tokens' sums of squares if the logits GEMM formed them
// (EPI_ROUTER_F32), else nullptr and the candidate kernel reads x for them.
// wsq [nsplit][ld]: the weight rows' sums of squares over each K part (the
// logits GEMM's second output), given exactly when router_small_fused holds;
// the whole repair then runs in one launch and wnorm, wr32, cand, ncand and
// the overflow queue are not touched.
hipError_t launch_router_fast_finish(const moe_desc_t& d, const float* s_fast, int ld, int nsplit, const void* x,
                                     const float* xnorm2, const void* w_router, const float* bias, float* wnorm,
                                     float* wr32, const float* wsq,
                                     uint16_t* cand, int32_t* ncand, int32_t* ovf_count, int32_t* ovf_list,
                                     int32_t* topk_idx, float* topk_gate, hipStream_t s);
// Whether the fast router takes the small-batch chain kernel (fp32 weight copy).
bool router_small_batch(const moe_desc_t& d);
// Whether the small-batch repair runs as one launch (K <= 8, E <= 256,
// d <= 4096): the logits GEMM then also forms the weight rows' sums of squares.
bool router_small_fused(const moe_desc_t& d);
int router_cand_slots(int K);
// Grouping of slots by expert; with a tile table (tiles != nullptr) the scan
// kernel also cuts the segments into M-tiles of bm rows (as launch_build_tiles).
hipError_t launch_permute(const moe_desc_t& d, const int32_t* topk_idx, int32_t* counts,
                          int32_t* offsets, int32_t* sorted_slots, int32_t* blockhist,
                          int32_t n_blocks, hipStream_t s, int32_t bm = 0, int32_t max_tiles = 0,
                          TileDesc* tiles = nullptr, int32_t* n_tiles = nullptr);
hipError_t launch_build_tiles(int32_t E, int32_t bm, int32_t max_tiles, const int32_t* offsets,
                              TileDesc* tiles, int32_t* n_tiles, hipStream_t s);
hipError_t launch_gemm(const moe_desc_t& d, int epilogue, int bm, const GemmArgs& a, hipStream_t s);
// Whether launch_gemm(EPI_COMBINE) supports this dense GEMM (M-tile bm, N columns, K = kdim).
bool gemm_combine_fusable(const moe_desc_t& d, int bm, int n, int kdim);
// Whether the backward's first-layer recompute and dA products run on the
// persistent kernel (which can also write their transposed outputs).
bool gemm_backward_transposed(const moe_desc_t& d, int bm);
// Backward data movement (backward.hip). Row sources of the transposing
// gather: rows already in sorted order, slot rows, token rows.
enum TransposeSource : int { SRC_SORTED = 0, SRC_SLOT = 1, SRC_TOKEN = 2 };
hipError_t launch_transpose_w(const void* in, int G, int R, int C, void* out, hipStream_t s);
// Stacked gate/up weights [G][2h][C] -> [G][C][2 ld], rows padded to ld each.
hipError_t launch_transpose_w13(const void* in, int G, int h, int ld, int C, void* out, hipStream_t s);
// [G][2 ld][C] fp32 with padded gate/up halves -> [G][2h][C].
hipError_t launch_compact_rows(const float* in, int G, int h, int ld, int C, float* out, hipStream_t s);
// Longest K window of one weight-gradient work item, in 64-column slabs.
constexpr int kWgradSlabs = 128;
hipError_t launch_wgrad_plan(const int32_t* offsets, int E, int32_t* koff, TileDesc* items, TileDesc* rlist,
                             int32_t* wcount, hipStream_t s);
hipError_t launch_wgrad_reduce(const float* partials, const TileDesc* rlist, const int32_t* wcount, int E,
                               size_t mn, float* out, hipStream_t s);
hipError_t launch_transpose_window(const void* in, int C, int mode, const int32_t* row_map, int K,
                                   const int32_t* offsets, const int32_t* koff, int E, void* out, int ld,
                                   hipStream_t s);
hipError_t launch_slot_sum(const float* dxs, int T, int K, int d, void* dx, hipStream_t s);
// Zeroes the windows of experts with no rows in a slab-major operand [ld / 64][C][64].
hipError_t launch_zero_empty_windows(void* out, int C, const int32_t* offsets, const int32_t* koff, int E,
                                     hipStream_t s);
hipError_t launch_bias_update(int32_t E, const int32_t* counts, float* bias, float alpha, int32_t rule,
                              hipStream_t s);
hipError_t launch_combine(const moe_desc_t& d, const void* expert_out, const float* gate,
                          const void* shared, int shared_is_f32, void* y, hipStream_t s);

}  // namespace moe
