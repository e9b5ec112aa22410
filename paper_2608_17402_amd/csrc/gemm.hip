// Grouped expert GEMMs (paper App. "MoE Kernel", Algorithm 1 Phases 2-3,
// with fc1 -> GELU -> fc2 experts; Sec. 3.3 "Optimized Kernel": all experts
// in one launch, activation fused into the GEMM epilogue).
//
// One launch covers every expert: a device-side tile list (TileDesc, built
// from the expert offsets) gives each M-tile's expert and rows, so the host
// never learns the per-expert loads. The grid is an upper bound; tiles past
// the device-side count exit at once.
//
// Block-to-tile order is XCD aware: MI355X dispatches consecutive workgroups
// round-robin over its 8 XCDs, each with its own L2, so workgroup b is mapped
// to logical tile (b % 8) * ceil(total / 8) + b / 8. Each XCD then walks a
// contiguous run of tiles, and the N-tiles of one M-tile (which share the
// gathered A rows) and the M-tiles of one expert (which share its weights)
// meet in the same L2.
//
// bf16: v_mfma_f32_32x32x16_bf16 with fp32 accumulators. Both operands are
// K-contiguous (token rows and nn.Linear weight rows) and stream global -> LDS
// in 64-wide K slabs through rings of a few slabs (buffer_load ... lds), with
// 16-byte chunks XOR-swizzled by row so that the rows a fragment read touches
// spread over the LDS banks. The kernels:
//   k_gemm_bf16  tiled, one tile per workgroup (256- or 64-row tiles, 64- to
//                256-column tiles); every epilogue, including the backward's
//   k_gemm_sp    256 x 256 tiles, four waves of 128 x 128, copies paced by
//                hand against the MFMAs (used where K is one slab)
//   k_gemm_pp    the persistent form of k_gemm_sp: one workgroup per CU walks
//                its tiles with the slab pipeline running across them; the
//                large-batch forward and backward products
//   k_gemm_f32   fp32 layers (VALU)
// Epilogues (EPI_*): GELU or SwiGLU to bf16 (first layer), scatter to slot
// order (second layer), fp32 store, the gate-weighted combine, and the
// backward's recompute (with fp32 pre-activations), dA through GELU' or
// SwiGLU', fp32 slot gradients and fp32 weight gradients.
#include "gemm_device.h"
#include "moe_internal.h"

#include <math.h>

#include <type_traits>
#include <utility>

namespace moe {
namespace {

__device__ __forceinline__ float gelu_erf(float v) {
    return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

struct TileCoord {
    int e, row0, rows, n0;
    bool valid;
};

// Logical tile of workgroup `b`: XCD-aware order, N-tiles of one M-tile adjacent.
// GROUPED: M-tiles come from the device-side tile table; otherwise one dense
// group of a.dense_rows rows.
template <bool GROUPED>
__device__ __forceinline__ TileCoord locate_tile(const GemmArgs& a, int bm, int bn) {
    TileCoord tc;
    tc.valid = false;
    const int n_n = a.N / bn;
    const int total_m = GROUPED ? *a.n_tiles : (a.dense_rows + bm - 1) / bm;
    const int total = total_m * n_n;
    const int per = (total + kNumXcd - 1) / kNumXcd;
    const int b = blockIdx.x;
    const int j = b / kNumXcd;
    if (j >= per) return tc;
    const int lid = (b % kNumXcd) * per + j;
    if (lid >= total) return tc;
    const int mt = lid / n_n;
    tc.n0 = (lid - mt * n_n) * bn;
    if (GROUPED) {
        const TileDesc t = a.tiles[mt];
        tc.e = t.e;
        tc.row0 = t.row0;
        tc.rows = t.rows;
    } else {
        tc.e = 0;
        tc.row0 = mt * bm;
        tc.rows = min(bm, a.dense_rows - tc.row0);
    }
    tc.valid = true;
    return tc;
}

// Gradients of SiLU(g) * u from the gradient da of the product: (dg, du) =
// (da u SiLU'(g), da SiLU(g)), SiLU'(g) = s (1 + g (1 - s)), s = Sigmoid(g).
__device__ __forceinline__ void swiglu_grad(float g, float u, float da, float& dg, float& du) {
    const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g * -1.44269504f));
    dg = da * u * (sg * fmaf(g, 1.0f - sg, 1.0f));
    du = da * (g * sg);
}

// SwiGLU activation of one column: SiLU(gate) * up, or 0 past the valid width.
__device__ __forceinline__ float swiglu_col(float g, float u, bool valid) {
    return valid ? silu_as(g) * u : 0.0f;
}

// Tile of workgroup `b` in the weight-gradient product: work items x (M / bm)
// row tiles x (N / bn) column tiles, in the same XCD-aware order as
// locate_tile (the tiles of one item are adjacent). M = a.dense_rows. tc.e is
// the work item here.
__device__ __forceinline__ TileCoord locate_wgrad_tile(const GemmArgs& a, int bm, int bn) {
    TileCoord tc;
    tc.valid = false;
    const int n_n = a.N / bn;
    const int m_per = a.dense_rows / bm;
    const int total = *a.n_tiles * m_per * n_n;
    const int per = (total + kNumXcd - 1) / kNumXcd;
    const int b = blockIdx.x;
    const int j = b / kNumXcd;
    if (j >= per) return tc;
    const int lid = (b % kNumXcd) * per + j;
    if (lid >= total) return tc;
    const int mt = lid / n_n;
    tc.n0 = (lid - mt * n_n) * bn;
    tc.e = mt / m_per;
    tc.row0 = (mt - tc.e * m_per) * bm;
    tc.rows = bm;
    tc.valid = true;
    return tc;
}

// Weight rows a tile may read: the group's rows (B rows past b_rows, when
// set, read as zeros through the buffer-resource bound).
__device__ __forceinline__ int weight_rows(const GemmArgs& a) { return a.b_rows > 0 ? a.b_rows : a.N; }

// Epilogues of a first expert layer: their token rows are gathered from x.
__host__ __device__ constexpr bool fc1_epi(int epi) {
    return epi == EPI_GELU_STORE || epi == EPI_SWIGLU_STORE || epi == EPI_SWIGLU_BWD;
}
// Epilogues of the persistent kernel that can also write their bf16 result
// transposed into the weight-gradient windows (GemmArgs::CT).
__host__ __device__ constexpr bool ct_epi(int epi) {
    return epi == EPI_GELU_BWD || epi == EPI_SWIGLU_BWD || epi == EPI_DGELU;
}

// Derivative of gelu_sig, so that the backward differentiates the function
// the forward evaluated: with sg = Sigmoid(s), e = exp(-s), 1 - sg = e sg and
// d/dx [x sg] = sg (1 + x e sg s'(x)), s'(x) = a0 + 3 a1 x^2 + 5 a2 x^4 (past
// the clamp e sg is below 1e-11 and the term vanishes). Its largest absolute
// difference from Phi(x) + x phi(x) is 1.1e-4.
__device__ __forceinline__ float gelu_sig_grad(float x) {
    const float xc = __builtin_amdgcn_fmed3f(x, -8.0f, 8.0f);
    const float x2 = xc * xc;
    const float e = __builtin_amdgcn_exp2f(xc * fmaf(fmaf(kGeluB2, x2, kGeluB1), x2, kGeluB0));
    const float sg = __builtin_amdgcn_rcpf(1.0f + e);
    const float ds = fmaf(fmaf(5.0f * kGeluA2, x2, 3.0f * kGeluA1), x2, kGeluA0);
    return sg * fmaf(x * e * sg, ds, 1.0f);
}

// bf16 grouped / dense GEMM, C[m, n] = sum_k X[m, k] W[n, k], fp32 accumulation.
//
// Tiles of BM token rows x BN output columns; WAVES_M x WAVES_N waves, each
// owning a (BM / WAVES_M) x (BN / WAVES_N) sub-tile of 32x32 MFMA blocks.
// The weight fragment is the MFMA's first operand and the token fragment the
// second, so each lane's accumulators hold ONE token row and, per block,
// four runs of four consecutive output columns: the epilogue writes 8- or
// 16-byte row-contiguous pieces with one row address per lane.
//
// K slabs of BK (32 or 64) stream global -> LDS through a ring of STAGES
// buffers with buffer_load ... lds (the K offset is a scalar, so issuing a
// copy costs no vector instructions), STAGES - 1 slabs ahead of the MFMAs. A
// wave fills whole 1 KB pieces: lane l of piece q lands in slot q*64 + l =
// (row, physical chunk) and loads logical chunk physical ^ swizzle(row); the
// swizzle puts the 16 rows read together by a quarter-wave of a fragment read
// on 16 distinct 16-byte bank groups of the 64-bank LDS. Fragments for the
// next 16-wide K step are read while the MFMAs of the current one run.
template <int BM, int BN, int WAVES_M, int WAVES_N, int BK, int STAGES, int EPI, bool GROUPED, int WPE>
__global__ __launch_bounds__(WAVES_M* WAVES_N* kWave) __attribute__((amdgpu_waves_per_eu(WPE, 8)))
void k_gemm_bf16(const GemmArgs a) {
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int NT = NW * kWave;
    constexpr int CPR = BK / 8;  // 16-byte chunks per LDS row
    constexpr int ROWB = BK * 2;
    constexpr int KS = BK / 16;  // MFMA K steps per slab
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int FM = WTM / 32;
    constexpr int FN = WTN / 32;
    static_assert(FM >= 1 && FN >= 1, "wave tile must hold at least one 32x32 block");
    constexpr int A_PIECES = BM * CPR / kWave;
    constexpr int B_PIECES = BN * CPR / kWave;
    static_assert(A_PIECES % NW == 0 && B_PIECES % NW == 0, "pieces must split evenly over waves");
    constexpr int AP = A_PIECES / NW;
    constexpr int BP = B_PIECES / NW;
    constexpr int STAGE = (BM + BN) * ROWB;
    static_assert(CPR == 4 || CPR == 8, "BK must be 32 or 64");
    static_assert(STAGES >= 2 && STAGES <= 5, "2 to 5 stages");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * STAGE];
    __shared__ int32_t srow[BM];
    constexpr bool WGRAD = EPI == EPI_WGRAD_F32;
    // A rows gathered through the row map (first layers, the backward's dA).
    constexpr bool A_GATHER = fc1_epi(EPI) || EPI == EPI_GELU_BWD || EPI == EPI_DGELU || EPI == EPI_DSWIGLU;
    // Output rows scattered to slot order (second layer, the backward's dx).
    constexpr bool O_SCATTER = EPI == EPI_SCATTER_SLOT || EPI == EPI_SCATTER_SLOT_F32;
    const TileCoord tc = WGRAD ? locate_wgrad_tile(a, BM, BN) : locate_tile<GROUPED>(a, BM, BN);
    if (!tc.valid) return;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // Row ids: gathered operand rows, or output slots.
    for (int r = tid; r < BM; r += NT) {
        const int rr = r < tc.rows ? r : tc.rows - 1;  // pad rows repeat the last valid row
        const int p = tc.row0 + rr;
        int v = p;
        if (A_GATHER && a.row_mode == ROWS_GATHER_TOKENS) v = a.row_map[p] / a.route_k;
        if (A_GATHER && a.row_mode == ROWS_GATHER_SLOTS) v = a.row_map[p];
        if (O_SCATTER) v = a.row_map[p];
        srow[r] = v;
    }
    __syncthreads();

    constexpr bool SWIGLU = EPI == EPI_SWIGLU_STORE || EPI == EPI_SWIGLU_BWD;
    constexpr bool DSW = EPI == EPI_DSWIGLU;  // two bf16 outputs per element (dG, dU)
    constexpr int HW = WTN / 2;  // SwiGLU: activation columns per wave
    static_assert(!SWIGLU || FN % 2 == 0, "SwiGLU waves hold gate and up blocks in pairs");
    const int Kd = a.Kdim;
    const __amdgpu_buffer_rsrc_t xres = make_rsrc(a.A, a.a_bytes);
    // SwiGLU: the group's 2 act_n weight rows; reads past them return zeros.
    const __amdgpu_buffer_rsrc_t wres =
        make_rsrc(static_cast<const bf16_t*>(a.B) + (WGRAD ? 0 : (size_t)tc.e * a.b_group_stride),
                  (uint32_t)(SWIGLU ? 2 * a.act_n : weight_rows(a)) * Kd * 2);

    constexpr int SWZ_SHIFT = CPR == 8 ? 1 : 2;
    constexpr int SWZ_MASK = CPR - 1;
    // Operand row stride. The weight-gradient operands are slab-major
    // ([K / 64][rows][64]): a row's 64-column piece is 128 bytes after the
    // previous row's, and a K slab is rows * 128 bytes.
    static_assert(!WGRAD || BK == 64, "slab-major operands have 64-column slabs");
    const uint32_t rstride = WGRAD ? 128u : (uint32_t)(Kd * 2);

    uint32_t xv[AP];
#pragma unroll
    for (int i = 0; i < AP; ++i) {
        const int sl = (wave + NW * i) * kWave + lane;
        const int r = sl / CPR, pch = sl % CPR;
        const int c = pch ^ ((r >> SWZ_SHIFT) & SWZ_MASK);
        int xrow;
        if (A_GATHER) xrow = srow[r];
        else xrow = tc.row0 + (r < tc.rows ? r : tc.rows - 1);
        xv[i] = (uint32_t)xrow * rstride + c * 16;
    }
    uint32_t wv[BP];
#pragma unroll
    for (int i = 0; i < BP; ++i) {
        const int sl = (wave + NW * i) * kWave + lane;
        const int r = sl / CPR, pch = sl % CPR;
        const int c = pch ^ ((r >> SWZ_SHIFT) & SWZ_MASK);
        // SwiGLU: tile column r is wave block r / WTN; its first HW columns
        // are the gate rows and the last HW the up rows of the same HW
        // activation columns. Gate rows past act_n read (finite) up rows,
        // whose activations the epilogue zeroes.
        int wrow = tc.n0 + r;
        if (SWIGLU) {
            const int w = r % WTN;
            wrow = tc.n0 / 2 + (r / WTN) * HW + w % HW + (w >= HW ? a.act_n : 0);
        }
        wv[i] = (uint32_t)wrow * rstride + c * 16;
    }

    f32x16_t acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.0f;

    // Per-lane fragment offsets: row fr of a 32-row block, chunk (ks*2 + fk)
    // swizzled; the swizzle depends only on fr because blocks start at
    // multiples of 32 rows.
    const int fr = lane & 31;
    const int fk = lane >> 5;
    const int lane_sw = (fr >> SWZ_SHIFT) & SWZ_MASK;
    uint32_t xoff[KS], woff[KS];
    const uint32_t base = lds_address(smem);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const uint32_t k = fr * ROWB + (((ks * 2 + fk) ^ lane_sw) << 4);
        xoff[ks] = base + (wm * WTM) * ROWB + k;
        woff[ks] = base + BM * ROWB + (wn * WTN) * ROWB + k;
    }
    // K range: the whole row, or (weight gradients) the group's window, or
    // (split K, dense fp32 output) part blockIdx.y of gridDim.y equal parts.
    int nk = Kd / BK;
    uint32_t kbase = 0;
    TileDesc item{};
    if (WGRAD) {
        item = a.tiles[tc.e];
        nk = item.rows / BK;
        kbase = (uint32_t)item.row0 * 2;
    }
    if constexpr (!GROUPED && EPI == EPI_STORE_F32) {
        nk /= (int)gridDim.y;
        kbase = (uint32_t)blockIdx.y * (uint32_t)nk * BK * 2;
    }

    auto issue = [&](int stage, int kslab) {
        uint8_t* buf = smem + stage * STAGE;
        uint32_t soff_a = kbase + (uint32_t)kslab * BK * 2, soff_b = soff_a;
        if (WGRAD) {
            const uint32_t slab = (uint32_t)(item.row0 / 64 + kslab);
            soff_a = slab * (uint32_t)a.dense_rows * 128u;
            soff_b = slab * (uint32_t)a.N * 128u;
        }
#pragma unroll
        for (int i = 0; i < AP; ++i) copy16_to_lds(xres, xv[i], soff_a, buf + (wave + NW * i) * 1024);
#pragma unroll
        for (int i = 0; i < BP; ++i) {
            // Weights read once in this launch (a.b_nt: one M-tile per expert
            // on average) stream past the caches.
            if (a.b_nt)
                copy16_to_lds_nt(wres, wv[i], soff_b, buf + BM * ROWB + (wave + NW * i) * 1024);
            else
                copy16_to_lds(wres, wv[i], soff_b, buf + BM * ROWB + (wave + NW * i) * 1024);
        }
    };
    auto read_frags = [&](uint32_t sbase, int ks, bf16x8_t* xf, bf16x8_t* wf) {
        const uint32_t xa = xoff[ks] + sbase, wa = woff[ks] + sbase;
        if constexpr (FM >= 1) xf[0] = lds_read16<0 * 32 * ROWB>(xa);
        if constexpr (FM >= 2) xf[1] = lds_read16<1 * 32 * ROWB>(xa);
        if constexpr (FM >= 3) xf[2] = lds_read16<2 * 32 * ROWB>(xa);
        if constexpr (FM >= 4) xf[3] = lds_read16<3 * 32 * ROWB>(xa);
        if constexpr (FN >= 1) wf[0] = lds_read16<0 * 32 * ROWB>(wa);
        if constexpr (FN >= 2) wf[1] = lds_read16<1 * 32 * ROWB>(wa);
        if constexpr (FN >= 3) wf[2] = lds_read16<2 * 32 * ROWB>(wa);
        if constexpr (FN >= 4) wf[3] = lds_read16<3 * 32 * ROWB>(wa);
        static_assert(FM <= 4 && FN <= 4, "at most 4x4 blocks per wave");
    };
    auto settle = [&](bf16x8_t* xf, bf16x8_t* wf) {
        wait_lgkmcnt0();
#pragma unroll
        for (int i = 0; i < FM; ++i) tie(xf[i]);
#pragma unroll
        for (int j = 0; j < FN; ++j) tie(wf[j]);
    };

    // Router logits of small batches (dense fp32 output with C2 set): the
    // workgroups of M-tile 0 also add up the squares of the weight rows of
    // their K part (the weight fragments pass through registers anyway), for
    // the norms of the router's interval test; C2 [parts][N] gets them.
    constexpr bool WSQ = !GROUPED && EPI == EPI_STORE_F32;
    const bool wsq_on = WSQ && a.C2 && tc.row0 == 0 && wm == 0;
    float wsq[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) wsq[j] = 0.0f;

#pragma unroll
    for (int sl = 0; sl < STAGES - 1; ++sl)
        if (sl < nk) issue(sl, sl);

    int cur_stage = 0;
    for (int kt = 0; kt < nk; ++kt) {
        // Slab kt must have landed; later prefetched slabs stay in flight.
        const int ahead = min(nk - 1 - kt, STAGES - 2);
        if constexpr (STAGES >= 4) { if (ahead >= 2) { wait_vmcnt<2 * (AP + BP)>(); goto waited; } }
        if constexpr (STAGES >= 3) { if (ahead >= 1) { wait_vmcnt<AP + BP>(); goto waited; } }
        wait_vmcnt<0>();
    waited:
        barrier_no_fence();
        if (kt + STAGES - 1 < nk) {
            int st = cur_stage + STAGES - 1;
            if (st >= STAGES) st -= STAGES;
            issue(st, kt + STAGES - 1);
        }
        const uint32_t sbase = cur_stage * STAGE;
        bf16x8_t xf[2][FM], wf[2][FN];
        read_frags(sbase, 0, xf[0], wf[0]);
        settle(xf[0], wf[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int c = ks & 1;
            if (ks + 1 < KS) read_frags(sbase, ks + 1, xf[c ^ 1], wf[c ^ 1]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[c][j], xf[c][i], acc[j][i], 0, 0, 0);
            if constexpr (WSQ) {
                if (wsq_on) {
#pragma unroll
                    for (int j = 0; j < FN; ++j)
#pragma unroll
                        for (int q = 0; q < 8; ++q) {
                            const float v = (float)wf[c][j][q];
                            wsq[j] = fmaf(v, v, wsq[j]);
                        }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            if (ks + 1 < KS) settle(xf[c ^ 1], wf[c ^ 1]);
        }
        if (++cur_stage == STAGES) cur_stage = 0;
    }
    if constexpr (WSQ) {
        if (wsq_on) {  // lanes l and l + 32 hold the two K halves of weight row l % 32
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const float v = wsq[j] + __shfl_xor(wsq[j], 32);
                const int col = tc.n0 + wn * WTN + j * 32 + fr;
                if (fk == 0 && col < a.N) static_cast<float*>(a.C2)[(size_t)blockIdx.y * a.N + col] = v;
            }
        }
    }

    // Epilogue, one 32-row block of the wave tile at a time. Block (j, i):
    // this lane's token row is i*32 + (lane & 31); accumulator 4g + q is column
    // j*32 + 8g + 4*(lane >> 5) + q. The block is activated / converted and
    // written to the wave's own LDS area row by row (rows padded by 16 bytes
    // so the 32 rows of one write spread over the banks), then read back as
    // 16-byte row pieces so that consecutive lanes store whole 128-byte lines.
    // The fused combine (dense, K <= 8) stages the shared expert's fp32 output.
    constexpr bool COMB = EPI == EPI_COMBINE;
    static_assert(!(COMB && GROUPED), "the fused combine is a dense (shared expert) epilogue");
    constexpr bool OUT_F32 = EPI == EPI_STORE_F32 || EPI == EPI_SCATTER_SLOT_F32 || WGRAD || COMB;
    constexpr int OES = OUT_F32 ? 4 : 2;           // staged element size
    constexpr int SEG = (SWIGLU ? HW : WTN) * OES * (DSW ? 2 : 1);  // bytes of one wave-tile row
    constexpr int RSTR = SEG + 16;                 // padded LDS row stride
    constexpr int CPRO = SEG / 16;                 // 16-byte pieces per row
    constexpr int PIECES = 32 * CPRO / kWave;      // pieces per lane per block
    static_assert(NW * 32 * RSTR <= STAGES * STAGE, "epilogue staging must fit in the stage buffers");
    static_assert((32 * CPRO) % kWave == 0, "row pieces must split evenly over the wave");
    __syncthreads();  // every wave is done with the stage buffers
    uint8_t* stg = smem + wave * 32 * RSTR;
    // First output column of this wave's rows (SwiGLU: activation column,
    // rows act_ld apart).
    const int ocol0 = SWIGLU ? tc.n0 / 2 + wn * HW : tc.n0 + wn * WTN;
    const size_t ostride = SWIGLU ? (size_t)a.act_ld : (DSW ? 2 * (size_t)a.act_ld : (size_t)a.N);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        if constexpr (DSW) {
            // dG in the first half of the staging row, dU in the second.
            const int r = wm * WTM + i * 32 + fr;
            const float* grow = static_cast<const float*>(a.aux) +
                                (size_t)(tc.row0 + (r < tc.rows ? r : tc.rows - 1)) * 2 * a.act_ld + ocol0;
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = j * 32 + 8 * g + 4 * fk;
                    const float4 gv = *reinterpret_cast<const float4*>(grow + c);
                    const float4 uv = *reinterpret_cast<const float4*>(grow + a.act_ld + c);
                    const float gg[4] = {gv.x, gv.y, gv.z, gv.w}, uu[4] = {uv.x, uv.y, uv.z, uv.w};
                    float dg[4], du[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        swiglu_grad(gg[q], uu[q], acc[j][i][4 * g + q], dg[q], du[q]);
                        if (ocol0 + c + q >= a.act_n) dg[q] = du[q] = 0.0f;
                    }
                    *reinterpret_cast<uint2*>(stg + fr * RSTR + c * 2) = pack4_bf16(dg[0], dg[1], dg[2], dg[3]);
                    *reinterpret_cast<uint2*>(stg + fr * RSTR + (WTN + c) * 2) =
                        pack4_bf16(du[0], du[1], du[2], du[3]);
                }
        } else if constexpr (SWIGLU) {
#pragma unroll
            for (int j = 0; j < FN / 2; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = j * 32 + 8 * g + 4 * fk;
                    float v[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        v[q] = swiglu_col(acc[j][i][4 * g + q], acc[j + FN / 2][i][4 * g + q],
                                          ocol0 + c + q < a.act_n);
                    *reinterpret_cast<uint2*>(stg + fr * RSTR + c * 2) = pack4_bf16(v[0], v[1], v[2], v[3]);
                }
        } else {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    float v0 = acc[j][i][4 * g + 0], v1 = acc[j][i][4 * g + 1];
                    float v2 = acc[j][i][4 * g + 2], v3 = acc[j][i][4 * g + 3];
                    uint8_t* dst = stg + fr * RSTR + (j * 32 + 8 * g + 4 * fk) * OES;
                    if (OUT_F32) {
                        *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
                    } else {
                        if (EPI == EPI_GELU_STORE || EPI == EPI_GELU_BWD) {
                            v0 = gelu_sig(v0); v1 = gelu_sig(v1); v2 = gelu_sig(v2); v3 = gelu_sig(v3);
                        }
                        if (EPI == EPI_DGELU) {  // times GELU' of the stored pre-activation
                            const int r = wm * WTM + i * 32 + fr;
                            const size_t p = (size_t)(tc.row0 + (r < tc.rows ? r : tc.rows - 1));
                            const float4 f = *reinterpret_cast<const float4*>(
                                static_cast<const float*>(a.aux) + p * a.N + ocol0 + j * 32 + 8 * g + 4 * fk);
                            v0 *= gelu_sig_grad(f.x); v1 *= gelu_sig_grad(f.y);
                            v2 *= gelu_sig_grad(f.z); v3 *= gelu_sig_grad(f.w);
                        }
                        *reinterpret_cast<uint2*>(dst) = pack4_bf16(v0, v1, v2, v3);
                    }
                }
        }
        // Each wave reads back only its own area: a wave-level sync suffices.
        wave_sync_lds();
#pragma unroll
        for (int k = 0; k < PIECES; ++k) {
            const int q = lane + kWave * k;
            const int rr = q / CPRO, pc = q % CPRO;
            const int r = wm * WTM + i * 32 + rr;
            const uint4 v = *reinterpret_cast<const uint4*>(stg + rr * RSTR + pc * 16);
            if constexpr (COMB) {
                // y for the piece's four columns, in the separate combine's
                // order: acc = 0, acc = fma(g_j, O_j, acc) for j = 0..K-1 over
                // the token's expert-output rows (slot order), then
                // fma(lambda, S, acc) and one rounding to bf16. Slots past K
                // re-read slot K - 1 and are not added.
                if (r < tc.rows) {
                    const int tok = tc.row0 + r;
                    const int col = ocol0 + pc * 4;
                    const int K = a.route_k;
                    const bf16_t* eo = static_cast<const bf16_t*>(a.eo);
                    float gj[kMaxCombineK];
                    uint2 o[kMaxCombineK];
#pragma unroll
                    for (int j = 0; j < kMaxCombineK; ++j) {
                        const int jj = j < K ? j : K - 1;
                        gj[j] = a.gate[(size_t)tok * K + jj];
                        o[j] = *reinterpret_cast<const uint2*>(eo + ((size_t)tok * K + jj) * a.N + col);
                    }
                    float c4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                    for (int j = 0; j < kMaxCombineK; ++j)
                        if (j < K) {
                            c4[0] = fmaf(gj[j], __uint_as_float(o[j].x << 16), c4[0]);
                            c4[1] = fmaf(gj[j], __uint_as_float(o[j].x & 0xffff0000u), c4[1]);
                            c4[2] = fmaf(gj[j], __uint_as_float(o[j].y << 16), c4[2]);
                            c4[3] = fmaf(gj[j], __uint_as_float(o[j].y & 0xffff0000u), c4[3]);
                        }
                    const float sv[4] = {__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                                         __uint_as_float(v.w)};
                    uint32_t h[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        uint32_t u = __float_as_uint(fmaf(a.lambda, sv[q], c4[q]));
                        u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest even (finite values)
                        h[q] = u >> 16;
                    }
                    *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.C) + (size_t)tok * a.N + col) =
                        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                }
                continue;
            }
            if (r < tc.rows && (!SWIGLU || ocol0 < a.act_ld)) {
                size_t orow = O_SCATTER ? (size_t)srow[r] : (size_t)(tc.row0 + r);
                void* obase = a.C;
                if constexpr (!GROUPED && EPI == EPI_STORE_F32)  // split K: this part's partial sums
                    obase = static_cast<float*>(a.C) + (size_t)blockIdx.y * a.dense_rows * a.N;
                if (WGRAD) {  // the expert's gradient, or the item's partial block
                    orow += (size_t)(item.pad < 0 ? item.e : item.pad) * a.dense_rows;
                    if (item.pad >= 0) obase = a.C2;
                }
                size_t ocol = (size_t)ocol0;
                int pcc = pc;
                if (DSW && pc >= CPRO / 2) {  // the dU half goes act_ld columns further on
                    ocol += a.act_ld;
                    pcc -= CPRO / 2;
                }
                uint8_t* out = static_cast<uint8_t*>(obase) + (orow * ostride + ocol) * OES + pcc * 16;
                *reinterpret_cast<uint4*>(out) = v;
            }
        }
        wave_sync_lds();
    }
    if constexpr (EPI == EPI_SWIGLU_BWD) {
        // Second output: the fp32 gate and up pre-activations, G at column c and
        // U at act_ld + c of C2's rows (2 act_ld), staged as [G | U] per row.
        constexpr int SEG2 = 2 * HW * 4, RSTR2 = SEG2 + 16, CPRO2 = SEG2 / 16, PIECES2 = 32 * CPRO2 / kWave;
        static_assert(NW * 32 * RSTR2 <= STAGES * STAGE, "epilogue staging must fit in the stage buffers");
        __syncthreads();  // the wider rows overlap other waves' first-pass areas
        uint8_t* stg2 = smem + wave * 32 * RSTR2;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN / 2; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = j * 32 + 8 * g + 4 * fk;
                    *reinterpret_cast<float4*>(stg2 + fr * RSTR2 + c * 4) =
                        make_float4(acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                                    acc[j][i][4 * g + 3]);
                    const int ju = j + FN / 2;
                    *reinterpret_cast<float4*>(stg2 + fr * RSTR2 + (HW + c) * 4) =
                        make_float4(acc[ju][i][4 * g + 0], acc[ju][i][4 * g + 1], acc[ju][i][4 * g + 2],
                                    acc[ju][i][4 * g + 3]);
                }
            wave_sync_lds();
#pragma unroll
            for (int k = 0; k < PIECES2; ++k) {
                const int q = lane + kWave * k;
                const int rr = q / CPRO2, pc = q % CPRO2;
                const int r = wm * WTM + i * 32 + rr;
                const uint4 v = *reinterpret_cast<const uint4*>(stg2 + rr * RSTR2 + pc * 16);
                if (r < tc.rows && ocol0 < a.act_ld) {
                    const bool up = pc >= CPRO2 / 2;
                    const size_t col = (size_t)ocol0 + (up ? a.act_ld : 0);
                    uint8_t* out = static_cast<uint8_t*>(a.C2) +
                                   ((size_t)(tc.row0 + r) * 2 * a.act_ld + col) * 4 + (pc - (up ? CPRO2 / 2 : 0)) * 16;
                    *reinterpret_cast<uint4*>(out) = v;
                }
            }
            wave_sync_lds();
        }
    }
    if constexpr (EPI == EPI_GELU_BWD) {
        // Second output: the pre-activation (acc) in fp32 (rows of N), the same staging.
        constexpr int SEG2 = WTN * 4, RSTR2 = SEG2 + 16, CPRO2 = SEG2 / 16, PIECES2 = 32 * CPRO2 / kWave;
        static_assert(NW * 32 * RSTR2 <= STAGES * STAGE, "epilogue staging must fit in the stage buffers");
        __syncthreads();  // the wider rows overlap other waves' first-pass areas
        uint8_t* stg2 = smem + wave * 32 * RSTR2;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<float4*>(stg2 + fr * RSTR2 + (j * 32 + 8 * g + 4 * fk) * 4) =
                        make_float4(acc[j][i][4 * g + 0], acc[j][i][4 * g + 1], acc[j][i][4 * g + 2],
                                    acc[j][i][4 * g + 3]);
            wave_sync_lds();
#pragma unroll
            for (int k = 0; k < PIECES2; ++k) {
                const int q = lane + kWave * k;
                const int rr = q / CPRO2, pc = q % CPRO2;
                const int r = wm * WTM + i * 32 + rr;
                const uint4 v = *reinterpret_cast<const uint4*>(stg2 + rr * RSTR2 + pc * 16);
                if (r < tc.rows) {
                    uint8_t* out = static_cast<uint8_t*>(a.C2) + ((size_t)(tc.row0 + r) * a.N + ocol0) * 4 + pc * 16;
                    *reinterpret_cast<uint4*>(out) = v;
                }
            }
            wave_sync_lds();
        }
    }
}

// bf16 grouped / dense GEMM, 256 x 256 tiles, four waves of 128 x 128 (one
// wave per SIMD, accumulators in the 256 accumulation registers), 64-wide K
// slabs (whole 128-byte row pieces per copy).
//
// A CU's global -> LDS copy path takes about as long to move a slab as the
// MFMAs take to consume it, so copies must leave at an even pace: every K
// step of 16 MFMAs carries exactly four copies (one after every fourth MFMA)
// and eight fragment reads for the next K step, in an order fixed by hand.
// The token operand has a ring of three slabs and the weight operand a ring
// of two (together the whole 160 KB of LDS), so token copies get more than a
// slab of lead and weight copies, mostly L2 hits, half a slab. One barrier per
// slab sits before its last K step: every wave has read the whole slab by
// then (its buffers can be refilled from that last step on) and has seen its
// own copies of the next slab land (its first fragments are read during that
// last step). Row ids come from the global row map, so no LDS is spent on them.
template <int EPI, bool GROUPED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_gemm_sp(const GemmArgs a) {
    constexpr int BM = 256, BN = 256, NW = 4, WT = 128, FB = WT / 32;
    constexpr int BK = 64, CPR = 8, ROWB = 128, KS = 4;
    constexpr int SLAB = BM * ROWB;           // 32 KB per operand and slab
    constexpr int AST = 3, WST = 2;           // ring depths
    constexpr int WBASE = AST * SLAB;         // weight ring after the token ring
    constexpr int AP = BM * CPR / kWave / NW;  // 8 token copy pieces per wave and slab
    constexpr int BP = BN * CPR / kWave / NW;  // 8 weight copy pieces
    static_assert(AP == 8 && BP == 8, "copy schedule is written for 8 + 8 pieces");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[AST * SLAB + WST * SLAB];

    const TileCoord tc = locate_tile<GROUPED>(a, BM, BN);
    if (!tc.valid) return;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int wm = wave >> 1, wn = wave & 1;
    const int Kd = a.Kdim;
    const int nk = Kd / BK;

    auto row_id = [&](int r) {  // operand / output row id of tile row r (pad rows repeat the last)
        const int p = tc.row0 + (r < tc.rows ? r : tc.rows - 1);
        if (EPI == EPI_GELU_STORE && a.row_mode == ROWS_GATHER_TOKENS) return a.row_map[p] / a.route_k;
        if (EPI == EPI_SCATTER_SLOT) return a.row_map[p];
        return p;
    };

    const __amdgpu_buffer_rsrc_t xres = make_rsrc(a.A, a.a_bytes);
    const __amdgpu_buffer_rsrc_t wres =
        make_rsrc(static_cast<const bf16_t*>(a.B) + (size_t)tc.e * a.b_group_stride, (uint32_t)weight_rows(a) * Kd * 2);
    const __amdgpu_buffer_rsrc_t xnull = make_rsrc(a.A, 0);
    const __amdgpu_buffer_rsrc_t wnull =
        make_rsrc(static_cast<const bf16_t*>(a.B) + (size_t)tc.e * a.b_group_stride, 0);
    uint32_t xv[AP], wv[BP];
#pragma unroll
    for (int i = 0; i < AP; ++i) {
        const int sl = (wave + NW * i) * kWave + lane;
        const int r = sl / CPR, pch = sl % CPR;
        const int c = pch ^ ((r >> 1) & 7);
        const int xrow = EPI == EPI_GELU_STORE ? row_id(r) : tc.row0 + (r < tc.rows ? r : tc.rows - 1);
        xv[i] = (uint32_t)xrow * (uint32_t)(Kd * 2) + c * 16;
    }
#pragma unroll
    for (int i = 0; i < BP; ++i) {
        const int sl = (wave + NW * i) * kWave + lane;
        const int r = sl / CPR, pch = sl % CPR;
        const int c = pch ^ ((r >> 1) & 7);
        wv[i] = (uint32_t)(tc.n0 + r) * (uint32_t)(Kd * 2) + c * 16;
    }

    f32x16_t acc[FB][FB];
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
        for (int i = 0; i < FB; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.0f;

    const int fr = lane & 31;
    const int fk = lane >> 5;
    const int lane_sw = (fr >> 1) & 7;
    uint32_t xoff[KS], woff[KS];
    const uint32_t base = lds_address(smem);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const uint32_t k = fr * ROWB + (((ks * 2 + fk) ^ lane_sw) << 4);
        xoff[ks] = base + (wm * WT) * ROWB + k;
        woff[ks] = base + WBASE + (wn * WT) * ROWB + k;
    }

    // Slab m's copy source: real slabs through the sized resources, slabs
    // past the last through the zero-size ones at an in-range offset.
    auto slab_src = [&](int m, uint32_t& soff, __amdgpu_buffer_rsrc_t& xr, __amdgpu_buffer_rsrc_t& wr) {
        const bool real = m < nk;
        soff = (uint32_t)(real ? m : nk - 1) * BK * 2;
        xr = real ? xres : xnull;
        wr = real ? wres : wnull;
    };
    // Copy piece L (constant) of this wave: token operand (IS_A) or weights.
    auto copy_a = [&](auto LC, int stage, uint32_t soff, __amdgpu_buffer_rsrc_t xr) {
        constexpr int L = decltype(LC)::value;
        copy16_to_lds(xr, xv[L], soff, smem + stage * SLAB + (wave + NW * L) * 1024);
    };
    auto copy_w = [&](auto LC, int stage, uint32_t soff, __amdgpu_buffer_rsrc_t wr) {
        constexpr int L = decltype(LC)::value;
        copy16_to_lds(wr, wv[L], soff, smem + WBASE + stage * SLAB + (wave + NW * L) * 1024);
    };

    bf16x8_t xf[2][FB], wf[2][FB];
    auto read_frag = [&](auto NBC, auto QC, uint32_t abase, uint32_t wbase, int ks) {
        constexpr int nb = decltype(NBC)::value, q = decltype(QC)::value;
        if constexpr (q < FB) xf[nb][q] = lds_read16<q * 32 * ROWB>(xoff[ks] + abase);
        else wf[nb][q - FB] = lds_read16<(q - FB) * 32 * ROWB>(woff[ks] + wbase);
    };
    auto settle = [&](auto CBC) {
        constexpr int cb = decltype(CBC)::value;
        wait_lgkmcnt0();
#pragma unroll
        for (int i = 0; i < FB; ++i) tie(xf[cb][i]);
#pragma unroll
        for (int j = 0; j < FB; ++j) tie(wf[cb][j]);
    };
    // One K step: 16 MFMAs on buffer CB, fragment q of the next K step after
    // MFMA q (q < 8), copy number q / 4 of the step's four after MFMA q when
    // q % 4 == 1. COPY(c) issues the step's c-th copy.
    auto kstep = [&](auto CBC, uint32_t rabase, uint32_t rwbase, int rks, auto&& copy) {
        constexpr int cb = decltype(CBC)::value;
        static_for<FB * FB>([&](auto QC) {
            constexpr int q = decltype(QC)::value;
            constexpr int j = q / FB, i = q % FB;
            acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[cb][j], xf[cb][i], acc[j][i], 0, 0, 0);
            if constexpr (q < 2 * FB)
                read_frag(std::integral_constant<int, cb ^ 1>{}, QC, rabase, rwbase, rks);
            if constexpr (q % 4 == 1) copy(std::integral_constant<int, q / 4>{});
            __builtin_amdgcn_sched_barrier(0);
        });
    };

    // Prologue: token slab 0, weight slab 0, token slab 1, the first half of
    // weight slab 1 (what the loop would have issued before step 0); wait for
    // slab 0 of both operands; read its first fragments.
    {
        uint32_t so;
        __amdgpu_buffer_rsrc_t xr, wr;
        slab_src(0, so, xr, wr);
        static_for<AP>([&](auto LC) { copy_a(LC, 0, so, xr); });
        static_for<BP>([&](auto LC) { copy_w(LC, 0, so, wr); });
        slab_src(1, so, xr, wr);
        static_for<AP>([&](auto LC) { copy_a(LC, 1, so, xr); });
        static_for<BP / 2>([&](auto LC) { copy_w(LC, 1, so, wr); });
    }
    wait_vmcnt<AP + BP / 2>();
    barrier_no_fence();
    static_for<2 * FB>([&](auto QC) { read_frag(std::integral_constant<int, 0>{}, QC, 0u, 0u, 0); });

    int as = 0, ws = 0;  // ring slots of slab kt
    for (int kt = 0; kt < nk; ++kt) {
        const uint32_t abase = (uint32_t)as * SLAB, wbase = (uint32_t)ws * SLAB;
        const int as1 = as == AST - 1 ? 0 : as + 1, as2 = as1 == AST - 1 ? 0 : as1 + 1;
        const int ws1 = ws ^ 1;
        uint32_t so1, so2, so2w;
        __amdgpu_buffer_rsrc_t xr1, wr1, xr2, wr2, xr2w, wr2w;
        slab_src(kt + 1, so1, xr1, wr1);
        slab_src(kt + 2, so2, xr2, wr2);
        (void)xr1; (void)xr2w; (void)wr2;
        so2w = so2; wr2w = wr2;
        // K step 0: second half of weight slab kt + 1.
        settle(std::integral_constant<int, 0>{});
        kstep(std::integral_constant<int, 0>{}, abase, wbase, 1, [&](auto CC) {
            copy_w(std::integral_constant<int, BP / 2 + decltype(CC)::value>{}, ws1, so1, wr1);
        });
        // K steps 1 and 2: token slab kt + 2.
        settle(std::integral_constant<int, 1>{});
        kstep(std::integral_constant<int, 1>{}, abase, wbase, 2, [&](auto CC) {
            copy_a(std::integral_constant<int, decltype(CC)::value>{}, as2, so2, xr2);
        });
        settle(std::integral_constant<int, 0>{});
        kstep(std::integral_constant<int, 0>{}, abase, wbase, 3, [&](auto CC) {
            copy_a(std::integral_constant<int, 4 + decltype(CC)::value>{}, as2, so2, xr2);
        });
        settle(std::integral_constant<int, 1>{});
        // Token and weight slab kt + 1 have landed for this wave (the token
        // slab kt + 2 copies may still be in flight); after the barrier, for
        // every wave, and every wave is done reading slab kt.
        wait_vmcnt<AP>();
        barrier_no_fence();
        // K step 3: first fragments of slab kt + 1; first half of weight slab
        // kt + 2 into the weight buffer of slab kt.
        kstep(std::integral_constant<int, 1>{}, (uint32_t)as1 * SLAB, (uint32_t)ws1 * SLAB, 0, [&](auto CC) {
            copy_w(std::integral_constant<int, decltype(CC)::value>{}, ws, so2w, wr2w);
        });
        as = as1;
        ws = ws1;
    }

    // Epilogue (as in k_gemm_bf16): row ids to LDS, then per 32-row block
    // activate / convert into the wave's LDS area, read back as 16-byte row
    // pieces, store whole lines.
    constexpr bool OUT_F32 = EPI == EPI_STORE_F32;
    constexpr int OES = OUT_F32 ? 4 : 2;
    constexpr int SEG = WT * OES;
    constexpr int RSTR = SEG + 16;
    constexpr int CPRO = SEG / 16;
    constexpr int PIECES = 32 * CPRO / kWave;
    static_assert(1024 + NW * 32 * RSTR <= AST * SLAB + WST * SLAB, "epilogue staging must fit");
    __syncthreads();
    int32_t* srow = reinterpret_cast<int32_t*>(smem);
    if (EPI == EPI_SCATTER_SLOT)
        for (int r = tid; r < BM; r += NW * kWave) srow[r] = row_id(r);
    __syncthreads();
    uint8_t* stg = smem + 1024 + wave * 32 * RSTR;
#pragma unroll
    for (int i = 0; i < FB; ++i) {
#pragma unroll
        for (int j = 0; j < FB; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float v0 = acc[j][i][4 * g + 0], v1 = acc[j][i][4 * g + 1];
                float v2 = acc[j][i][4 * g + 2], v3 = acc[j][i][4 * g + 3];
                uint8_t* dst = stg + fr * RSTR + (j * 32 + 8 * g + 4 * fk) * OES;
                if (OUT_F32) {
                    *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
                } else {
                    if (EPI == EPI_GELU_STORE) {
                        v0 = gelu_sig(v0); v1 = gelu_sig(v1); v2 = gelu_sig(v2); v3 = gelu_sig(v3);
                    }
                    *reinterpret_cast<uint2*>(dst) = pack4_bf16(v0, v1, v2, v3);
                }
            }
        wave_sync_lds();
#pragma unroll
        for (int k = 0; k < PIECES; ++k) {
            const int q = lane + kWave * k;
            const int rr = q / CPRO, pc = q % CPRO;
            const int r = wm * WT + i * 32 + rr;
            const uint4 v = *reinterpret_cast<const uint4*>(stg + rr * RSTR + pc * 16);
            if (r < tc.rows) {
                const size_t orow = EPI == EPI_SCATTER_SLOT ? (size_t)srow[r] : (size_t)(tc.row0 + r);
                uint8_t* out = static_cast<uint8_t*>(a.C) + (orow * a.N + tc.n0 + wn * WT) * OES + pc * 16;
                *reinterpret_cast<uint4*>(out) = v;
            }
        }
        wave_sync_lds();
    }
}

// Persistent form of k_gemm_sp: one workgroup per CU walks its share of the
// tiles (the XCD-aware order of locate_tile, a stride of gridDim / 8 tiles
// apart), and the slab pipeline runs on across tile boundaries. While the last
// two slabs of one tile are multiplied, the first two slabs of the next are
// already being copied, so a tile costs its K loop plus its epilogue. The
// per-tile start-up of the one-tile-per-workgroup kernel disappears: dispatch,
// the tile-table and row-map reads, and the first copies' latency.
//
// The epilogue stages each wave's 32-row blocks through the token-ring slot
// of the tile's last slab. That is the only slot not being filled at that
// moment: the next tile's first slab sits in the next slot and its second is
// still landing in the one after. Row pieces are XOR-swizzled instead of
// padded so that four waves' staging fits in one 32 KB slot. Tile metadata
// flows through a short pipeline: tile-table entries are read two tiles ahead,
// and gathered token rows (fc1) and output slots (fc2) one tile ahead. Their
// loads are issued where the wait the compiler places before their first use
// falls after long independent work.
//
// Token operand without gathering: its buffer resource starts at the tile's
// first row and spans its valid rows, so pad rows read as zeros. Gathered rows
// repeat the tile's last valid row, as in k_gemm_sp. Requires K >= 128 (at
// least two slabs per tile).
template <int EPI, bool GROUPED, int KC = 8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_gemm_pp(const GemmArgs a) {
    constexpr int BM = 256, BN = 256, NW = 4, WT = 128, FB = WT / 32;
    constexpr int BK = 64, CPR = 8, ROWB = 128, KS = 4;
    constexpr int SLAB = BM * ROWB;            // 32 KB per operand and slab
    constexpr int AST = 3, WST = 2;            // ring depths
    constexpr int WBASE = AST * SLAB;          // weight ring after the token ring
    constexpr int AP = BM * CPR / kWave / NW;  // 8 token copy pieces per wave and slab
    constexpr int BP = BN * CPR / kWave / NW;  // 8 weight copy pieces
    static_assert(AP == 8 && BP == 8, "copy schedule is written for 8 + 8 pieces");
    constexpr bool BWD1 = EPI == EPI_GELU_BWD;  // bf16 GELU, then the fp32 pre-activation into C2
    constexpr bool DG = EPI == EPI_DGELU;       // bf16 of acc times GELU'(aux)
    constexpr bool DSW = EPI == EPI_DSWIGLU;    // dG and dU (bf16) from acc and the stored G, U
    constexpr bool GATHER = GROUPED && (fc1_epi(EPI) || BWD1 || DG || DSW);
    constexpr bool SWIGLU = EPI == EPI_SWIGLU_STORE || EPI == EPI_SWIGLU_BWD;
    constexpr bool SWBWD = EPI == EPI_SWIGLU_BWD;  // and the fp32 gate / up pre-activations into C2
    constexpr bool SCATTER = EPI == EPI_SCATTER_SLOT || EPI == EPI_SCATTER_SLOT_F32;
    // Weight gradients: slab-major operands, a K window per work item, fp32
    // output to the expert's gradient or a partial block.
    constexpr bool WG = EPI == EPI_WGRAD_F32;
    static_assert(!WG || GROUPED, "weight-gradient tiles come from the work-item table");
    constexpr bool RNORM = EPI == EPI_ROUTER_F32;  // EPI_STORE_F32 and the token rows' sums of squares
    constexpr bool OUT_F32 = EPI == EPI_STORE_F32 || EPI == EPI_SCATTER_SLOT_F32 || WG || RNORM;
    constexpr bool COMBINE = EPI == EPI_COMBINE;
    constexpr bool STAGE_F32 = OUT_F32 || COMBINE;  // accumulators staged as fp32
    constexpr int OES = OUT_F32 ? 4 : 2;
    constexpr int NH = (STAGE_F32 || EPI == EPI_DSWIGLU) ? 2 : 1;  // column halves per staged block
    static_assert(!(COMBINE && GROUPED), "the fused combine is a dense (shared expert) epilogue");
    constexpr int STG_WAVE = 32 * 256;         // staging bytes per wave
    static_assert(NW * STG_WAVE == SLAB, "staging must fill exactly one token slot");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[AST * SLAB + WST * SLAB];

    const int n_n = a.N / BN;
    const int m_per = WG ? a.dense_rows / BM : 1;  // row tiles per work item
    const int total =
        (GROUPED ? __builtin_amdgcn_readfirstlane(*a.n_tiles) * m_per : (a.dense_rows + BM - 1) / BM) * n_n;
    const int per = (total + kNumXcd - 1) / kNumXcd;
    const int xcd = blockIdx.x % kNumXcd;
    const int wpx = gridDim.x / kNumXcd;  // workgroups per XCD: the tile stride
    const int lid_end = min(total, (xcd + 1) * per);
    int lid = xcd * per + (int)blockIdx.x / kNumXcd;
    if (lid >= lid_end) return;
    // The combine epilogue streams K expert-output rows per output element
    // (1 MB per tile at ViT-G) and is HBM-bound when every CU runs it at once;
    // tiles cost the same, so the workgroups stay in step from the start.
    // Workgroups of odd XCDs start about 80k cycles later, so that their
    // epilogues overlap the other XCDs' K loops (whole XCDs, so that each L2
    // still sees its tiles in step). Measured at ViT-G: the layer -1.3 %.
    // "xcd" is blockIdx mod kNumXcd, which names the XCD only under the
    // round-robin dispatch of MI355X; under another dispatch a different half
    // of the workgroups waits, which changes the speed, never the tiles.
    if constexpr (EPI == EPI_COMBINE) {
        if (xcd & 1)
            for (int q = 0; q < 10; ++q) __builtin_amdgcn_s_sleep(127);
    }

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int wm = wave >> 1, wn = wave & 1;
    const int Kd = a.Kdim;
    const int nk = Kd / BK;
    const int ncols = a.ldc > 0 ? a.ldc : a.N;  // real output columns (N may be rounded up to BN)
    // Slab-major operands (weight gradients): a row's piece of one K slab is
    // 128 bytes after the previous row's.
    const uint32_t rowbytes = WG ? 128u : (uint32_t)Kd * 2;

    struct Tile {
        int e, row0, rows, n0;
        int slab0, nk, dest;  // weight gradients: first K slab, K slabs, partial block or -1
    };
    // Tile-table entry of tile l (grouped): read through the vector path (the
    // kernel's own stores keep the compiler from proving the table constant).
    // Indices past this workgroup's share read its last tile instead.
    auto tile_entry = [&](int l) {
        TileDesc d{};
        if (GROUPED) d = a.tiles[min(l, lid_end - 1) / n_n / m_per];
        return d;
    };
    // Tile l from its table entry; the entry is the same for every lane, so it
    // goes back to scalar registers.
    auto tile_of = [&](int l, const TileDesc& d) {
        Tile t;
        const int mt = l / n_n;
        t.n0 = (l - mt * n_n) * BN;
        t.slab0 = 0;
        t.nk = nk;
        t.dest = -1;
        if (WG) {
            t.e = __builtin_amdgcn_readfirstlane(d.e);
            t.row0 = (mt - (mt / m_per) * m_per) * BM;
            t.rows = BM;
            t.slab0 = __builtin_amdgcn_readfirstlane(d.row0) / BK;
            t.nk = __builtin_amdgcn_readfirstlane(d.rows) / BK;
            t.dest = __builtin_amdgcn_readfirstlane(d.pad);
        } else if (GROUPED) {
            t.e = __builtin_amdgcn_readfirstlane(d.e);
            t.row0 = __builtin_amdgcn_readfirstlane(d.row0);
            t.rows = __builtin_amdgcn_readfirstlane(d.rows);
        } else {
            t.e = 0;
            t.row0 = mt * BM;
            t.rows = min(BM, a.dense_rows - t.row0);
        }
        return t;
    };
    auto tile_at = [&](int l) { return tile_of(l, tile_entry(l)); };
    const bf16_t* const Bw = static_cast<const bf16_t*>(a.B);
    const bf16_t* const Ax = static_cast<const bf16_t*>(a.A);
    // SwiGLU: a tile of BN columns computes activation columns [n0 / 2,
    // n0 / 2 + 128); the resource starts at gate row n0 / 2 and ends with the
    // group's last up row, so rows past it read as zeros.
    // The row counts are uniform; readfirstlane keeps the resource in scalar
    // registers (the compiler cannot prove it and would wrap every copy in a
    // waterfall loop).
    auto wres_of = [&](const Tile& t) {
        if (SWIGLU)
            return make_rsrc(Bw + (size_t)t.e * a.b_group_stride + (size_t)(t.n0 / 2) * Kd,
                             (uint32_t)__builtin_amdgcn_readfirstlane(2 * a.act_n - t.n0 / 2) * rowbytes);
        // Weight gradients: every K slab of rows n0 .. (slab-major operand).
        if (WG) return make_rsrc(Bw + (size_t)t.n0 * 64, (uint32_t)ncols * (uint32_t)Kd * 2u - (uint32_t)t.n0 * 128u);
        const int rows = __builtin_amdgcn_readfirstlane(max(0, min(BN, weight_rows(a) - t.n0)));
        return make_rsrc(Bw + (size_t)t.e * a.b_group_stride + (size_t)t.n0 * Kd, (uint32_t)rows * rowbytes);
    };
    auto xres_of = [&](const Tile& t) {
        if (GATHER) return make_rsrc(Ax, a.a_bytes);
        if (WG) return make_rsrc(Ax + (size_t)t.row0 * 64, a.a_bytes - (uint32_t)t.row0 * 128u);
        return make_rsrc(Ax + (size_t)t.row0 * Kd, (uint32_t)t.rows * rowbytes);
    };
    // Source offset of K slab s of tile t: s slabs along the rows, or
    // (slab-major) slab t.slab0 + s of rows x 128 bytes.
    auto soff_a = [&](const Tile& t, int s) -> uint32_t {
        return WG ? (uint32_t)(t.slab0 + s) * (uint32_t)a.dense_rows * 128u : (uint32_t)s * (BK * 2);
    };
    auto soff_b = [&](const Tile& t, int s) -> uint32_t {
        return WG ? (uint32_t)(t.slab0 + s) * (uint32_t)ncols * 128u : (uint32_t)s * (BK * 2);
    };
    const __amdgpu_buffer_rsrc_t xnull = make_rsrc(Ax, 0);
    const __amdgpu_buffer_rsrc_t wnull = make_rsrc(Bw, 0);

    // Row offsets of this lane's copy pieces: row r of the slab, 16-byte chunk
    // c (swizzled). The weight offsets (and the token offsets without
    // gathering) are the same for every tile.
    auto piece_rc = [&](int i, int& r, int& c) {
        const int sl = (wave + NW * i) * kWave + lane;
        r = sl / CPR;
        c = (sl % CPR) ^ ((r >> 1) & 7);
    };
    // SwiGLU: wave column block wn (tile columns [128 wn, 128 wn + 128)) holds
    // the gate rows of activation columns [64 wn, 64 wn + 64) of the tile,
    // then their up rows (act_n rows further on). Gate rows past act_n read
    // (finite) up rows, whose activations the epilogue zeroes.
    // Token offsets without gathering (tv) are the plain row layout; for
    // every epilogue but SwiGLU they equal the weight offsets.
    uint32_t wv[BP], tv[AP];
#pragma unroll
    for (int i = 0; i < BP; ++i) {
        int r, c;
        piece_rc(i, r, c);
        const int wrow = SWIGLU ? (r / WT) * (WT / 2) + r % (WT / 2) + ((r % WT) >= WT / 2 ? a.act_n : 0) : r;
        wv[i] = (uint32_t)wrow * rowbytes + c * 16;
        tv[i] = (uint32_t)r * rowbytes + c * 16;
    }
    // Gathered token rows: slot -> token, rows past the tile's end repeat its last row.
    auto load_tokens = [&](const Tile& t, int32_t (&tok)[AP]) {
#pragma unroll
        for (int i = 0; i < AP; ++i) {
            int r, c;
            piece_rc(i, r, c);
            tok[i] = a.row_map[t.row0 + min(r, t.rows - 1)];
        }
    };
    // Row map entries are slots; the operand row is the slot's token (slot /
    // K) or, gathering slot rows, the slot itself.
    const int rdiv = a.row_mode == ROWS_GATHER_SLOTS ? 1 : a.route_k;
    auto token_offsets = [&](const int32_t (&tok)[AP], uint32_t (&xv)[AP]) {
#pragma unroll
        for (int i = 0; i < AP; ++i) {
            int r, c;
            piece_rc(i, r, c);
            xv[i] = (uint32_t)(tok[i] / rdiv) * rowbytes + c * 16;
        }
    };
    // Output slot of staged piece k of 32-row block i (fc2 scatter).
    int32_t orow[FB][8];
    auto load_slots = [&](const Tile& t) {
#pragma unroll
        for (int i = 0; i < FB; ++i)
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int r = wm * WT + i * 32 + (lane >> 4) + 4 * k;
                orow[i][k] = a.row_map[t.row0 + min(r, t.rows - 1)];
            }
    };

    // Current tile (c), next (n) and the one after (nn, table entry only).
    Tile tc = tile_at(lid);
    bool has_n = lid + wpx < lid_end;
    Tile tn = has_n ? tile_at(lid + wpx) : tc;
    bool has_nn = lid + 2 * wpx < lid_end;
    Tile tnn = has_nn ? tile_at(lid + 2 * wpx) : tn;
    // Table entry three tiles ahead, read one tile before it is needed.
    TileDesc ent3 = tile_entry(lid + 3 * wpx);
    __amdgpu_buffer_rsrc_t xres_c = xres_of(tc), wres_c = wres_of(tc);
    __amdgpu_buffer_rsrc_t xres_n = has_n ? xres_of(tn) : xnull;
    __amdgpu_buffer_rsrc_t wres_n = has_n ? wres_of(tn) : wnull;
    uint32_t xv_c[AP], xv_n[AP];
    int32_t tok[AP];
    if (GATHER) {
        load_tokens(tc, tok);
        token_offsets(tok, xv_c);
        load_tokens(tn, tok);
        token_offsets(tok, xv_n);
    }
    if (SCATTER) load_slots(tc);

    f32x16_t acc[FB][FB];
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
        for (int i = 0; i < FB; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.0f;

    const int fr = lane & 31;
    const int fk = lane >> 5;
    const int lane_sw = (fr >> 1) & 7;
    uint32_t xoff[KS], woff[KS];
    const uint32_t base = lds_address(smem);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const uint32_t k = fr * ROWB + (((ks * 2 + fk) ^ lane_sw) << 4);
        xoff[ks] = base + (wm * WT) * ROWB + k;
        woff[ks] = base + WBASE + (wn * WT) * ROWB + k;
    }

    auto copy_a = [&](auto LC, int stage, uint32_t soff, __amdgpu_buffer_rsrc_t xr, const uint32_t (&xv)[AP]) {
        constexpr int L = decltype(LC)::value;
        copy16_to_lds(xr, xv[L], soff, smem + stage * SLAB + (wave + NW * L) * 1024);
    };
    auto copy_w = [&](auto LC, int stage, uint32_t soff, __amdgpu_buffer_rsrc_t wr) {
        constexpr int L = decltype(LC)::value;
        copy16_to_lds(wr, wv[L], soff, smem + WBASE + stage * SLAB + (wave + NW * L) * 1024);
    };

    bf16x8_t xf[2][FB], wf[2][FB];
    auto read_frag = [&](auto NBC, auto QC, uint32_t abase, uint32_t wbase, int ks) {
        constexpr int nb = decltype(NBC)::value, q = decltype(QC)::value;
        if constexpr (q < FB) xf[nb][q] = lds_read16<q * 32 * ROWB>(xoff[ks] + abase);
        else wf[nb][q - FB] = lds_read16<(q - FB) * 32 * ROWB>(woff[ks] + wbase);
    };
    auto settle = [&](auto CBC) {
        constexpr int cb = decltype(CBC)::value;
        wait_lgkmcnt0();
#pragma unroll
        for (int i = 0; i < FB; ++i) tie(xf[cb][i]);
#pragma unroll
        for (int j = 0; j < FB; ++j) tie(wf[cb][j]);
    };
    // Router logits: per lane, the sums of squares of its four token rows'
    // values in the token fragments (lanes l and l + 32 hold the two halves
    // of each K step of row l % 32 of a 32-row block).
    float xsq[FB];
#pragma unroll
    for (int i = 0; i < FB; ++i) xsq[i] = 0.0f;

    // One K step: 16 MFMAs on buffer CB, fragment q of the next K step after
    // MFMA q (q < 8), copy q / 4 of the step's four after MFMA q when q % 4 == 1.
    // Router logits: after MFMA q, the squares of the two values in 32-bit
    // word q % 4 of token fragment q / 4 (VALU work beside the MFMAs).
    auto kstep = [&](auto CBC, uint32_t rabase, uint32_t rwbase, int rks, auto&& copy) {
        constexpr int cb = decltype(CBC)::value;
        static_for<FB * FB>([&](auto QC) {
            constexpr int q = decltype(QC)::value;
            constexpr int j = q / FB, i = q % FB;
            acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[cb][j], xf[cb][i], acc[j][i], 0, 0, 0);
            if constexpr (RNORM) {
                const uint32_t u = __builtin_bit_cast(u32x4_t, xf[cb][q / 4])[q % 4];
                const float lo = __uint_as_float(u << 16), hi = __uint_as_float(u & 0xffff0000u);
                xsq[q / 4] = fmaf(lo, lo, xsq[q / 4]);
                xsq[q / 4] = fmaf(hi, hi, xsq[q / 4]);
            }
            if constexpr (q < 2 * FB)
                read_frag(std::integral_constant<int, cb ^ 1>{}, QC, rabase, rwbase, rks);
            if constexpr (q % 4 == 1) copy(std::integral_constant<int, q / 4>{});
            __builtin_amdgcn_sched_barrier(0);
        });
    };

    // Fused combine (K = KC) for one staged fp32 block of the shared expert's
    // output S: 32 rows x 64 columns, pieces of 8 columns (lanes 8 r + c take
    // row r, column piece c; four rows per lane). Per piece, in the order of
    // the separate combine: acc = 0, acc = fma(g_j, O_j, acc) for j = 0..K-1,
    // acc = fma(lambda, S, acc), one rounding to bf16.
    auto combine_block = [&](const Tile& t, uint32_t stg, int i, int h) {
        const int cp = lane & 7;
        const bf16_t* const eo = static_cast<const bf16_t*>(a.eo);
        // y rows of this tile; stores of pad rows fall outside and are dropped,
        // so the four pieces need no branch and can be scheduled together.
        const __amdgpu_buffer_rsrc_t yres =
            make_rsrc(static_cast<uint8_t*>(a.C) + (size_t)t.row0 * a.N * 2, (uint32_t)t.rows * a.N * 2);
        u32x4_t s0[4], s1[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int rr = (lane >> 3) + 8 * k;
            s0[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)((2 * cp) ^ (rr & 15)) << 4));
            s1[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)((2 * cp + 1) ^ (rr & 15)) << 4));
        }
        // No memory clobber: the loads below may be scheduled across it.
        asm volatile("s_waitcnt lgkmcnt(0)");
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            tie(s0[k]);
            tie(s1[k]);
        }
        // Two pieces per step: both pieces' loads are issued before either is
        // used (twenty 16-byte loads in flight per lane).
#pragma unroll
        for (int kp = 0; kp < 4; kp += 2) {
            float gj[2][KC];
            u32x4_t o[2][KC];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int rr = (lane >> 3) + 8 * (kp + u);
                const int tok = t.row0 + min(wm * WT + i * 32 + rr, t.rows - 1);
                const int c0 = t.n0 + wn * WT + h * 64 + cp * 8;
                if constexpr (KC % 4 == 0) {
#pragma unroll
                    for (int j = 0; j < KC; j += 4) {
                        const float4 g4 = *reinterpret_cast<const float4*>(a.gate + (size_t)tok * KC + j);
                        gj[u][j] = g4.x; gj[u][j + 1] = g4.y; gj[u][j + 2] = g4.z; gj[u][j + 3] = g4.w;
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < KC; ++j) gj[u][j] = a.gate[(size_t)tok * KC + j];
                }
#pragma unroll
                for (int j = 0; j < KC; ++j)
                    o[u][j] = *reinterpret_cast<const u32x4_t*>(eo + ((size_t)tok * KC + j) * a.N + c0);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int k = kp + u;
                const int r = wm * WT + i * 32 + (lane >> 3) + 8 * k;
                const int c0 = t.n0 + wn * WT + h * 64 + cp * 8;
                float acc8[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) acc8[q] = 0.0f;
#pragma unroll
                for (int j = 0; j < KC; ++j) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc8[2 * q] = fmaf(gj[u][j], __uint_as_float(o[u][j][q] << 16), acc8[2 * q]);
                        acc8[2 * q + 1] = fmaf(gj[u][j], __uint_as_float(o[u][j][q] & 0xffff0000u), acc8[2 * q + 1]);
                    }
                }
                const float sv[8] = {__uint_as_float(s0[k].x), __uint_as_float(s0[k].y), __uint_as_float(s0[k].z),
                                     __uint_as_float(s0[k].w), __uint_as_float(s1[k].x), __uint_as_float(s1[k].y),
                                     __uint_as_float(s1[k].z), __uint_as_float(s1[k].w)};
                u32x4_t out;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t lo = __float_as_uint(fmaf(a.lambda, sv[2 * q], acc8[2 * q]));
                    uint32_t hi = __float_as_uint(fmaf(a.lambda, sv[2 * q + 1], acc8[2 * q + 1]));
                    lo += 0x7fffu + ((lo >> 16) & 1u);  // round to nearest even (finite values)
                    hi += 0x7fffu + ((hi >> 16) & 1u);
                    out[q] = (lo >> 16) | (hi & 0xffff0000u);
                }
                // y is written only here and read by nothing in this kernel, so
                // the store needs no memory clobber.
                const uint32_t yoff = ((uint32_t)r * (uint32_t)a.N + (uint32_t)c0) * 2u;
                asm volatile("buffer_store_dwordx4 %0, %1, %2, 0 offen nt\n\ts_nop 0" ::"v"(out), "v"(yoff), "s"(yres));
            }
        }
    };

    // Epilogue of tile t from the accumulators, staged through the token slot
    // `stslot`: per 32-row block (and 64-column half for fp32 output) each
    // lane writes its row's runs into the wave's 8 KB, then reads back 16-byte
    // row pieces (16 lanes per 256-byte row) and stores whole lines.
    // Backward: the staged bf16 block i (32 rows of this wave, ncc columns of
    // the 256-byte staging rows) also goes to the weight-gradient K windows,
    // transposed and slab-major: staged column cc becomes row colmap(cc) (or
    // nothing for -1); rows past the tile's valid rows are written as 0 up to
    // the window's end, rows past the window are not written. Window starts
    // are multiples of 64 and tiles start 256 rows apart inside an expert, so
    // each 8-row piece lies inside one 64-position slab.
    constexpr bool HAS_CT = ct_epi(EPI);
    auto store_ct = [&](const Tile& t, uint32_t stg, int i, int ncc, auto&& colmap) {
        const int e = t.e;
        const int gpos = t.row0 - a.goff[e] + wm * WT + i * 32;  // first row of the block within its expert
        const int wq = a.koff[e] + gpos;
        const int wlen = a.koff[e + 1] - a.koff[e];
        const int vrows = t.rows - (wm * WT + i * 32);  // rows of the block that exist
        uint8_t* const ct = static_cast<uint8_t*>(a.CT);
        // Piece k of a lane: staged column cc = 16 k + lane % 16, rows 8 g ..
        // 8 g + 7 with g = lane / 16, as two transposing 8-byte reads, the even
        // rows 8 g, 8 g + 2, .. and the odd rows 8 g + 1, 8 g + 3, ..: in each
        // read the 16 lanes of a quarter-wave name 4 rows x 16 columns (lane r:
        // row r / 4 of the four, columns 4 (r % 4) ..) and each receives its
        // column's 4 rows, which are then interleaved into the row order the
        // window stores. Rows two apart keep the 16-byte pieces a quarter-wave
        // reads in distinct banks under the staging swizzle. Two pieces in
        // flight: the reads of piece k + 1 are issued before piece k is stored.
        const int nit = ncc / 16;
        // The lane index through an opaque copy: the per-piece addresses are
        // then computed here instead of being hoisted out of the tile loop.
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int g = ln >> 4, c16 = ln & 15;
        u32x2_t w[2][2];
        auto issue = [&](int k, u32x2_t(&dst)[2]) {
            const int col = 16 * k + 4 * (c16 & 3);
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int row = 8 * g + hh + 2 * (c16 >> 2);
                lds_read_tr8_asm(dst[hh], stg + (uint32_t)row * 256u +
                                              ((uint32_t)((col >> 3) ^ (row & 15)) << 4) + (uint32_t)(col & 7) * 2u);
            }
        };
        issue(0, w[0]);
#pragma unroll
        for (int k = 0; k < nit; ++k) {
            __builtin_amdgcn_sched_barrier(0);
            if (k + 1 < nit) {
                issue(k + 1, w[(k + 1) & 1]);
                wait_lgkmcnt<2>();
            } else {
                wait_lgkmcnt0();
            }
            tie(w[k & 1][0]);
            tie(w[k & 1][1]);
            const int orow = colmap(16 * k + c16);
            if (orow < 0 || gpos + g * 8 >= wlen) continue;
            const u32x2_t ev = w[k & 1][0], od = w[k & 1][1];  // rows 0, 2, 4, 6 and 1, 3, 5, 7 of the piece
            u32x4_t v = {(ev.x & 0xffffu) | (od.x << 16), (ev.x >> 16) | (od.x & 0xffff0000u),
                         (ev.y & 0xffffu) | (od.y << 16), (ev.y >> 16) | (od.y & 0xffff0000u)};
            if (vrows < 32) {  // the expert's last rows: zeros past them
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (g * 8 + 2 * u >= vrows) v[u] &= 0xffff0000u;
                    if (g * 8 + 2 * u + 1 >= vrows) v[u] &= 0x0000ffffu;
                }
            }
            const int q = wq + g * 8;
            store16_asm(ct + (((size_t)(q / 64) * a.ct_cols + orow) * 64 + q % 64) * 2, v);
        }
    };

    auto epilogue = [&](const Tile& t, int stslot) {
        const uint32_t stg = base + (uint32_t)stslot * SLAB + (uint32_t)wave * STG_WAVE;
        const uint32_t wrow = stg + (uint32_t)fr * 256u;
        const int sw = fr & 15;
        uint8_t* const cbase = static_cast<uint8_t*>(a.C);
        // DSW: row stride 2 act_ld, columns past act_ld (N rounded up) not stored.
        const size_t ostr = DSW ? 2 * (size_t)a.act_ld : (size_t)ncols;
        // DSW: stage half h of block i (64 columns) as [dG | dU] per 256-byte
        // row, G and U read once.
        auto dsw_stage = [&](const Tile& tt, int i, int h) {
            const int r = wm * WT + i * 32 + fr;
            const float* grow = static_cast<const float*>(a.aux) +
                                (size_t)(tt.row0 + min(r, tt.rows - 1)) * 2 * a.act_ld;
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int j = 2 * h + jj;
                __builtin_amdgcn_sched_barrier(0);
                float4 gv[4], uv[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = tt.n0 + wn * WT + j * 32 + 8 * g + 4 * fk;
                    gv[g] = make_float4(0.f, 0.f, 0.f, 0.f);
                    uv[g] = gv[g];
                    if (c < a.act_ld) {  // act_ld is a multiple of 64: whole float4s
                        gv[g] = *reinterpret_cast<const float4*>(grow + c);
                        uv[g] = *reinterpret_cast<const float4*>(grow + a.act_ld + c);
                    }
                }
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = tt.n0 + wn * WT + j * 32 + 8 * g + 4 * fk;
                    const float gg[4] = {gv[g].x, gv[g].y, gv[g].z, gv[g].w};
                    const float uu[4] = {uv[g].x, uv[g].y, uv[g].z, uv[g].w};
                    float dg[4], du[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        swiglu_grad(gg[q], uu[q], acc_read(acc[j][i][4 * g + q]), dg[q], du[q]);
                        if (c + q >= a.act_n) dg[q] = du[q] = 0.0f;
                    }
                    const uint2 pg = pack4_bf16(dg[0], dg[1], dg[2], dg[3]);
                    const uint2 pu = pack4_bf16(du[0], du[1], du[2], du[3]);
                    const int chunk = 4 * jj + g;  // 16-byte chunk of the half's 64 columns
                    lds_write8_asm(wrow + ((uint32_t)(chunk ^ sw) << 4) + (uint32_t)fk * 8u, (u32x2_t){pg.x, pg.y});
                    lds_write8_asm(wrow + ((uint32_t)((8 + chunk) ^ sw) << 4) + (uint32_t)fk * 8u,
                                   (u32x2_t){pu.x, pu.y});
                }
            }
        };
#pragma unroll
        for (int i = 0; i < FB; ++i) {
#pragma unroll
            for (int h = 0; h < NH; ++h) {
                __builtin_amdgcn_sched_barrier(0);
                if (STAGE_F32) {
#pragma unroll
                    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int j = 2 * h + jj;
                            const u32x4_t v = {__float_as_uint(acc_read(acc[j][i][4 * g + 0])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 1])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 2])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 3]))};
                            const int chunk = 8 * jj + 2 * g + fk;
                            lds_write16_asm(wrow + ((uint32_t)(chunk ^ sw) << 4), v);
                        }
                } else if (SWIGLU) {
                    // Blocks j < 2 are gate columns, j + 2 the up columns of
                    // the same activation columns: 64 per wave row.
#pragma unroll
                    for (int j = 0; j < FB / 2; ++j)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int c = t.n0 / 2 + wn * (WT / 2) + j * 32 + 8 * g + 4 * fk;
                            float v[4];
#pragma unroll
                            for (int q = 0; q < 4; ++q)
                                v[q] = swiglu_col(acc_read(acc[j][i][4 * g + q]),
                                                  acc_read(acc[j + FB / 2][i][4 * g + q]), c + q < a.act_n);
                            const uint2 pk = pack4_bf16(v[0], v[1], v[2], v[3]);
                            lds_write8_asm(wrow + ((uint32_t)((4 * j + g) ^ sw) << 4) + (uint32_t)fk * 8u,
                                           (u32x2_t){pk.x, pk.y});
                        }
                } else if (DSW) {
                    dsw_stage(t, i, h);
                } else {
                    // dH: GELU' of the stored pre-activation of this lane's row and columns.
                    float4 fac[FB][4];
                    if constexpr (DG) {
                        const int r = wm * WT + i * 32 + fr;
                        const float* arow = static_cast<const float*>(a.aux) +
                                            (size_t)(t.row0 + min(r, t.rows - 1)) * a.N + t.n0 + wn * WT + 4 * fk;
#pragma unroll
                        for (int j = 0; j < FB; ++j)
#pragma unroll
                            for (int g = 0; g < 4; ++g)
                                fac[j][g] = *reinterpret_cast<const float4*>(arow + j * 32 + 8 * g);
                    }
#pragma unroll
                    for (int j = 0; j < FB; ++j)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            float v0 = acc_read(acc[j][i][4 * g + 0]), v1 = acc_read(acc[j][i][4 * g + 1]);
                            float v2 = acc_read(acc[j][i][4 * g + 2]), v3 = acc_read(acc[j][i][4 * g + 3]);
                            if (EPI == EPI_GELU_STORE || BWD1) {
                                v0 = gelu_sig(v0); v1 = gelu_sig(v1); v2 = gelu_sig(v2); v3 = gelu_sig(v3);
                            }
                            if constexpr (DG) {
                                v0 *= gelu_sig_grad(fac[j][g].x); v1 *= gelu_sig_grad(fac[j][g].y);
                                v2 *= gelu_sig_grad(fac[j][g].z); v3 *= gelu_sig_grad(fac[j][g].w);
                            }
                            const int chunk = 4 * j + g;
                            const uint2 pk = pack4_bf16(v0, v1, v2, v3);
                            lds_write8_asm(wrow + ((uint32_t)(chunk ^ sw) << 4) + (uint32_t)fk * 8u,
                                           (u32x2_t){pk.x, pk.y});
                        }
                }
                if constexpr (COMBINE) {
                    combine_block(t, stg, i, h);
                    continue;
                }
                if constexpr (SWBWD) {
                    if (a.CT) {  // the activation only feeds dW2: its transpose alone
                        const int ocol = t.n0 / 2 + wn * (WT / 2);
                        store_ct(t, stg, i, WT / 2, [&](int cc) { return ocol < a.act_ld ? ocol + cc : -1; });
                        continue;
                    }
                }
                if constexpr (SWIGLU) {
                    // 128-byte activation rows: 8 lanes per row, 8 rows per read.
                    const int ocol = t.n0 / 2 + wn * (WT / 2);
                    u32x4_t v[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int rr = (lane >> 3) + 8 * k;
                        v[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)((lane & 7) ^ (rr & 15)) << 4));
                    }
                    wait_lgkmcnt0();
#pragma unroll
                    for (int k = 0; k < 4; ++k) tie(v[k]);
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int r = wm * WT + i * 32 + (lane >> 3) + 8 * k;
                        if (r < t.rows && ocol < a.act_ld)
                            store16_asm(cbase + ((size_t)(t.row0 + r) * a.act_ld + ocol) * 2 + (lane & 7) * 16, v[k]);
                    }
                    continue;
                }
                if constexpr (HAS_CT && !SWIGLU) {
                    if (a.CT) {
                        const int c0 = t.n0 + wn * WT + h * 64;
                        store_ct(t, stg, i, WT, [&](int cc) { return c0 + cc; });
                        if constexpr (BWD1) continue;  // the activation only feeds dW2
                    }
                }
                u32x4_t v[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int rr = (lane >> 4) + 4 * k;
                    const int pc = lane & 15;
                    v[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)(pc ^ (rr & 15)) << 4));
                }
                wait_lgkmcnt0();
#pragma unroll
                for (int k = 0; k < 8; ++k) tie(v[k]);
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int rr = (lane >> 4) + 4 * k;
                    const int r = wm * WT + i * 32 + rr;
                    // DSW: pieces 0..7 of the row are dG, 8..15 dU (act_ld further on).
                    const int pcol = DSW ? (lane & 7) * 8 : (lane & 15) * (16 / OES);
                    const int col = t.n0 + wn * WT + h * 64 + pcol;
                    if (r < t.rows && t.n0 + wn * WT + h * 64 < ncols && (!DSW || col < a.act_ld)) {
                        size_t orw = SCATTER ? (size_t)orow[i][k] : (size_t)(t.row0 + r);
                        uint8_t* ob = cbase;
                        if (WG) {  // the expert's gradient, or the work item's partial block
                            orw += (size_t)(t.dest < 0 ? t.e : t.dest) * a.dense_rows;
                            if (t.dest >= 0) ob = static_cast<uint8_t*>(a.C2);
                        }
                        uint8_t* out = ob + (orw * ostr + t.n0 + wn * WT + h * 64) * OES + (lane & 15) * 16;
                        if (DSW) out = ob + (orw * ostr + ((lane & 8) ? a.act_ld : 0) + col) * 2;
                        store16_asm(out, v[k]);
                    }
                }
            }
            if constexpr (SWBWD) {
                // Second output: the gate (q = 0) and up (q = 1) pre-activations
                // of this wave's 64 activation columns as fp32 rows of C2
                // [rows, 2 act_ld]: G at column c, U at act_ld + c.
                const int ocol = t.n0 / 2 + wn * (WT / 2);
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int j = 2 * q + jj;
                            const u32x4_t v = {__float_as_uint(acc_read(acc[j][i][4 * g + 0])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 1])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 2])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 3]))};
                            const int chunk = 8 * jj + 2 * g + fk;
                            lds_write16_asm(wrow + ((uint32_t)(chunk ^ sw) << 4), v);
                        }
                    u32x4_t v[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int rr = (lane >> 4) + 4 * k;
                        v[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)((lane & 15) ^ (rr & 15)) << 4));
                    }
                    wait_lgkmcnt0();
#pragma unroll
                    for (int k = 0; k < 8; ++k) tie(v[k]);
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int r = wm * WT + i * 32 + (lane >> 4) + 4 * k;
                        if (r < t.rows && ocol < a.act_ld)
                            store16_asm(static_cast<uint8_t*>(a.C2) +
                                            ((size_t)(t.row0 + r) * 2 * a.act_ld + q * a.act_ld + ocol) * 4 +
                                            (lane & 15) * 16,
                                        v[k]);
                    }
                }
            }
            if constexpr (BWD1) {
                // Second output: the pre-activation (acc) as fp32 rows of C2,
                // two 64-column halves through the same staging rows.
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int j = 2 * h + jj;
                            const u32x4_t v = {__float_as_uint(acc_read(acc[j][i][4 * g + 0])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 1])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 2])),
                                               __float_as_uint(acc_read(acc[j][i][4 * g + 3]))};
                            const int chunk = 8 * jj + 2 * g + fk;
                            lds_write16_asm(wrow + ((uint32_t)(chunk ^ sw) << 4), v);
                        }
                    u32x4_t v[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int rr = (lane >> 4) + 4 * k;
                        v[k] = lds_read16u_asm(stg + (uint32_t)rr * 256u + ((uint32_t)((lane & 15) ^ (rr & 15)) << 4));
                    }
                    wait_lgkmcnt0();
#pragma unroll
                    for (int k = 0; k < 8; ++k) tie(v[k]);
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int r = wm * WT + i * 32 + (lane >> 4) + 4 * k;
                        if (r < t.rows)
                            store16_asm(static_cast<uint8_t*>(a.C2) +
                                            ((size_t)(t.row0 + r) * a.N + t.n0 + wn * WT + h * 64) * 4 + (lane & 15) * 16,
                                        v[k]);
                    }
                }
            }
        }
    };

    // Prologue: token slab 0, weight slab 0, token slab 1, the first half of
    // weight slab 1; wait for slab 0 of both operands; read its first fragments.
    static_for<AP>([&](auto LC) { copy_a(LC, 0, soff_a(tc, 0), xres_c, GATHER ? xv_c : tv); });
    static_for<BP>([&](auto LC) { copy_w(LC, 0, soff_b(tc, 0), wres_c); });
    static_for<AP>([&](auto LC) { copy_a(LC, 1, soff_a(tc, 1), xres_c, GATHER ? xv_c : tv); });
    static_for<BP / 2>([&](auto LC) { copy_w(LC, 1, soff_b(tc, 1), wres_c); });
    wait_vmcnt<AP + BP / 2>();
    barrier_no_fence();
    static_for<2 * FB>([&](auto QC) { read_frag(std::integral_constant<int, 0>{}, QC, 0u, 0u, 0); });

    int as = 0, ws = 0;  // ring slots of the slab being multiplied
    for (;;) {
        int kt = 0;
        do {  // nk >= 2 slabs: written as do-while so the compiler counts the copies
            const uint32_t abase = (uint32_t)as * SLAB, wbase = (uint32_t)ws * SLAB;
            const int as1 = as == AST - 1 ? 0 : as + 1, as2 = as1 == AST - 1 ? 0 : as1 + 1;
            const int ws1 = ws ^ 1;
            // Slabs kt + 1 and kt + 2 may belong to the next tile.
            const int nkc = tc.nk;
            const bool n1 = kt + 1 >= nkc, n2 = kt + 2 >= nkc;
            const uint32_t so1 = soff_b(n1 ? tn : tc, n1 ? kt + 1 - nkc : kt + 1);
            const uint32_t so2 = soff_a(n2 ? tn : tc, n2 ? kt + 2 - nkc : kt + 2);
            const uint32_t so2w = soff_b(n2 ? tn : tc, n2 ? kt + 2 - nkc : kt + 2);
            const __amdgpu_buffer_rsrc_t wr1 = n1 ? wres_n : wres_c;
            const __amdgpu_buffer_rsrc_t xr2 = n2 ? xres_n : xres_c;
            const __amdgpu_buffer_rsrc_t wr2 = n2 ? wres_n : wres_c;
            uint32_t xv2[AP];
#pragma unroll
            for (int i = 0; i < AP; ++i) xv2[i] = GATHER ? (n2 ? xv_n[i] : xv_c[i]) : tv[i];
            // K step 0: second half of weight slab kt + 1.
            settle(std::integral_constant<int, 0>{});
            kstep(std::integral_constant<int, 0>{}, abase, wbase, 1, [&](auto CC) {
                copy_w(std::integral_constant<int, BP / 2 + decltype(CC)::value>{}, ws1, so1, wr1);
            });
            // K steps 1 and 2: token slab kt + 2.
            settle(std::integral_constant<int, 1>{});
            kstep(std::integral_constant<int, 1>{}, abase, wbase, 2, [&](auto CC) {
                copy_a(std::integral_constant<int, decltype(CC)::value>{}, as2, so2, xr2, xv2);
            });
            settle(std::integral_constant<int, 0>{});
            kstep(std::integral_constant<int, 0>{}, abase, wbase, 3, [&](auto CC) {
                copy_a(std::integral_constant<int, 4 + decltype(CC)::value>{}, as2, so2, xr2, xv2);
            });
            settle(std::integral_constant<int, 1>{});
            // Token and weight slab kt + 1 have landed for this wave (only the
            // eight token copies of slab kt + 2 may be younger); after the
            // barrier, for every wave, and every wave is done reading slab kt.
            wait_vmcnt<AP>();
            barrier_no_fence();
            // K step 3: first fragments of slab kt + 1; first half of weight
            // slab kt + 2 into the weight slot of slab kt.
            kstep(std::integral_constant<int, 1>{}, (uint32_t)as1 * SLAB, (uint32_t)ws1 * SLAB, 0, [&](auto CC) {
                copy_w(std::integral_constant<int, decltype(CC)::value>{}, ws, so2w, wr2);
            });
            as = as1;
            ws = ws1;
        } while (++kt < tc.nk);

        // The last K step also read the next tile's first fragments; let them
        // land (their registers are reused by the epilogue) and read them again
        // after it.
        settle(std::integral_constant<int, 0>{});
        // Gathered rows of the tile after next: read now, used after the epilogue.
        if (GATHER && has_nn) load_tokens(tnn, tok);
        // Router logits: the tile's token rows' sums of squares (the first
        // column tile's waves of column block 0 write them), then zero for
        // the next tile.
        if constexpr (RNORM) {
#pragma unroll
            for (int i = 0; i < FB; ++i) {
                const float v = xsq[i] + __shfl_xor(xsq[i], 32);
                const int r = wm * WT + i * 32 + fr;
                if (tc.n0 == 0 && wn == 0 && fk == 0 && r < tc.rows)
                    store4_asm(static_cast<float*>(a.C2) + tc.row0 + r, __float_as_uint(v));
                xsq[i] = 0.0f;
            }
        }
        // The last slab's token slot is free (and read by no wave any more).
        epilogue(tc, as == 0 ? AST - 1 : as - 1);
        // The combine's loads land in registers the next K loop reuses; a wait
        // the compiler sees (vmcnt(0)) retires them here, once per tile,
        // instead of the conservative waits it would otherwise put at the head
        // of every K step.
        if (COMBINE) __builtin_amdgcn_s_waitcnt(0xF70);
        if (!has_n) break;

        // Advance: n -> c, nn -> n, and the table entry of the tile after that.
        lid += wpx;
        tc = tn;
        xres_c = xres_n;
        wres_c = wres_n;
        has_n = has_nn;
        tn = tnn;
        xres_n = has_n ? xres_of(tn) : xnull;
        wres_n = has_n ? wres_of(tn) : wnull;
        if (GATHER) {
#pragma unroll
            for (int i = 0; i < AP; ++i) xv_c[i] = xv_n[i];
            if (has_n) token_offsets(tok, xv_n);
        }
        has_nn = lid + 2 * wpx < lid_end;
        if (has_nn) tnn = tile_of(lid + 2 * wpx, ent3);
        ent3 = tile_entry(lid + 3 * wpx);
        if (SCATTER) load_slots(tc);
#pragma unroll
        for (int j = 0; j < FB; ++j)
#pragma unroll
            for (int i = 0; i < FB; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.0f;
        // Every wave has read its staged rows before the next tile's token
        // copies refill that slot.
        barrier_no_fence();
        static_for<2 * FB>([&](auto QC) {
            read_frag(std::integral_constant<int, 0>{}, QC, (uint32_t)as * SLAB, (uint32_t)ws * SLAB, 0);
        });
    }
    wait_vmcnt<0>();
}

// fp32 path (used by the fp32 layer): 64x64 tiles on the vector ALUs, 4x4
// outputs per thread, K slabs of 16 staged through LDS.
template <int EPI, bool GROUPED>
__global__ __launch_bounds__(256) void k_gemm_f32(const GemmArgs a) {
    constexpr int BM = 64, BN = 64, BK = 16;
    __shared__ __attribute__((aligned(16))) float As[BK][BM + 4];
    __shared__ __attribute__((aligned(16))) float Bs[BK][BN + 4];
    __shared__ int32_t srow[BM];
    const TileCoord tc = locate_tile<GROUPED>(a, BM, BN);
    if (!tc.valid) return;
    const int tid = threadIdx.x;
    for (int r = tid; r < BM; r += 256) {
        const int rr = r < tc.rows ? r : tc.rows - 1;
        const int p = tc.row0 + rr;
        int v = p;
        if (EPI == EPI_GELU_STORE && a.row_mode == ROWS_GATHER_TOKENS) v = a.row_map[p] / a.route_k;
        if (EPI == EPI_SCATTER_SLOT) v = a.row_map[p];
        srow[r] = v;
    }
    __syncthreads();
    const float* __restrict__ A = static_cast<const float*>(a.A);
    const float* __restrict__ B = static_cast<const float*>(a.B) + (size_t)tc.e * a.b_group_stride;
    const int Kd = a.Kdim;
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int arow = (EPI == EPI_GELU_STORE) ? srow[lr] : tc.row0 + (lr < tc.rows ? lr : tc.rows - 1);
    const float* ap = A + (size_t)arow * Kd + lk;
    const float* bp = B + (size_t)(tc.n0 + lr) * Kd + lk;
    const int tx = tid & 15, ty = tid >> 4;
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
    for (int k0 = 0; k0 < Kd; k0 += BK) {
        const float4 va = *reinterpret_cast<const float4*>(ap + k0);
        const float4 vb = *reinterpret_cast<const float4*>(bp + k0);
        As[lk + 0][lr] = va.x; As[lk + 1][lr] = va.y; As[lk + 2][lr] = va.z; As[lk + 3][lr] = va.w;
        Bs[lk + 0][lr] = vb.x; Bs[lk + 1][lr] = vb.y; Bs[lk + 2][lr] = vb.z; Bs[lk + 3][lr] = vb.w;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < BK; ++k) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[k][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[k][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = ty + 16 * i;
        if (r >= tc.rows) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = tc.n0 + tx + 16 * j;
            const float val = acc[i][j];
            float* C = static_cast<float*>(a.C);
            if (EPI == EPI_GELU_STORE) C[(size_t)(tc.row0 + r) * a.N + c] = gelu_erf(val);
            else if (EPI == EPI_SCATTER_SLOT) C[(size_t)srow[r] * a.N + c] = val;
            else C[(size_t)(tc.row0 + r) * a.N + c] = val;
        }
    }
}

template <int BM, int BN, int WM, int WN, int BK, int ST, int WPE, int EPI, bool GROUPED>
hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
    if (a.CT) return hipErrorInvalidValue;  // transposed outputs exist on the persistent kernel only
    const int n_n = a.N / BN;
    const long long total = (long long)a.max_tiles * n_n;
    const long long grid = (total + kNumXcd - 1) / kNumXcd * kNumXcd;
    // Split K (dense fp32 output only): the parts along the grid's y.
    const int splits = (!GROUPED && EPI == EPI_STORE_F32 && a.k_splits > 1) ? a.k_splits : 1;
    if (splits > 1 && (a.Kdim / BK) % splits) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, BK, ST, EPI, GROUPED, WPE>), dim3((unsigned)grid, splits),
                       dim3(WM * WN * kWave), 0, s, a);
    return hipGetLastError();
}

// Workgroups of the persistent kernel: one per CU (a multiple of the XCD
// count), fewer when the grid-sizing bound on the tiles is smaller.
int persistent_grid(long long tile_bound) {
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < kNumXcd)
            n = 256;
        cus[dev] = n / kNumXcd * kNumXcd;
    }
    const long long bound = (tile_bound + kNumXcd - 1) / kNumXcd * kNumXcd;
    return (int)(bound < cus[dev] ? bound : cus[dev]);
}

template <int EPI, bool GROUPED, int KC = 8>
hipError_t launch_pp(const GemmArgs& a, hipStream_t s) {
    if (a.CT && !ct_epi(EPI)) return hipErrorInvalidValue;
    const int grid = persistent_grid((long long)a.max_tiles * (a.N / 256));
    hipLaunchKernelGGL((k_gemm_pp<EPI, GROUPED, KC>), dim3((unsigned)grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// The fused combine is compiled for each K (its gate and expert-row loads are
// unrolled over the K slots).
hipError_t launch_pp_combine(const GemmArgs& a, hipStream_t s) {
    switch (a.route_k) {
        case 1: return launch_pp<EPI_COMBINE, false, 1>(a, s);
        case 2: return launch_pp<EPI_COMBINE, false, 2>(a, s);
        case 3: return launch_pp<EPI_COMBINE, false, 3>(a, s);
        case 4: return launch_pp<EPI_COMBINE, false, 4>(a, s);
        case 5: return launch_pp<EPI_COMBINE, false, 5>(a, s);
        case 6: return launch_pp<EPI_COMBINE, false, 6>(a, s);
        case 7: return launch_pp<EPI_COMBINE, false, 7>(a, s);
        case 8: return launch_pp<EPI_COMBINE, false, 8>(a, s);
    }
    return hipErrorInvalidValue;
}

template <int EPI, bool GROUPED>
hipError_t launch_sp(const GemmArgs& a, hipStream_t s) {
    const int n_n = a.N / 256;
    const long long total = (long long)a.max_tiles * n_n;
    const long long grid = (total + kNumXcd - 1) / kNumXcd * kNumXcd;
    hipLaunchKernelGGL((k_gemm_sp<EPI, GROUPED>), dim3((unsigned)grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int EPI, bool GROUPED>
hipError_t launch_f32(const GemmArgs& a, hipStream_t s) {
    const int n_n = a.N / 64;
    const long long total = (long long)a.max_tiles * n_n;
    const long long grid = (total + kNumXcd - 1) / kNumXcd * kNumXcd;
    hipLaunchKernelGGL((k_gemm_f32<EPI, GROUPED>), dim3((unsigned)grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// Tile shapes. Large groups (M-tiles of 256 token rows): 256 x 256 on the
// persistent kernel when N allows and K spans at least two slabs (the paced
// one-tile kernel for one slab), else 256 x 128 or 256 x 64 tiled. Small
// groups (M-tiles of 64 rows, the weight-read-bound regime where an expert
// sees a few dozen tokens): 64 x 128 or 64 x 64 with three slabs in the ring
// and several workgroups per CU, to keep many weight loads in flight.
template <int EPI, bool GROUPED>
hipError_t dispatch_bf16(int bm, const GemmArgs& a, hipStream_t s) {
    if (bm == 256) {
        if (a.N % 256 == 0) {
            const bool gather_ok = !(GROUPED && EPI == EPI_GELU_STORE) || a.row_mode == ROWS_GATHER_TOKENS;
            if (a.Kdim >= 128 && gather_ok) return launch_pp<EPI, GROUPED>(a, s);
            return launch_sp<EPI, GROUPED>(a, s);
        }
        // The grouped layers with N an odd multiple of 128 (ViT-B's h = 384):
        // N rounded up to the persistent kernel's 256-column tile, weight rows
        // past N read as zeros and columns past N not stored. A third more
        // MFMA work than the 256 x 128 tiles, but on the persistent kernel.
        if constexpr (GROUPED && (EPI == EPI_GELU_STORE || EPI == EPI_SCATTER_SLOT))
            if (a.N % 128 == 0 && a.Kdim >= 128 &&
                (EPI == EPI_SCATTER_SLOT || a.row_mode == ROWS_GATHER_TOKENS)) {
                GemmArgs p = a;
                p.b_rows = a.N;
                p.ldc = a.N;
                p.N = (a.N + 255) / 256 * 256;
                return launch_pp<EPI, GROUPED>(p, s);
            }
        if (a.N % 128 == 0) return launch_bf16<256, 128, 2, 2, 64, 2, 1, EPI, GROUPED>(a, s);
        return launch_bf16<256, 64, 4, 1, 64, 2, 1, EPI, GROUPED>(a, s);
    }
    if (bm == 64) {
        if (a.N % 128 == 0) return launch_bf16<64, 128, 1, 4, 64, 3, 2, EPI, GROUPED>(a, s);
        return launch_bf16<64, 64, 2, 2, 64, 3, 2, EPI, GROUPED>(a, s);
    }
    return hipErrorInvalidValue;
}

// Backward products: the persistent kernel on 256-row tiles where the widths
// allow (rounded up to the tile for SwiGLU dA and the weight gradients), else
// the tiled kernel with 256- or 64-row tiles.
template <int EPI, bool GROUPED>
hipError_t dispatch_tiled(int bm, const GemmArgs& a, hipStream_t s) {
    constexpr bool ROW_PRODUCT = EPI == EPI_GELU_BWD || EPI == EPI_DGELU || EPI == EPI_SCATTER_SLOT_F32;
    if constexpr (ROW_PRODUCT)
        if (bm == 256 && a.N % 256 == 0 && a.Kdim >= 128) return launch_pp<EPI, GROUPED>(a, s);
    // SwiGLU dA: N = act_ld rounded up to the tile width; W2's transposed rows
    // past act_ld read as zeros and those columns are not stored.
    if constexpr (EPI == EPI_DSWIGLU)
        if (bm == 256 && a.Kdim >= 128) {
            GemmArgs p = a;
            p.b_rows = a.act_ld;
            p.N = (a.act_ld + 255) / 256 * 256;
            return launch_pp<EPI, GROUPED>(p, s);
        }
    // Weight gradients: every work item spans at least two K slabs; N is
    // rounded up to the tile width (B rows past N only feed unstored columns).
    if constexpr (EPI == EPI_WGRAD_F32)
        if (bm == 256 && a.dense_rows % 256 == 0) {
            GemmArgs p = a;
            p.ldc = a.N;
            p.N = (a.N + 255) / 256 * 256;
            return launch_pp<EPI, GROUPED>(p, s);
        }
    if (bm == 256) {
        if (a.N % 128 == 0) return launch_bf16<256, 128, 2, 2, 64, 2, 1, EPI, GROUPED>(a, s);
        return launch_bf16<256, 64, 4, 1, 64, 2, 1, EPI, GROUPED>(a, s);
    }
    if (bm == 64) {
        if (a.N % 128 == 0) return launch_bf16<64, 128, 1, 4, 64, 3, 2, EPI, GROUPED>(a, s);
        return launch_bf16<64, 64, 2, 2, 64, 3, 2, EPI, GROUPED>(a, s);
    }
    return hipErrorInvalidValue;
}

// SwiGLU first layer: the virtual column count N follows from the tile shape
// (each tile of BN columns computes BN / 2 activation columns).
template <bool GROUPED>
hipError_t dispatch_swiglu(int bm, GemmArgs a, hipStream_t s) {
    if (a.act_n < 1 || a.act_ld < a.act_n || a.act_ld % 64) return hipErrorInvalidValue;
    if (bm == 256) {
        if (a.Kdim < 128 || (GROUPED && a.row_mode != ROWS_GATHER_TOKENS)) return hipErrorInvalidValue;
        a.N = 2 * ((a.act_ld + 127) / 128 * 128);
        return launch_pp<EPI_SWIGLU_STORE, GROUPED>(a, s);
    }
    if (bm == 64) {
        a.N = 2 * a.act_ld;
        return launch_bf16<64, 128, 2, 2, 64, 3, 2, EPI_SWIGLU_STORE, GROUPED>(a, s);
    }
    return hipErrorInvalidValue;
}

// Backward's first-layer recompute for SwiGLU experts: the persistent kernel
// (as the forward), else the tiled kernel with 2 x 2 waves (each wave 32 gate
// + 32 up columns), N = 2 act_ld.
hipError_t dispatch_swiglu_bwd(int bm, GemmArgs a, hipStream_t s) {
    if (a.act_n < 1 || a.act_ld < a.act_n || a.act_ld % 64) return hipErrorInvalidValue;
    if (bm == 256 && a.Kdim >= 128) {
        a.N = 2 * ((a.act_ld + 127) / 128 * 128);
        return launch_pp<EPI_SWIGLU_BWD, true>(a, s);
    }
    a.N = 2 * a.act_ld;
    if (bm == 256) return launch_bf16<256, 128, 2, 2, 64, 2, 1, EPI_SWIGLU_BWD, true>(a, s);
    if (bm == 64) return launch_bf16<64, 128, 2, 2, 64, 3, 2, EPI_SWIGLU_BWD, true>(a, s);
    return hipErrorInvalidValue;
}

template <bool GROUPED>
hipError_t dispatch(const moe_desc_t& d, int epilogue, int bm, const GemmArgs& a, hipStream_t s) {
    if (d.dtype == MOE_BF16) {
        switch (epilogue) {
            case EPI_GELU_STORE: return dispatch_bf16<EPI_GELU_STORE, GROUPED>(bm, a, s);
            case EPI_SWIGLU_STORE: return dispatch_swiglu<GROUPED>(bm, a, s);
            case EPI_GELU_BWD:
                if (GROUPED) return dispatch_tiled<EPI_GELU_BWD, true>(bm, a, s);
                break;
            case EPI_DGELU:
                if (GROUPED) return dispatch_tiled<EPI_DGELU, true>(bm, a, s);
                break;
            case EPI_SCATTER_SLOT_F32:
                if (GROUPED) return dispatch_tiled<EPI_SCATTER_SLOT_F32, true>(bm, a, s);
                break;
            case EPI_WGRAD_F32:
                if (GROUPED && a.dense_rows % bm == 0) return dispatch_tiled<EPI_WGRAD_F32, true>(bm, a, s);
                break;
            case EPI_SWIGLU_BWD:
                if (GROUPED) return dispatch_swiglu_bwd(bm, a, s);
                break;
            case EPI_DSWIGLU:
                if (GROUPED) return dispatch_tiled<EPI_DSWIGLU, true>(bm, a, s);
                break;
            case EPI_SCATTER_SLOT:
                if (GROUPED) return dispatch_bf16<EPI_SCATTER_SLOT, true>(bm, a, s);
                break;
            case EPI_STORE_F32:
                if (!GROUPED) return dispatch_bf16<EPI_STORE_F32, false>(bm, a, s);
                break;
            case EPI_ROUTER_F32:
                if (!GROUPED && bm == 256 && a.N % 256 == 0 && a.Kdim >= 128 && a.k_splits <= 1 && a.C2)
                    return launch_pp<EPI_ROUTER_F32, false>(a, s);
                break;
            case EPI_COMBINE:
                if (!GROUPED && gemm_combine_fusable(d, bm, a.N, a.Kdim) && a.route_k == d.K)
                {
                    if (bm == 256) return launch_pp_combine(a, s);
                    if (a.N % 128 == 0) return launch_bf16<64, 128, 1, 4, 64, 3, 2, EPI_COMBINE, false>(a, s);
                    return launch_bf16<64, 64, 2, 2, 64, 3, 2, EPI_COMBINE, false>(a, s);
                }
                break;
        }
    } else {
        if (bm != 64) return hipErrorInvalidValue;
        switch (epilogue) {
            case EPI_GELU_STORE: return launch_f32<EPI_GELU_STORE, GROUPED>(a, s);
            case EPI_SCATTER_SLOT:
                if (GROUPED) return launch_f32<EPI_SCATTER_SLOT, true>(a, s);
                break;
            case EPI_STORE_F32:
                if (!GROUPED) return launch_f32<EPI_STORE_F32, false>(a, s);
                break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

int gemm_tile_bm(int32_t dtype, int64_t avg_rows) {
    if (dtype != MOE_BF16) return 64;
    return avg_rows >= 512 ? 256 : 64;
}

int gemm_dense_bm(int32_t dtype, int64_t rows, int32_t n) {
    if (dtype != MOE_BF16) return 64;
    // 256-row tiles only when they still give a few workgroups per CU.
    const int64_t tiles = (rows + 255) / 256 * (n / 256 > 0 ? n / 256 : 1);
    return tiles >= 512 ? 256 : 64;
}

bool gemm_backward_transposed(const moe_desc_t& d, int bm) {
    // The same conditions under which dispatch_tiled / dispatch_swiglu_bwd pick
    // the persistent kernel for the recompute (K = d) and dA (K = d) products.
    if (d.dtype != MOE_BF16 || bm != 256 || d.d < 128) return false;
    if (d.flags & MOE_FLAG_SWIGLU) return true;  // widths rounded up to the tile
    return d.h % 256 == 0;
}

bool gemm_combine_fusable(const moe_desc_t& d, int bm, int n, int kdim) {
    // The persistent 256 x 256 kernel with its combine epilogue, or the
    // 64-row tiled kernel with its own (K <= 8 either way).
    if (d.dtype != MOE_BF16 || d.K > kMaxCombineK) return false;
    return (bm == 256 && n % 256 == 0 && kdim >= 128) || (bm == 64 && n % 64 == 0);
}

hipError_t launch_gemm(const moe_desc_t& d, int epilogue, int bm, const GemmArgs& a, hipStream_t s) {
    // Grouped (routed experts, tile table) and dense (shared expert) launches
    // are separate kernel instances.
    if (a.tiles) return dispatch<true>(d, epilogue, bm, a, s);
    return dispatch<false>(d, epilogue, bm, a, s);
}

}  // namespace moe
