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
// K-contiguous (token rows and nn.Linear weight rows), staged through LDS in
// 64-wide K slabs, double-buffered, one barrier per slab. A 16-byte chunk c of
// LDS row r is stored at chunk c ^ (r & 7), so the 32 rows a fragment read
// touches spread over all banks.
#include "moe_internal.h"

#include <math.h>

namespace moe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

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

template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI, bool GROUPED>
__global__ __launch_bounds__(WAVES_M* WAVES_N* kWave) void k_gemm_bf16(const GemmArgs a) {
    constexpr int NT = WAVES_M * WAVES_N * kWave;
    constexpr int BK = 64;             // K slab: 64 bf16 = 128 bytes = 8 chunks per row
    constexpr int ROWB = BK * 2;
    constexpr int WTM = BM / WAVES_M;  // wave tile
    constexpr int WTN = BN / WAVES_N;
    constexpr int FM = WTM / 32;
    constexpr int FN = WTN / 32;
    constexpr int ACH = BM * 8 / NT;  // 16-byte chunks per thread per slab
    constexpr int BCH = BN * 8 / NT;
    static_assert(ACH * NT == BM * 8 && BCH * NT == BN * 8, "tile / thread mismatch");
    constexpr int STAGE = (BM + BN) * ROWB;
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];
    __shared__ int32_t srow[BM];

    const TileCoord tc = locate_tile<GROUPED>(a, BM, BN);
    if (!tc.valid) return;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // Row ids of this tile: A source rows (gather) or output rows (scatter).
    for (int r = tid; r < BM; r += NT) {
        const int rr = r < tc.rows ? r : tc.rows - 1;  // pad rows repeat the last valid row
        const int p = tc.row0 + rr;
        int v = p;
        if (EPI == EPI_GELU_STORE && a.row_mode == ROWS_GATHER_TOKENS) v = a.row_map[p] / a.route_k;
        if (EPI == EPI_SCATTER_SLOT) v = a.row_map[p];
        srow[r] = v;
    }
    __syncthreads();

    const bf16_t* __restrict__ A = static_cast<const bf16_t*>(a.A);
    const bf16_t* __restrict__ B = static_cast<const bf16_t*>(a.B) + (size_t)tc.e * a.b_group_stride;
    const int Kd = a.Kdim;

    const bf16_t* ap[ACH];
    int a_lds[ACH];
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
        const int q = tid + NT * i;
        const int r = q >> 3, c = q & 7;
        int arow;
        if (EPI == EPI_GELU_STORE) arow = srow[r];  // gathered token row or identity row
        else arow = tc.row0 + (r < tc.rows ? r : tc.rows - 1);
        ap[i] = A + (size_t)arow * Kd + c * 8;
        a_lds[i] = r * ROWB + ((c ^ (r & 7)) << 4);
    }
    const bf16_t* bp[BCH];
    int b_lds[BCH];
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
        const int q = tid + NT * i;
        const int r = q >> 3, c = q & 7;
        bp[i] = B + (size_t)(tc.n0 + r) * Kd + c * 8;
        b_lds[i] = BM * ROWB + r * ROWB + ((c ^ (r & 7)) << 4);
    }

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    u32x4_t ra[ACH], rb[BCH];
#define MOE_GLOAD(k0)                                                                        \
    do {                                                                                     \
        _Pragma("unroll") for (int i = 0; i < ACH; ++i) ra[i] =                              \
            *reinterpret_cast<const u32x4_t*>(ap[i] + (k0));                                   \
        _Pragma("unroll") for (int i = 0; i < BCH; ++i) rb[i] =                              \
            *reinterpret_cast<const u32x4_t*>(bp[i] + (k0));                                   \
    } while (0)
#define MOE_LSTORE(stage)                                                                    \
    do {                                                                                     \
        uint8_t* base_ = smem + (stage) * STAGE;                                             \
        _Pragma("unroll") for (int i = 0; i < ACH; ++i)                                      \
            *reinterpret_cast<u32x4_t*>(base_ + a_lds[i]) = ra[i];                             \
        _Pragma("unroll") for (int i = 0; i < BCH; ++i)                                      \
            *reinterpret_cast<u32x4_t*>(base_ + b_lds[i]) = rb[i];                             \
    } while (0)

    // Fragment rows of this lane (the same for every slab).
    const int fr = lane & 31;   // row within a 32-row block
    const int fk = lane >> 5;   // which 8-wide half of each 16-wide K step

    const int nk = Kd / BK;
    MOE_GLOAD(0);
    MOE_LSTORE(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk) MOE_GLOAD((kt + 1) * BK);
        const uint8_t* base = smem + (kt & 1) * STAGE;
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int ch = ks * 2 + fk;
            bf16x8_t af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = wm * WTM + i * 32 + fr;
                af[i] = *reinterpret_cast<const bf16x8_t*>(base + r * ROWB + ((ch ^ (r & 7)) << 4));
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = wn * WTN + j * 32 + fr;
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(base + BM * ROWB + r * ROWB + ((ch ^ (r & 7)) << 4));
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) MOE_LSTORE((kt + 1) & 1);
        __syncthreads();
    }
#undef MOE_GLOAD
#undef MOE_LSTORE

    // Epilogue. Accumulator v of a 32x32 block sits at row 8*(v/4) + 4*(lane/32)
    // + v%4 and column lane%32.
    const int col_in = lane & 31;
    const int row_in = (lane >> 5) * 4;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int c = tc.n0 + wn * WTN + j * 32 + col_in;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = wm * WTM + i * 32 + (v >> 2) * 8 + row_in + (v & 3);
                if (r >= tc.rows) continue;
                const float val = acc[i][j][v];
                if (EPI == EPI_GELU_STORE) {
                    static_cast<bf16_t*>(a.C)[(size_t)(tc.row0 + r) * a.N + c] = f32_to_bf16_rne(gelu_erf(val));
                } else if (EPI == EPI_SCATTER_SLOT) {
                    static_cast<bf16_t*>(a.C)[(size_t)srow[r] * a.N + c] = f32_to_bf16_rne(val);
                } else {
                    static_cast<float*>(a.C)[(size_t)(tc.row0 + r) * a.N + c] = val;
                }
            }
        }
    }
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

template <int BM, int BN, int WM, int WN, int EPI, bool GROUPED>
hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
    const int n_n = a.N / BN;
    const long long total = (long long)a.max_tiles * n_n;
    const long long grid = (total + kNumXcd - 1) / kNumXcd * kNumXcd;
    hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, EPI, GROUPED>), dim3((unsigned)grid), dim3(WM * WN * kWave),
                       0, s, a);
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

template <int EPI, bool GROUPED>
hipError_t dispatch_bf16(int bm, const GemmArgs& a, hipStream_t s) {
    if (bm != 128) return hipErrorInvalidValue;
    if (a.N % 128 == 0) return launch_bf16<128, 128, 2, 2, EPI, GROUPED>(a, s);
    return launch_bf16<128, 64, 2, 2, EPI, GROUPED>(a, s);
}

template <bool GROUPED>
hipError_t dispatch(const moe_desc_t& d, int epilogue, int bm, const GemmArgs& a, hipStream_t s) {
    if (d.dtype == MOE_BF16) {
        switch (epilogue) {
            case EPI_GELU_STORE: return dispatch_bf16<EPI_GELU_STORE, GROUPED>(bm, a, s);
            case EPI_SCATTER_SLOT: return dispatch_bf16<EPI_SCATTER_SLOT, GROUPED>(bm, a, s);
            case EPI_STORE_F32: return dispatch_bf16<EPI_STORE_F32, GROUPED>(bm, a, s);
        }
    } else {
        if (bm != 64) return hipErrorInvalidValue;
        switch (epilogue) {
            case EPI_GELU_STORE: return launch_f32<EPI_GELU_STORE, GROUPED>(a, s);
            case EPI_SCATTER_SLOT: return launch_f32<EPI_SCATTER_SLOT, GROUPED>(a, s);
            case EPI_STORE_F32: return launch_f32<EPI_STORE_F32, GROUPED>(a, s);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

int gemm_tile_bm(int32_t dtype) { return dtype == MOE_BF16 ? 128 : 64; }

hipError_t launch_gemm(const moe_desc_t& d, int epilogue, int bm, const GemmArgs& a, hipStream_t s) {
    // Grouped (routed experts, tile table) and dense (shared expert) launches
    // are separate kernel instances.
    if (a.tiles) {
        // Only the two routed stages run grouped.
        if (epilogue == EPI_STORE_F32) return hipErrorInvalidValue;
        return dispatch<true>(d, epilogue, bm, a, s);
    }
    if (epilogue == EPI_SCATTER_SLOT) return hipErrorInvalidValue;
    return dispatch<false>(d, epilogue, bm, a, s);
}

}  // namespace moe
