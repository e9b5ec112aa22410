// Data-movement kernels of the expert-MLP backward: weight transposes, the
// plan of the weight-gradient products (per-expert K windows cut into work
// items) and the sum of their partial blocks, the transposing gather into the
// windows and the zeroing of empty experts' windows, and the per-token sum of
// the slot gradients. The
// products themselves run on the MFMA kernels of gemm.hip.
#include "moe_internal.h"

namespace moe {
namespace {

// 16-byte store with the non-temporal hint: the transposed operands are read
// by a later kernel, and keeping their lines in L2 only evicts data still in
// use (1 % of the backward at ViT-G).
__device__ __forceinline__ void store16_nt(void* p, const uint4& v) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4*>(p));
}

constexpr int TT = 64;  // transpose tile (rows x columns)

// out[g][c][r] = in[g][src(r)][c]: the transpose of a [G][Rs][C] bf16 tensor
// viewed as R rows (R, C multiples of 64). Without padding (ld = 0) src(r) =
// r and R = Rs. With padding (stacked gate and up rows of h each, ld = h
// rounded up to 64, R = 2 ld): rows r < ld are gate row r, rows ld + i are up
// row h + i, and rows past h in either half are zero. One 64 x 64 tile per
// workgroup through LDS: 16-byte row pieces in, 16-byte pieces of the
// transposed rows out.
__global__ __launch_bounds__(256) void k_transpose_w(const bf16_t* __restrict__ in, int Rs, int R, int C, int h,
                                                    int ld, bf16_t* __restrict__ out) {
    __shared__ bf16_t tile[TT][TT + 2];
    const int r0 = blockIdx.x * TT, c0 = blockIdx.y * TT;
    const size_t g = blockIdx.z;
    const bf16_t* src = in + g * (size_t)Rs * C;
    bf16_t* dst = out + g * (size_t)R * C;
    const int tid = threadIdx.x;
    for (int q = tid; q < TT * TT / 8; q += 256) {
        const int r = q / (TT / 8), c = (q % (TT / 8)) * 8;
        int sr = r0 + r;
        if (ld > 0) {
            const int up = sr >= ld, i = sr - (up ? ld : 0);
            sr = i < h ? i + (up ? h : 0) : -1;
        }
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (sr >= 0) v = *reinterpret_cast<const uint4*>(src + (size_t)sr * C + c0 + c);
        const bf16_t* e = reinterpret_cast<const bf16_t*>(&v);
#pragma unroll
        for (int k = 0; k < 8; ++k) tile[r][c + k] = e[k];
    }
    __syncthreads();
    for (int q = tid; q < TT * TT / 8; q += 256) {
        const int c = q / (TT / 8), r = (q % (TT / 8)) * 8;
        uint4 v;
        bf16_t* e = reinterpret_cast<bf16_t*>(&v);
#pragma unroll
        for (int k = 0; k < 8; ++k) e[k] = tile[r + k][c];
        store16_nt(dst + (size_t)(c0 + c) * R + r0 + r, v);
    }
}

// Plan of the weight-gradient products, one workgroup:
//  - K windows: expert e owns columns koff[e] .. koff[e+1] of the transposed
//    operands, its row count rounded up to a multiple of 64 (the K slab) and
//    to at least two slabs (the persistent kernel's pipeline holds two; an
//    empty expert's window is all zeros, so its gradient comes out 0);
//  - work items: each window cut into pieces of at most kWgradSlabs slabs,
//    split evenly (sizes differ by at most one slab, and every piece keeps
//    at least two slabs, as a window does), so that no tile runs
//    much longer than the others under a skewed load. An expert with one
//    piece writes its gradient directly (dest = -1); the pieces of a longer
//    window write partial blocks dest = first .. first + n - 1, summed
//    afterwards in that order;
//  - rlist: the split experts {e, first partial block, pieces}.
// wcount[0] = items, wcount[1] = split experts.
__global__ __launch_bounds__(1024) void k_wgrad_plan(const int32_t* __restrict__ offsets, int E,
                                                    int32_t* __restrict__ koff, TileDesc* __restrict__ items,
                                                    TileDesc* __restrict__ rlist, int32_t* __restrict__ wcount) {
    __shared__ int32_t len[kMaxE], pieces[kMaxE], pfirst[kMaxE], rslot[kMaxE];
    __shared__ int32_t cursor[kWgradSlabs + 1];  // next item position per piece length (slabs)
    __shared__ int32_t nitems_s;
    constexpr int CHUNK = kWgradSlabs * 64;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        len[e] = max(128, (offsets[e + 1] - offsets[e] + 63) / 64 * 64);
        pieces[e] = (len[e] + CHUNK - 1) / CHUNK;
    }
    __syncthreads();
    for (int i = threadIdx.x; i <= kWgradSlabs; i += blockDim.x) cursor[i] = 0;
    if (threadIdx.x == 0) {
        int32_t k = 0, it = 0, pt = 0, rs = 0;
        for (int e = 0; e < E; ++e) {
            koff[e] = k;
            pfirst[e] = pieces[e] > 1 ? pt : -1;
            rslot[e] = pieces[e] > 1 ? rs : -1;
            k += len[e];
            it += pieces[e];
            if (pieces[e] > 1) {
                pt += pieces[e];
                ++rs;
            }
        }
        koff[E] = k;
        wcount[0] = it;
        nitems_s = it;
        wcount[1] = rs;
    }
    __syncthreads();
    // Items in descending order of length (slabs, 2 .. kWgradSlabs), so that
    // the persistent workgroups running neighbouring items stay in step and
    // the row and column tiles of one item meet in L2 slab by slab (and the
    // longest items start first), dealt round-robin over the XCDs: each XCD
    // walks a contiguous range of the list, so rank p goes to range p % 8 as
    // its (p / 8)-th item, and every range gets the same mix of lengths.
    // Placement within one length follows LDS atomics; every item writes
    // fixed outputs, so the order changes no result.
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        const int slabs = len[e] / 64, n = pieces[e];
        const int base = slabs / n, extra = slabs % n;
        if (extra) atomicAdd(&cursor[base + 1], extra);
        if (n > extra) atomicAdd(&cursor[base], n - extra);
    }
    __syncthreads();
    const int nitems = nitems_s;
    if (threadIdx.x == 0) {
        int run = 0;
        for (int sz = kWgradSlabs; sz >= 0; --sz) {
            const int c = cursor[sz];
            cursor[sz] = run;
            run += c;
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        const int slabs = len[e] / 64, n = pieces[e];
        const int base = slabs / n, extra = slabs % n;  // the first `extra` pieces take one more slab
        int s0 = 0;
        for (int c = 0; c < n; ++c) {
            const int sz = base + (c < extra ? 1 : 0);
            TileDesc t;
            t.e = e;
            t.row0 = koff[e] + s0 * 64;
            t.rows = sz * 64;
            t.pad = pfirst[e] < 0 ? -1 : pfirst[e] + c;
            const int p = atomicAdd(&cursor[sz], 1), b = p % kNumXcd;
            items[b * (nitems / kNumXcd) + min(b, nitems % kNumXcd) + p / kNumXcd] = t;
            s0 += sz;
        }
        if (rslot[e] >= 0) rlist[rslot[e]] = TileDesc{e, pfirst[e], pieces[e], 0};
    }
}

// Gradients of the split experts: out[e] = sum of its partial blocks in
// order (fp32), four elements per thread. The split experts (their number is
// known on the device only) are dealt to the gridDim.y rows of workgroups in
// turn, so that the grid does not hold a row per expert that mostly exits.
__global__ __launch_bounds__(256) void k_wgrad_reduce(const float* __restrict__ partials,
                                                     const TileDesc* __restrict__ rlist,
                                                     const int32_t* __restrict__ wcount, size_t mn,
                                                     float* __restrict__ out) {
    const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (i >= mn) return;
    const int nsplit = wcount[1];
    for (int y = blockIdx.y; y < nsplit; y += gridDim.y) {
        const TileDesc r = rlist[y];
        float4 acc = *reinterpret_cast<const float4*>(partials + (size_t)r.row0 * mn + i);
        for (int c = 1; c < r.rows; ++c) {
            const float4 v = *reinterpret_cast<const float4*>(partials + ((size_t)r.row0 + c) * mn + i);
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        *reinterpret_cast<float4*>(out + (size_t)r.e * mn + i) = acc;
    }
}

// Transposing gather into the K windows: out[c][q] for window position q of
// expert e (q = koff[e] + i) is in[src(offsets[e] + i)][c] when i < count_e,
// and 0 in the padding up to the window's end. src(p) is p (rows already in
// sorted order), row_map[p] (slot rows) or row_map[p] / K (token rows).
// in: [rows, C] bf16; out: [C, ld] bf16 stored slab-major, [ld / 64][C][64]
// (element (c, q) at ((q / 64) C + c) 64 + q % 64), so that one 64-column K
// slab of a product's operand tile is contiguous. C a multiple of 64.
// Positions past koff[E] are left alone.
//
// A workgroup moves one 64-position block across all C columns. Windows are
// multiples of 64, so the block lies in one expert's window: one search per
// workgroup. Lane (rg, cg) of a wave holds an 8 x 8 block, positions 8 rg ..
// 8 rg + 7 and 8 columns: it loads 8 16-byte row pieces, transposes them in
// registers and stores 8 16-byte column pieces. The 8 lanes of one cg cover a
// whole 128-byte line both ways: 8 rows' 8 columns in, one column's 64
// positions out. The 4 waves take 64-column quarters of each 256-column step.
__device__ __forceinline__ uint32_t pair16(uint32_t a, uint32_t b, bool high) {
    return high ? (a >> 16) | (b & 0xFFFF0000u) : (a & 0xFFFFu) | (b << 16);
}
__device__ __forceinline__ uint32_t word_of(const uint4& v, int w) {
    return w == 0 ? v.x : (w == 1 ? v.y : (w == 2 ? v.z : v.w));
}

__global__ __launch_bounds__(256) void k_transpose_window(const bf16_t* __restrict__ in, int C, int mode,
                                                         const int32_t* __restrict__ row_map, int K,
                                                         const int32_t* __restrict__ offsets,
                                                         const int32_t* __restrict__ koff, int E,
                                                         bf16_t* __restrict__ out) {
    const int q0 = blockIdx.x * TT;
    const int total = koff[E];
    if (q0 >= total) return;  // uniform per workgroup
    int lo = 0, hi = E - 1;   // last expert with koff[e] <= q0
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (koff[mid] <= q0) lo = mid;
        else hi = mid - 1;
    }
    const int base = offsets[lo], count = offsets[lo + 1] - base;
    const int i0 = q0 - koff[lo];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int rg = lane & 7, cg = lane >> 3;
    // Source rows of the lane's 8 positions (-1: padding, zeros).
    int srow[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int i = i0 + rg * 8 + j;
        int v = -1;
        if (i < count) {
            const int p = base + i;
            v = mode == SRC_SORTED ? p : (mode == SRC_SLOT ? row_map[p] : row_map[p] / K);
        }
        srow[j] = v;
    }
    bf16_t* const ob = out + (size_t)(q0 / TT) * C * TT + rg * 8;
    for (int c = wave * 64 + cg * 8; c < C; c += 256) {
        // Padding positions load row 0 (T >= 1, so it exists) and keep zeros:
        // no branch, so all 8 loads are in flight together.
        uint4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint4 t = *reinterpret_cast<const uint4*>(in + (size_t)(srow[j] < 0 ? 0 : srow[j]) * C + c);
            v[j] = srow[j] >= 0 ? t : make_uint4(0u, 0u, 0u, 0u);
        }
        // Column k of the block: element k of each row, rows in pairs per word.
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int w = k >> 1;
            const bool high = k & 1;
            uint4 o;
            o.x = pair16(word_of(v[0], w), word_of(v[1], w), high);
            o.y = pair16(word_of(v[2], w), word_of(v[3], w), high);
            o.z = pair16(word_of(v[4], w), word_of(v[5], w), high);
            o.w = pair16(word_of(v[6], w), word_of(v[7], w), high);
            store16_nt(ob + (size_t)(c + k) * TT, o);
        }
    }
}

// out[g][r][:] = in[g][src(r)][:] for the 2h stacked rows of a [G][2 ld][C]
// fp32 tensor (src(r) = r for r < h, ld + r - h after): the padded weight
// gradient of stacked gate and up rows back to the unpadded layout.
__global__ __launch_bounds__(256) void k_compact_rows(const float* __restrict__ in, int G, int h, int ld, int C,
                                                     float* __restrict__ out) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t q = C / 4;
    if (i >= (size_t)G * 2 * h * q) return;
    const size_t row = i / q, g = row / (2 * h);
    const int r = (int)(row - g * 2 * h), c = (int)(i % q) * 4;
    const int sr = r < h ? r : ld + r - h;
    *reinterpret_cast<float4*>(out + row * C + c) =
        *reinterpret_cast<const float4*>(in + (g * 2 * ld + sr) * (size_t)C + c);
}

// Zero the K window of every expert with no rows (its two slabs of the
// slab-major operand [ld / 64][C][64]); one workgroup per expert.
__global__ __launch_bounds__(256) void k_zero_empty_windows(bf16_t* __restrict__ out, int C,
                                                           const int32_t* __restrict__ offsets,
                                                           const int32_t* __restrict__ koff) {
    const int e = blockIdx.x;
    if (offsets[e + 1] != offsets[e]) return;
    uint4* p = reinterpret_cast<uint4*>(out + (size_t)koff[e] * C);
    const size_t n = (size_t)(koff[e + 1] - koff[e]) * C / 8;
    for (size_t i = threadIdx.x; i < n; i += blockDim.x) p[i] = make_uint4(0u, 0u, 0u, 0u);
}

__device__ __forceinline__ uint32_t pack2_bf16_rne(float lo, float hi) {
    uint32_t a = __float_as_uint(lo), b = __float_as_uint(hi);
    a += 0x7fffu + ((a >> 16) & 1u);
    b += 0x7fffu + ((b >> 16) & 1u);
    return (a >> 16) | (b & 0xffff0000u);
}

// dx[t, :] = bf16(sum_j dxs[t K + j, :]) in slot order (fp32 sums), 4 columns
// per thread.
__global__ __launch_bounds__(256) void k_slot_sum(const float* __restrict__ dxs, int T, int K, int d,
                                                 bf16_t* __restrict__ dx) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int q = d / 4;
    if (i >= (size_t)T * q) return;
    const size_t t = i / q;
    const int c = (int)(i % q) * 4;
    float4 acc = *reinterpret_cast<const float4*>(dxs + (t * K) * d + c);
    for (int j = 1; j < K; ++j) {
        const float4 v = *reinterpret_cast<const float4*>(dxs + (t * K + j) * d + c);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    uint2 o;
    o.x = pack2_bf16_rne(acc.x, acc.y);
    o.y = pack2_bf16_rne(acc.z, acc.w);
    *reinterpret_cast<uint2*>(dx + t * d + c) = o;
}

}  // namespace

hipError_t launch_transpose_w(const void* in, int G, int R, int C, void* out, hipStream_t s) {
    hipLaunchKernelGGL(k_transpose_w, dim3(R / TT, C / TT, G), dim3(256), 0, s, static_cast<const bf16_t*>(in), R, R,
                       C, 0, 0, static_cast<bf16_t*>(out));
    return hipGetLastError();
}

hipError_t launch_transpose_w13(const void* in, int G, int h, int ld, int C, void* out, hipStream_t s) {
    hipLaunchKernelGGL(k_transpose_w, dim3(2 * ld / TT, C / TT, G), dim3(256), 0, s, static_cast<const bf16_t*>(in),
                       2 * h, 2 * ld, C, h, ld, static_cast<bf16_t*>(out));
    return hipGetLastError();
}

hipError_t launch_compact_rows(const float* in, int G, int h, int ld, int C, float* out, hipStream_t s) {
    const size_t n = (size_t)G * 2 * h * (C / 4);
    hipLaunchKernelGGL(k_compact_rows, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, in, G, h, ld, C, out);
    return hipGetLastError();
}

hipError_t launch_wgrad_plan(const int32_t* offsets, int E, int32_t* koff, TileDesc* items, TileDesc* rlist,
                             int32_t* wcount, hipStream_t s) {
    hipLaunchKernelGGL(k_wgrad_plan, dim3(1), dim3(1024), 0, s, offsets, E, koff, items, rlist, wcount);
    return hipGetLastError();
}

hipError_t launch_wgrad_reduce(const float* partials, const TileDesc* rlist, const int32_t* wcount, int E,
                               size_t mn, float* out, hipStream_t s) {
    const size_t blocks = (mn / 4 + 255) / 256;
    hipLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)blocks, (unsigned)(E < 8 ? E : 8)), dim3(256), 0, s, partials,
                       rlist, wcount, mn, out);
    return hipGetLastError();
}

hipError_t launch_transpose_window(const void* in, int C, int mode, const int32_t* row_map, int K,
                                   const int32_t* offsets, const int32_t* koff, int E, void* out, int ld,
                                   hipStream_t s) {
    hipLaunchKernelGGL(k_transpose_window, dim3(ld / TT), dim3(256), 0, s, static_cast<const bf16_t*>(in), C, mode,
                       row_map, K, offsets, koff, E, static_cast<bf16_t*>(out));
    return hipGetLastError();
}

hipError_t launch_zero_empty_windows(void* out, int C, const int32_t* offsets, const int32_t* koff, int E,
                                     hipStream_t s) {
    hipLaunchKernelGGL(k_zero_empty_windows, dim3(E), dim3(256), 0, s, static_cast<bf16_t*>(out), C, offsets, koff);
    return hipGetLastError();
}

hipError_t launch_slot_sum(const float* dxs, int T, int K, int d, void* dx, hipStream_t s) {
    const size_t n = (size_t)T * (d / 4);
    hipLaunchKernelGGL(k_slot_sum, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dxs, T, K, d,
                       static_cast<bf16_t*>(dx));
    return hipGetLastError();
}

}  // namespace moe
