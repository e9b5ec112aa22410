// Grouping of slots by expert (paper App. "MoE Kernel", Algorithm 1 Phase 1:
// sort the flattened expert ids, bincount, cumulative sum) as three
// deterministic passes with no global atomics:
//   1. k_hist     per-chunk expert histograms (LDS atomics; order-free)
//   2. k_scan     per-expert prefix over chunks, exclusive scan over experts
//                 -> counts, offsets and each chunk's base position per expert
//   3. k_scatter  stable scatter: every wave walks its part of the chunk in
//                 slot order and ranks equal experts inside a round with
//                 ballots, so slots of one expert keep ascending slot order.
// Plus k_build_tiles, which cuts every expert's segment into M-tiles for the
// grouped GEMMs (the device-side tile list that replaces a host round trip),
// and k_permute_small, all of it in one block for small batches (up to 16384
// slots).
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kScanMax = 16384;  // chunk-histogram entries the scan keeps in LDS

// Exclusive prefix sum over a 1024-thread block; returns the exclusive value
// and writes the block total to *total. `tmp` holds >= 16 ints of LDS.
__device__ int block_exclusive_scan_1024(int v, int* tmp, int* total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(incl, off);
        if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) tmp[wave] = incl;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int w = 0; w < (int)(blockDim.x / kWave); ++w) {
            const int c = tmp[w];
            tmp[w] = run;
            run += c;
        }
        tmp[16] = run;
    }
    __syncthreads();
    const int excl = incl - v + tmp[wave];
    *total = tmp[16];
    __syncthreads();
    return excl;
}

__global__ __launch_bounds__(1024) void k_hist(const int32_t* __restrict__ idx, int64_t n_slots,
                                              int E, int64_t chunk, int32_t* __restrict__ blockhist) {
    __shared__ int h[kMaxE];
    for (int e = threadIdx.x; e < E; e += blockDim.x) h[e] = 0;
    __syncthreads();
    const int64_t start = (int64_t)blockIdx.x * chunk;
    const int64_t end = min(n_slots, start + chunk);
    for (int64_t n = start + threadIdx.x; n < end; n += blockDim.x) {
        const int e = idx[n];
        if ((unsigned)e < (unsigned)E) atomicAdd(&h[e], 1);  // ids outside [0, E) are dropped
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) blockhist[(size_t)blockIdx.x * E + e] = h[e];
}

// M-tiles of height bm over every expert's segment, in expert order, by one
// 1024-thread block. off: the E + 1 segment offsets (global memory or LDS);
// start: kMaxE + 1 ints of LDS; tmp: 32 ints of LDS.
__device__ void build_tiles_block(int E, int bm, int max_tiles, const int32_t* off, TileDesc* __restrict__ tiles,
                                  int32_t* __restrict__ n_tiles, int* start, int* tmp) {
    const int e = threadIdx.x;
    int nt = 0;
    if (e < E) {
        const int cnt = off[e + 1] - off[e];
        nt = cnt > 0 ? (cnt + bm - 1) / bm : 0;
    }
    int total;
    const int excl = block_exclusive_scan_1024(nt, tmp, &total);
    // Offsets from a caller could describe more tiles than the table holds.
    total = min(total, max_tiles);
    if (e < E) start[e] = excl;
    if (e == 0) start[E] = total;
    __syncthreads();
    for (int q = threadIdx.x; q < total; q += blockDim.x) {
        int lo = 0, hi = E;  // largest expert with start[expert] <= q
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (start[mid] <= q) lo = mid; else hi = mid;
        }
        const int i = q - start[lo];
        const int seg0 = off[lo];
        const int cnt = off[lo + 1] - seg0;
        TileDesc t;
        t.e = lo;
        t.row0 = seg0 + i * bm;
        t.rows = min(bm, cnt - i * bm);
        t.pad = 0;
        tiles[q] = t;
    }
    if (threadIdx.x == 0) *n_tiles = total;
}

// One 1024-thread block. blockhist [nb][E] in: chunk histograms; out: the
// position where chunk b's first slot of expert e goes. With a tile table
// (tiles != nullptr) it also cuts the segments into M-tiles of bm rows, as
// k_build_tiles does, saving that launch.
__global__ __launch_bounds__(1024) void k_scan(int32_t* __restrict__ blockhist, int nb, int E,
                                              int32_t* __restrict__ counts,
                                              int32_t* __restrict__ offsets, int bm, int max_tiles,
                                              TileDesc* __restrict__ tiles, int32_t* __restrict__ n_tiles) {
    __shared__ int buf[kScanMax];
    __shared__ int segtot[1024];
    __shared__ int tmp[32];
    __shared__ int offl[kMaxE + 1];
    __shared__ int start[kMaxE + 1];
    const int tid = threadIdx.x;
    const int n = nb * E;
    {  // 16-byte loads, four per thread in flight (n <= kScanMax = 16 x 1024)
        const int n4 = n / 4;
        const int4* bh4 = reinterpret_cast<const int4*>(blockhist);
        const int nt = blockDim.x;
        for (int i = tid; i < n4; i += 4 * nt) {
            int4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (i + u * nt < n4) v[u] = bh4[i + u * nt];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (i + u * nt < n4) {
                    const int j = 4 * (i + u * nt);
                    buf[j] = v[u].x;
                    buf[j + 1] = v[u].y;
                    buf[j + 2] = v[u].z;
                    buf[j + 3] = v[u].w;
                }
        }
        for (int i = 4 * n4 + tid; i < n; i += nt) buf[i] = blockhist[i];
    }
    // Each expert's column of chunk counts is cut into S segments of
    // consecutive chunks, thread (segment g, expert e) = tid g E + e.
    const int S = max(1, min(nb, (int)blockDim.x / E));
    const int per = (nb + S - 1) / S;
    const int e = tid % E, g = tid / E;
    const bool act = g < S;
    const int b0 = min(nb, g * per), b1 = min(nb, b0 + per);
    __syncthreads();
    int seg = 0;
    if (act)
        for (int b = b0; b < b1; ++b) seg += buf[b * E + e];
    if (act) segtot[g * E + e] = seg;
    __syncthreads();
    // The segment's start within its expert, then the exclusive prefix of
    // every chunk of the segment; thread (0, e) also forms the expert's total.
    int cnt = 0;
    if (act) {
        int run = 0;
        for (int q = 0; q < g; ++q) run += segtot[q * E + e];
        for (int b = b0; b < b1; ++b) {
            const int v = buf[b * E + e];
            buf[b * E + e] = run;
            run += v;
        }
        if (g == 0)
            for (int q = 0; q < S; ++q) cnt += segtot[q * E + e];
    }
    int total;
    const int excl = block_exclusive_scan_1024(tid < E ? cnt : 0, tmp, &total);
    if (tid < E) {
        counts[tid] = cnt;
        offsets[tid] = excl;
        offl[tid] = excl;
    }
    if (tid == 0) {
        offsets[E] = total;
        offl[E] = total;
    }
    __syncthreads();
    for (int i = tid; i < n; i += blockDim.x) blockhist[i] = buf[i] + offl[i % E];
    if (tiles) build_tiles_block(E, bm, max_tiles, offl, tiles, n_tiles, start, tmp);
}

// Lanes of the wave whose `key` equals this lane's (only lanes with `valid`
// set take part), from one ballot per key bit.
__device__ __forceinline__ uint64_t match_peers(int key, bool valid, int nbits) {
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = (key >> b) & 1;
        const uint64_t ones = __ballot(valid && bit);
        peers &= bit ? ones : ~ones;
    }
    return peers;
}

__global__ __launch_bounds__(1024) void k_scatter(const int32_t* __restrict__ idx, int64_t n_slots,
                                                  int E, int nbits, int64_t chunk,
                                                  const int32_t* __restrict__ blockbase,
                                                  int32_t* __restrict__ sorted_slots) {
    constexpr int kWaves = 16;  // each wave ranks one sixteenth of the chunk, in slot order
    __shared__ int base[kWaves][kMaxE];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t start = (int64_t)blockIdx.x * chunk;
    const int64_t end = min(n_slots, start + chunk);
    const int64_t sub = (chunk + kWaves - 1) / kWaves;
    const int64_t ws = min(end, start + wave * sub);
    const int64_t we = min(end, ws + sub);

    for (int i = threadIdx.x; i < kWaves * kMaxE; i += blockDim.x) (&base[0][0])[i] = 0;
    __syncthreads();
    for (int64_t n = ws + lane; n < we; n += kWave) {
        const int e = idx[n];
        if ((unsigned)e < (unsigned)E) atomicAdd(&base[wave][e], 1);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        int run = blockbase[(size_t)blockIdx.x * E + e];
        for (int w = 0; w < kWaves; ++w) {
            const int c = base[w][e];
            base[w][e] = run;
            run += c;
        }
    }
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int64_t r0 = ws; r0 < we; r0 += kWave) {
        const int64_t n = r0 + lane;
        const int e_raw = n < we ? idx[n] : -1;
        const bool valid = (unsigned)e_raw < (unsigned)E;
        const int e = valid ? e_raw : 0;
        const uint64_t peers = match_peers(e, valid, nbits);
        if (valid) {
            const int rank = __popcll(peers & lt);
            const int pos = base[wave][e] + rank;
            sorted_slots[pos] = (int32_t)n;
            if (rank == 0) base[wave][e] = pos + __popcll(peers);
        }
    }
}

// Small batches (up to kPermuteOneBlock slots): the three passes in one
// 1024-thread block, so the permute is one launch. Each of the 16 waves takes
// a sixteenth of the slots in slot order, all of its indices loaded at once
// (up to 16 per lane, kept in registers): its expert histogram (LDS atomics),
// then per expert the waves' bases in wave order, the counts, the exclusive
// scan over experts (offsets), the stable scatter as in k_scatter, and the
// tile table as in k_scan.
constexpr int kPermuteRounds = 16;  // 64-slot rounds per wave
constexpr int64_t kPermuteOneBlock = 16 * kWave * kPermuteRounds;

__global__ __launch_bounds__(1024) void k_permute_small(const int32_t* __restrict__ idx, int64_t n_slots, int E,
                                                        int nbits, int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ offsets,
                                                        int32_t* __restrict__ sorted_slots, int bm, int max_tiles,
                                                        TileDesc* __restrict__ tiles, int32_t* __restrict__ n_tiles) {
    constexpr int kWaves = 16;
    __shared__ int base[kWaves][kMaxE];
    __shared__ int tmp[32];
    __shared__ int offl[kMaxE + 1];
    __shared__ int start[kMaxE + 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int sub = (int)((n_slots + kWaves - 1) / kWaves);  // <= kWave * kPermuteRounds
    const int ws = (int)min(n_slots, (int64_t)wave * sub);
    const int we = (int)min(n_slots, (int64_t)ws + sub);

    // Expert of slot ws + 64 r + lane, or -1 past the wave's range. The loads
    // are unconditional (past the range they re-read the last slot), so all
    // sixteen are in flight together.
    int ev[kPermuteRounds];
#pragma unroll
    for (int r = 0; r < kPermuteRounds; ++r) {
        const int n = ws + kWave * r + lane;
        ev[r] = idx[n < n_slots ? n : n_slots - 1];
    }
#pragma unroll
    for (int r = 0; r < kPermuteRounds; ++r)
        if (ws + kWave * r + lane >= we) ev[r] = -1;
    for (int i = threadIdx.x; i < kWaves * kMaxE; i += blockDim.x) (&base[0][0])[i] = 0;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPermuteRounds; ++r)
        if ((unsigned)ev[r] < (unsigned)E) atomicAdd(&base[wave][ev[r]], 1);  // ids outside [0, E) are dropped
    __syncthreads();
    // Per expert: each wave's start within the expert, and the expert's count.
    int cnt = 0;
    if ((int)threadIdx.x < E) {
        const int e = threadIdx.x;
        for (int w = 0; w < kWaves; ++w) {
            const int c = base[w][e];
            base[w][e] = cnt;
            cnt += c;
        }
    }
    int total;
    const int excl = block_exclusive_scan_1024((int)threadIdx.x < E ? cnt : 0, tmp, &total);
    if ((int)threadIdx.x < E) {
        counts[threadIdx.x] = cnt;
        offsets[threadIdx.x] = excl;
        offl[threadIdx.x] = excl;
    }
    if (threadIdx.x == 0) {
        offsets[E] = total;
        offl[E] = total;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kWaves * E; i += blockDim.x) base[i / E][i % E] += offl[i % E];
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
#pragma unroll
    for (int r = 0; r < kPermuteRounds; ++r) {
        if (ws + kWave * r >= we) break;  // uniform: the wave's rounds are done
        const bool valid = (unsigned)ev[r] < (unsigned)E;
        const int e = valid ? ev[r] : 0;
        const uint64_t peers = match_peers(e, valid, nbits);
        if (valid) {
            const int rank = __popcll(peers & lt);
            const int pos = base[wave][e] + rank;
            sorted_slots[pos] = (int32_t)(ws + kWave * r + lane);
            if (rank == 0) base[wave][e] = pos + __popcll(peers);
        }
    }
    if (tiles) build_tiles_block(E, bm, max_tiles, offl, tiles, n_tiles, start, tmp);
}

// M-tiles of height bm over every expert's segment, in expert order.
__global__ __launch_bounds__(1024) void k_build_tiles(int E, int bm, int max_tiles,
                                                     const int32_t* __restrict__ offsets,
                                                     TileDesc* __restrict__ tiles,
                                                     int32_t* __restrict__ n_tiles) {
    __shared__ int start[kMaxE + 1];
    __shared__ int tmp[32];
    build_tiles_block(E, bm, max_tiles, offsets, tiles, n_tiles, start, tmp);
}

}  // namespace

hipError_t launch_permute(const moe_desc_t& d, const int32_t* topk_idx, int32_t* counts,
                          int32_t* offsets, int32_t* sorted_slots, int32_t* blockhist,
                          int32_t n_blocks, hipStream_t s, int32_t bm, int32_t max_tiles, TileDesc* tiles,
                          int32_t* n_tiles) {
    const int64_t n_slots = (int64_t)d.T * d.K;
    const int64_t chunk = (n_slots + n_blocks - 1) / n_blocks;
    int nbits = 0;
    while ((1 << nbits) < d.E) ++nbits;
    if (n_slots <= kPermuteOneBlock) {
        hipLaunchKernelGGL(k_permute_small, dim3(1), dim3(1024), 0, s, topk_idx, n_slots, d.E, nbits, counts, offsets,
                           sorted_slots, bm, max_tiles, tiles, n_tiles);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_hist, dim3(n_blocks), dim3(1024), 0, s, topk_idx, n_slots, d.E, chunk, blockhist);
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, blockhist, n_blocks, d.E, counts, offsets, bm, max_tiles,
                       tiles, n_tiles);
    hipLaunchKernelGGL(k_scatter, dim3(n_blocks), dim3(1024), 0, s, topk_idx, n_slots, d.E, nbits, chunk,
                       blockhist, sorted_slots);
    return hipGetLastError();
}

hipError_t launch_build_tiles(int32_t E, int32_t bm, int32_t max_tiles, const int32_t* offsets,
                              TileDesc* tiles, int32_t* n_tiles, hipStream_t s) {
    hipLaunchKernelGGL(k_build_tiles, dim3(1), dim3(1024), 0, s, E, bm, max_tiles, offsets, tiles, n_tiles);
    return hipGetLastError();
}

int32_t permute_blocks(int64_t n_slots, int32_t E) {
    int64_t nb = (n_slots + 1023) / 1024;
    const int64_t cap = kScanMax / E;
    if (nb > cap) nb = cap;
    if (nb < 1) nb = 1;
    return (int32_t)nb;
}

}  // namespace moe
