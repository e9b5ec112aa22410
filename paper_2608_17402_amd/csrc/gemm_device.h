// Device helpers of the bf16 GEMM kernels (gemm.hip): vector types, the bf16
// rounding and activation functions of the expert MLPs, global -> LDS copies,
// LDS fragment reads, explicit waits and the epilogue's memory operations.
#pragma once

#include "moe_internal.h"

#include <type_traits>
#include <utility>

namespace moe {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

// GELU for the bf16 path: GELU(x) = x Phi(x) with the normal CDF Phi taken
// as Sigmoid(s(x)), s(x) = x (a0 + a1 x^2 + a2 x^4) evaluated on x clamped
// to [-8, 8]. The coefficients minimise the largest absolute error of the
// GELU over the real line (2.6e-5 in fp32, against a bf16 rounding step of
// 2^-9 relative for the stored activation); past the clamp the sigmoid is
// within 1e-11 of 0 or 1. With the hardware exp2 and reciprocal: 7 VALU
// operations and 2 transcendentals per element. The folded constants are
// -a_k log2(e), so that exp2 of x (b0 + b1 x^2 + b2 x^4) is exp(-s(x)).
constexpr float kGeluA0 = 1.59501576f, kGeluA1 = 0.0740112886f, kGeluA2 = -7.03033584e-4f;
constexpr float kGeluB0 = -2.30112123f, kGeluB1 = -0.106775723f, kGeluB2 = 1.01426302e-3f;
__device__ __forceinline__ float gelu_sig(float x) {
    const float xc = __builtin_amdgcn_fmed3f(x, -8.0f, 8.0f);
    const float x2 = xc * xc;
    const float t = xc * fmaf(fmaf(kGeluB2, x2, kGeluB1), x2, kGeluB0);
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}

// SiLU(v) = v / (1 + exp(-v)) from the hardware exp2 and reciprocal; for
// very negative v, exp2 overflows to +inf and the reciprocal to 0, the limit.
__device__ __forceinline__ float silu_as(float v) {
    return v * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v * -1.44269504f));
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Four fp32 values -> four bf16 (round to nearest even) packed in 8 bytes.
__device__ __forceinline__ uint2 pack4_bf16(float a, float b, float c, float d) {
    const bf16x2_t lo = __builtin_convertvector((f32x2_t){a, b}, bf16x2_t);
    const bf16x2_t hi = __builtin_convertvector((f32x2_t){c, d}, bf16x2_t);
    uint2 r;
    r.x = __builtin_bit_cast(uint32_t, lo);
    r.y = __builtin_bit_cast(uint32_t, hi);
    return r;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_lgkmcnt() {
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Workgroup barrier without the memory fence of __syncthreads (which would
// wait for every copy still in flight, including slabs prefetched ahead).
// Each wave waits for its own copies of the current slab with vmcnt before
// arriving, and every LDS read of the slab before has been consumed by MFMAs,
// so the bare barrier is enough.
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

// Buffer resource over `bytes` bytes at `base` (raw buffer, gfx9 format word).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from (rsrc, voffset + soffset) straight into LDS at
// lds + 16 * lane; lds is the same for the whole wave.
__device__ __forceinline__ void copy16_to_lds(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                              uint8_t* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, (int)voff,
                                             (int)soff, 0, 0);
}
// The same copy with the non-temporal hint: the lines are streamed through
// the caches and evicted first, so data read once (the expert weights of the
// weight-read-bound small batches) does not push out rows that other tiles
// read again (the gathered token rows, the activation rows).
__device__ __forceinline__ void copy16_to_lds_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                                 uint8_t* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, (int)voff,
                                             (int)soff, 0, 2);
}

__device__ __forceinline__ uint32_t lds_address(const uint8_t* p) {
    return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) uint8_t*)p);
}

// One 16-byte fragment from LDS. Issued as inline assembly so the compiler
// does not pair it with the in-flight copies into other stages (it cannot
// tell them apart and would wait for all of them); completion is awaited
// explicitly with wait_lgkmcnt0 and pinned with tie().
template <int OFF>
__device__ __forceinline__ bf16x8_t lds_read16(uint32_t addr) {
    bf16x8_t r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
__device__ __forceinline__ void tie(bf16x8_t& v) { asm volatile("" : "+v"(v)); }

// Lanes of one wave handing data to each other through LDS: orders the
// writes before the reads (and the reads before the next writes) for every
// lane. Without it the compiler may treat the exchange as a data race and
// move a lane's reads away from the other lanes' writes.
__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Memory operations of the persistent kernel's epilogue, as inline assembly.
// The compiler's wait bookkeeping does not see them. Loads and stores can
// retire out of order relative to each other on this target, so a store the
// compiler knew about would turn each later wait for a load result into a full
// drain of the slab copies in flight. The kernel waits for them explicitly.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
// (The s_nop is the wait state a store of more than 8 bytes needs before its
// data registers may be overwritten; the compiler cannot see that here.)
// Output stores carry the non-temporal hint: results are not read again by
// this kernel, and without it their lines stay in L2 and push out operand
// slabs that neighbouring tiles still read (the backward's fp32 outputs
// especially; 3 % of the backward, 1 % of the forward).
__device__ __forceinline__ void store16_asm(void* p, u32x4_t v) {
    asm volatile("global_store_dwordx4 %0, %1, off nt\n\ts_nop 0" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store4_asm(void* p, uint32_t v) {
    asm volatile("global_store_dword %0, %1, off" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_write8_asm(uint32_t addr, u32x2_t v) {
    asm volatile("ds_write_b64 %0, %1" ::"v"(addr), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_write16_asm(uint32_t addr, u32x4_t v) {
    asm volatile("ds_write_b128 %0, %1" ::"v"(addr), "v"(v) : "memory");
}
__device__ __forceinline__ u32x4_t lds_read16u_asm(uint32_t addr) {
    u32x4_t r;
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr));
    return r;
}
__device__ __forceinline__ void tie(u32x4_t& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ void lds_read_u16_asm(uint32_t& r, uint32_t addr) {
    asm volatile("ds_read_u16 %0, %1" : "=v"(r) : "v"(addr));
}
__device__ __forceinline__ void tie(uint32_t& v) { asm volatile("" : "+v"(v)); }
// Transposing 8-byte LDS read (ds_read_b64_tr_b16, CDNA4). Within each group
// of 16 lanes, lane r names 4 consecutive 16-bit values M[r][0..3]; lane i
// receives M[i / 4 + 4 j][i % 4] as its 16-bit element j (j = 0..3). With
// lane r pointing at row r / 4 and columns 4 (r % 4) .. of a 4 x 16 block,
// lane i gets column i of the 4 rows, row j in element j.
__device__ __forceinline__ void lds_read_tr8_asm(u32x2_t& r, uint32_t addr) {
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(addr));
}
__device__ __forceinline__ void tie(u32x2_t& v) { asm volatile("" : "+v"(v)); }
// One accumulator moved to a vector register at this point of the program
// (volatile: not hoisted, so only one staged block's values are live at once).
__device__ __forceinline__ float acc_read(float x) {
    float v;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(x));
    return v;
}

// Compile-time loop: f(std::integral_constant<int, 0>{}) ... f(<N - 1>).
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

}  // namespace
}  // namespace moe
