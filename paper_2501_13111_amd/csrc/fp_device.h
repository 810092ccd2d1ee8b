// Device helpers shared by the gfx950 kernels of the fingerprint forward pass.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp_internal.h"

namespace fpk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- rounding
// float -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }
__device__ __forceinline__ float bfround(float f) { return bf2f(f2bf(f)); }

// Two floats -> a packed pair by the hardware conversions (round to nearest even),
// for MFMA operands that only need to be within tolerance (probabilities, queries).
__device__ __forceinline__ uint32_t pack_bf16_hw(float lo, float hi) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t pack_f16_hw(float lo, float hi) {
    const f16x2 v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t f2h(float f) {
    _Float16 h = (_Float16)f;                      // v_cvt_f16_f32, round to nearest even
    return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float h2f(uint16_t b) {
    return (float)__builtin_bit_cast(_Float16, b);
}

// Activation formats of a GEMM's A operand: bf16 (bf16 weights) or fp16 (quantised
// weights).  Values are always bf16-rounded first; the fp16 copy of a bf16 value is
// exact in fp16's normal range.
__device__ __forceinline__ uint16_t act_store(float bf16_valued, int fmt) {
    return fmt == ACT_BF16 ? f2bf(bf16_valued) : f2h(bf16_valued);
}
__device__ __forceinline__ float act_load(uint16_t bits, int fmt) {
    return fmt == ACT_BF16 ? bf2f(bits) : h2f(bits);
}

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
    return v;
}

// block-wide sum for blockDim.x a multiple of 64 (<= 1024); `red` holds >= 16 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
    for (int i = 0; i < nw; ++i) t += red[i];
    return t;
}
__device__ __forceinline__ float block_max(float v, float* red) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_max(v);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float t = red[0];
    for (int i = 1; i < nw; ++i) t = fmaxf(t, red[i]);
    return t;
}

// ---------------------------------------------------------------- MFMA
__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}
template <int FMT>
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
    if constexpr (FMT == ACT_BF16) return mfma_bf16(a, b, c);
    else return mfma_f16(a, b, c);
}

// 32x32x16 MFMA (twice the throughput of 16x16x32 on this part): lane l supplies row
// (l % 32) of A and column (l % 32) of B, each with the 8 consecutive k from 8 (l / 32);
// accumulator element e of lane l is C[8 (e / 4) + 4 (l / 32) + e % 4][l % 32].
typedef float f32x16 __attribute__((ext_vector_type(16)));
template <int FMT>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
    if constexpr (FMT == ACT_BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------- dequantisation
// int8 codes (4 per dword) -> exact fp16 values, two per dword.
// u = b ^ 0x80 in [0, 255]; fp16 bits 0x6400 | u encode 1024 + u = 1152 + b; subtracting
// 1152 is exact.
__device__ __forceinline__ u32x2 i8x4_to_f16x4(uint32_t w) {
    const uint32_t u = w ^ 0x80808080u;
    const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, u, 0x04010400u);  // bytes 0,1
    const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, u, 0x04030402u);  // bytes 2,3
    const f16x2 bias = {(_Float16)1152.0f, (_Float16)1152.0f};
    f16x2 a = __builtin_bit_cast(f16x2, lo) - bias;
    f16x2 b = __builtin_bit_cast(f16x2, hi) - bias;
    u32x2 r;
    r.x = __builtin_bit_cast(uint32_t, a);
    r.y = __builtin_bit_cast(uint32_t, b);
    return r;
}

// int4 word in the device nibble order (nibble p holds column offset 2p for p < 4 and
// 2(p-4)+1 for p >= 4) -> 8 exact fp16 values (q - z) in column order.
// fp16 bits 0x6400 | q encode 1024 + q; subtracting 1024 + z is exact.
// (a & m) | o in one VOP3 instruction (m in an SGPR, o in a VGPR: one scalar operand per
// VOP3 instruction; the compiler splits the pattern into two instructions otherwise).
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t m, uint32_t o) {
    uint32_t d;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(m), "v"(o));
    return d;
}

__device__ __forceinline__ u32x4 i4x8_to_f16x8(uint32_t w, f16x2 bias) {
    u32x4 r;
    const uint32_t p0 = and_or(w, 0x000F000Fu, 0x64006400u);
    const uint32_t p1 = and_or(w >> 4, 0x000F000Fu, 0x64006400u);
    const uint32_t p2 = and_or(w >> 8, 0x000F000Fu, 0x64006400u);
    const uint32_t p3 = and_or(w >> 12, 0x000F000Fu, 0x64006400u);
    r.x = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p0) - bias);
    r.y = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p1) - bias);
    r.z = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p2) - bias);
    r.w = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p3) - bias);
    return r;
}

// Packed fp16 multiply of a dword holding two fp16 values.  Takes the dword by value:
// bit-casting an element of an ext_vector in place does not read that element.
__device__ __forceinline__ uint32_t mul_h2(uint32_t v, f16x2 s) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, v) * s);
}

// Sum of ks partial sums p[0], p[stride], ..., added in increasing order; the loads
// are issued in batches of eight (the partials were written by the previous kernel,
// so each batch costs one memory round trip).
__device__ __forceinline__ float sum_parts(const float* __restrict__ p, int ks, int64_t stride) {
    float acc = 0.f;
    for (int s = 0; s < ks; s += 8) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (s + i < ks) ? p[(s + i) * stride] : 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc += v[i];
    }
    return acc;
}

// Split-K sums of NS columns (p[c][s * stride] over s < ks, in split order, as sum_parts
// adds them), with the loads of eight splits of every column in flight together: one
// memory round trip per eight splits instead of one per column.  Columns with p[c] null
// give 0 and load nothing.
template <int NS>
__device__ __forceinline__ void sum_parts_cols(const float* const (&p)[NS], int ks, int64_t stride, float (&out)[NS]) {
#pragma unroll
    for (int c = 0; c < NS; ++c) out[c] = 0.f;
    for (int s = 0; s < ks; s += 8) {
        float v[NS][8];
#pragma unroll
        for (int c = 0; c < NS; ++c)
#pragma unroll
            for (int i = 0; i < 8; ++i) v[c][i] = (p[c] != nullptr && s + i < ks) ? p[c][(s + i) * stride] : 0.f;
#pragma unroll
        for (int c = 0; c < NS; ++c)
#pragma unroll
            for (int i = 0; i < 8; ++i) out[c] += v[c][i];
    }
}

// Raw buffer resource over [base, base + bytes), bytes < 2^32.  A load at or past the
// end returns zeros without a memory access, so a pipelined loop can issue the same
// loads on every trip (exact wait counts) and pay nothing for the trips past its range.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// 16-byte non-temporal load at byte offset off (zeros if off >= the resource's size)
__device__ __forceinline__ u32x4 buf_load_nt(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}
// LDS pointer type of the buffer-to-LDS copy builtin
typedef __attribute__((address_space(3))) void lvoid_t;
constexpr uint32_t BUF_OOB = 0xFFFFFFF0u;   // an offset past the end of every resource

// off if live, else BUF_OOB.  The mask passes through an empty asm statement, so the
// compiler cannot turn the choice into a branch around the load: on a uniform
// condition it otherwise does, and the wait counts it inserts at the join drain every
// load in flight.
__device__ __forceinline__ uint32_t off_or_oob(bool live, uint32_t off) {
    uint32_t m = live ? 0u : 0xFFFFFFFFu;
    asm volatile("" : "+v"(m));
    return off + ((BUF_OOB - off) & m);
}
// the same for a condition that is uniform across the wave (the mask stays scalar)
__device__ __forceinline__ uint32_t off_or_oob_uniform(bool live, uint32_t off) {
    uint32_t m = __builtin_amdgcn_readfirstlane(live ? 0u : 0xFFFFFFFFu);
    asm volatile("" : "+s"(m));
    return off + ((BUF_OOB - off) & m);
}

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

}  // namespace fpk
