// Weight synthesis and quantisation on the device.
//
// The fingerprint Generator (paper Sec. 5.1) reads a checkpoint; these kernels
// synthesise its stand-in from a seed with a counter-based SplitMix64 hash
// (Steele, Lea & Flood, OOPSLA 2014) and apply the compression menu of Sec. 3.2:
// int8 symmetric per output row and int4 asymmetric per group of 128 inputs,
// both with fp16 scales.  Quantiser arithmetic uses correctly rounded fp32
// division, round-half-to-even and no contraction, so codes are a pure function
// of the bf16 weights.
#include <algorithm>

#include "fp_device.h"
#include "fp_internal.h"

#pragma clang fp contract(off)

namespace fpk {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z ^= z >> 30; z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27; z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

#define FP_GAMMA 0x9E3779B97F4A7C15ull

__global__ void fill_bf16_kernel(uint16_t* __restrict__ dst, int64_t n, uint64_t key, float mean,
                                 float sigma) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const uint64_t base = key + FP_GAMMA * (3ull * (uint64_t)i + 1ull);
        uint32_t s = 0;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            const uint64_t w = mix64(base + FP_GAMMA * (uint64_t)c);
            s += (uint32_t)(w & 0xFFFFu) + (uint32_t)((w >> 16) & 0xFFFFu) +
                 (uint32_t)((w >> 32) & 0xFFFFu) + (uint32_t)(w >> 48);
        }
        const float z = (float)((int32_t)s - 393210) * (1.0f / 65536.0f);
        const float t = __fmul_rn(sigma, z);
        dst[i] = f2bf(__fadd_rn(mean, t));
    }
}

// One workgroup per row: s = fp16(absmax / 127), code = clamp(rint(w / s), -127, 127).
__global__ void __launch_bounds__(256) quant_int8_rows_kernel(const uint16_t* __restrict__ w, int K,
                                                               int8_t* __restrict__ codes,
                                                               uint16_t* __restrict__ scales) {
    __shared__ float red[16];
    const int64_t row = blockIdx.x;
    const uint16_t* wr = w + row * (int64_t)K;
    float am = 0.f;
    for (int k = threadIdx.x; k < K; k += blockDim.x) am = fmaxf(am, fabsf(bf2f(wr[k])));
    am = block_max(am, red);
    const uint16_t sh = f2h(__fdiv_rn(am, 127.0f));
    const float s = h2f(sh);
    int8_t* cr = codes + row * (int64_t)K;
    for (int k = threadIdx.x; k < K; k += blockDim.x) {
        float c = 0.f;
        if (s != 0.f) c = fminf(fmaxf(rintf(__fdiv_rn(bf2f(wr[k]), s)), -127.f), 127.f);
        cr[k] = (int8_t)(int)c;
    }
    if (threadIdx.x == 0) scales[row] = sh;
}

// One wave per (row, group of 128).  Codes are written in the device nibble order:
// nibble p of the word for columns 8w..8w+7 holds column 8w + 2p (p < 4) or
// 8w + 2(p-4) + 1 (p >= 4), so that extracting nibble pairs (p, p+4) yields
// consecutive columns.
__global__ void __launch_bounds__(256) quant_int4_kernel(const uint16_t* __restrict__ w, int N, int K,
                                                          uint32_t* __restrict__ codes,
                                                          uint16_t* __restrict__ scales,
                                                          uint16_t* __restrict__ zeros) {
    const int lane = threadIdx.x & 63;
    const int64_t gidx = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const int G = K / 128;
    if (gidx >= (int64_t)N * G) return;
    const int64_t row = gidx / G;
    const int g = (int)(gidx % G);
    const uint16_t* wr = w + row * (int64_t)K + g * 128;
    const float w0 = bf2f(wr[2 * lane]), w1 = bf2f(wr[2 * lane + 1]);
    const float lo = fminf(0.f, wave_min(fminf(w0, w1)));
    const float hi = fmaxf(0.f, wave_max(fmaxf(w0, w1)));
    uint16_t sh;
    if (hi == lo) sh = f2h(1.0f);
    else sh = f2h(__fdiv_rn(__fsub_rn(hi, lo), 15.0f));
    const float s = h2f(sh);
    const float z = fminf(fmaxf(rintf(__fdiv_rn(-lo, s)), 0.f), 15.f);
    const uint32_t q0 = (uint32_t)fminf(fmaxf(rintf(__fdiv_rn(w0, s)) + z, 0.f), 15.f);
    const uint32_t q1 = (uint32_t)fminf(fmaxf(rintf(__fdiv_rn(w1, s)) + z, 0.f), 15.f);
    const int j = lane & 3;   // columns 2j, 2j+1 of the lane's word
    uint32_t part = (q0 << (4 * j)) | (q1 << (4 * (j + 4)));
    part |= __shfl_xor(part, 1, 64);
    part |= __shfl_xor(part, 2, 64);
    if (j == 0) codes[row * (int64_t)(K / 8) + g * 16 + (lane >> 2)] = part;
    if (lane == 0) {
        scales[row * (int64_t)G + g] = sh;
        zeros[row * (int64_t)G + g] = f2h(z);
    }
}

// Row-major [n, K] codes (n % 16 == 0) -> fragment-major tiles of the destination
// matrix starting at row row0: block (row / 16, k / KS) of 1024 bytes holds, for lane
// L = r + 16 g, the 16 bytes of row 16 * (row / 16) + r covering k in
// [KS * step + g * KS / 4, + KS / 4).  Columns beyond K (padding up to a multiple
// of KS) are zero.  ebits: element size in bits (16, 8 or 4).
__global__ void __launch_bounds__(256) tile_kernel(const uint8_t* __restrict__ src, int n, int K, int ebits,
                                                   int KS, uint8_t* __restrict__ dst, int row0) {
    const int nst = (K + KS - 1) / KS;
    const int64_t total = (int64_t)(n / 16) * nst * 64;
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= total) return;
    const int L = (int)(c % 64);
    const int64_t blk = c / 64;
    const int step = (int)(blk % nst);
    const int ntl = (int)(blk / nst);
    const int r = L & 15, g = L >> 4;
    const int row = ntl * 16 + r;
    const int k0 = step * KS + g * (KS / 4);
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (k0 < K) {
        const int64_t rowbytes = (int64_t)K * ebits / 8;
        v = *(const u32x4*)(src + row * rowbytes + (int64_t)k0 * ebits / 8);
    }
    const int64_t nt = row0 / 16 + ntl;
    *(u32x4*)(dst + ((nt * nst + step) * 64 + L) * 16) = v;
}

hipError_t launch_tile(const void* src, int n, int K, int ebits, int KS, void* dst, int row0, hipStream_t st) {
    const int nst = (K + KS - 1) / KS;
    const int64_t total = (int64_t)(n / 16) * nst * 64;
    FP_LAUNCH(tile_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                       (const uint8_t*)src, n, K, ebits, KS, (uint8_t*)dst, row0);
    return hipGetLastError();
}

hipError_t launch_fill_bf16(uint16_t* dst, int64_t n, uint64_t key, float mean, float sigma,
                            hipStream_t st) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    FP_LAUNCH(fill_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, st, dst, n, key, mean,
                       sigma);
    return hipGetLastError();
}

hipError_t launch_quant_int8(const uint16_t* w, int N, int K, int8_t* codes, uint16_t* scales,
                             hipStream_t st) {
    FP_LAUNCH(quant_int8_rows_kernel, dim3(N), dim3(256), 0, st, w, K, codes, scales);
    return hipGetLastError();
}

// int4 groups: scale and zero point of each (row, group) packed into one word
// (scale bits low, zero bits high), so a kernel fetches both with one load.  The words
// are stored group-major, sz[g * N + n]: the rows a wave streams through one group are
// consecutive words (one cache line for 32 rows) rather than one line per row.
__global__ void __launch_bounds__(256) pack_sz_kernel(const uint16_t* __restrict__ scales,
                                                      const uint16_t* __restrict__ zeros, int N, int ng,
                                                      uint32_t* __restrict__ sz) {
    const int64_t n_all = (int64_t)N * ng;
    for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < n_all; o += (int64_t)gridDim.x * 256) {
        const int64_t g = o / N, n = o % N;
        const int64_t i = n * ng + g;                 // [N, ng] index of scales and zeros
        sz[o] = (uint32_t)scales[i] | ((uint32_t)zeros[i] << 16);
    }
}

hipError_t launch_pack_sz(const uint16_t* scales, const uint16_t* zeros, int N, int ng, uint32_t* sz,
                          hipStream_t st) {
    const int64_t n = (int64_t)N * ng;
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
    FP_LAUNCH(pack_sz_kernel, dim3((unsigned)blocks), dim3(256), 0, st, scales, zeros, N, ng, sz);
    return hipGetLastError();
}

hipError_t launch_quant_int4(const uint16_t* w, int N, int K, uint32_t* codes, uint16_t* scales,
                             uint16_t* zeros, hipStream_t st) {
    const int64_t groups = (int64_t)N * (K / 128);
    const int64_t blocks = (groups + 3) / 4;
    FP_LAUNCH(quant_int4_kernel, dim3((unsigned)blocks), dim3(256), 0, st, w, N, K, codes,
                       scales, zeros);
    return hipGetLastError();
}

}  // namespace fpk
