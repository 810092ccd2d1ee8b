// The fingerprint's blocks outside the hidden layers (paper Sec. 5.1, Fig. 2: the token
// embedding, the normalisation layer and the LM head around the hidden layers).  Their
// time is the "other" share of TTFT and TPOT (Sec. 5.3, Eq. 2 and Eq. 3).
//   x = E[id]                                     embedding gather (bf16 rows)
//   yn = bf16(y * rsqrt(mean(y^2) + eps) * g)     final RMSNorm of each sequence's last position
//   logits = yn W_lm^T                            LM head: the decode projection kernels on
//                                                 a bf16 [vocab, hidden] matrix
//   next = argmax(logits)                         greedy; lowest id among equal maxima
// The LM head's split-K partial sums are reduced here in increasing split order, with
// the logits written (optionally) and each 2048-logit block's best value and id; a
// second kernel picks each row's best block.
#include <climits>

#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

// One workgroup per token, 16-byte copies (hidden is a multiple of 16).  Ids outside
// [0, vocab) give a zero row; the load address is clamped to row 0 so nothing outside
// the table is read.
__global__ void __launch_bounds__(256) embed_kernel(const int* __restrict__ ids, const uint16_t* __restrict__ E,
                                                     int V, int H, uint16_t* __restrict__ x) {
    const int64_t m = blockIdx.x;
    const int id = ids[m];
    const bool ok = id >= 0 && id < V;
    const u32x4* src = (const u32x4*)(E + (ok ? (int64_t)id : 0) * H);
    u32x4* dst = (u32x4*)(x + m * (int64_t)H);
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
    for (int c = threadIdx.x; c < H / 8; c += 256) {
        const u32x4 v = src[c];
        dst[c] = ok ? v : zero;
    }
}

// Final RMSNorm of row (b, T - 1) of y [B, T, H]: out[b] = bf16(y * r * g), bf16.
__global__ void __launch_bounds__(256) head_norm_kernel(const uint16_t* __restrict__ y, int T, int H,
                                                         const uint16_t* __restrict__ g, float eps,
                                                         uint16_t* __restrict__ out) {
    __shared__ float red[16];
    const int64_t b = blockIdx.x;
    const u32x4* yr = (const u32x4*)(y + (b * T + (T - 1)) * (int64_t)H);
    const int nv = H / 8;
    float ss = 0.f;
    for (int c = threadIdx.x; c < nv; c += 256) {
        const u32x4 v = yr[c];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float e0 = __uint_as_float(w4[j] << 16), e1 = __uint_as_float(w4[j] & 0xFFFF0000u);
            ss += e0 * e0 + e1 * e1;
        }
    }
    ss = block_sum(ss, red);
    const float r = 1.0f / __fsqrt_rn(ss / (float)H + eps);
    u32x4* orow = (u32x4*)(out + b * (int64_t)H);
    const u32x4* gv = (const u32x4*)g;
    for (int c = threadIdx.x; c < nv; c += 256) {
        const u32x4 v = yr[c], gg = gv[c];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w}, g4[4] = {gg.x, gg.y, gg.z, gg.w};
        uint32_t o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float e0 = bfround(__uint_as_float(w4[j] << 16) * r * __uint_as_float(g4[j] << 16));
            const float e1 = bfround(__uint_as_float(w4[j] & 0xFFFF0000u) * r * __uint_as_float(g4[j] & 0xFFFF0000u));
            o[j] = (uint32_t)f2bf(e0) | ((uint32_t)f2bf(e1) << 16);
        }
        orow[c] = u32x4{o[0], o[1], o[2], o[3]};
    }
}

// (value, id) pairs: the larger value wins, the lower id on equal values.
__device__ __forceinline__ void best_of(float& v, int& i, float ov, int oi) {
    if (ov > v || (ov == v && oi < i)) {
        v = ov;
        i = oi;
    }
}

__device__ __forceinline__ void wave_best(float& v, int& i) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(v, o, 64);
        const int oi = __shfl_xor(i, o, 64);
        best_of(v, i, ov, oi);
    }
}

constexpr int LG_BLK = 2048;      // logits per workgroup: 256 threads x 8 consecutive ids

// Sum the ks partials of logits [b, v0 .. v0 + 2047] (vocab is a multiple of 8), write
// them to logits (if non-NULL) and the block's best (value, id) to bval / bidx [B, nblk].
__global__ void __launch_bounds__(256) logits_kernel(const float* __restrict__ part, int ks, int B, int V,
                                                      float* __restrict__ logits, float* __restrict__ bval,
                                                      int* __restrict__ bidx) {
    __shared__ float sv[4];
    __shared__ int si[4];
    const int64_t b = blockIdx.y;
    const int v0 = blockIdx.x * LG_BLK + threadIdx.x * 8;
    float best = -INFINITY;
    int bi = INT_MAX;
    if (v0 < V) {
        float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int k = 0; k < ks; ++k) {
            const f32x4* p = (const f32x4*)(part + ((int64_t)k * B + b) * V + v0);
            const f32x4 a = p[0], c = p[1];
            s[0] += a[0]; s[1] += a[1]; s[2] += a[2]; s[3] += a[3];
            s[4] += c[0]; s[5] += c[1]; s[6] += c[2]; s[7] += c[3];
        }
        if (logits) {
            f32x4* q = (f32x4*)(logits + b * V + v0);
            q[0] = f32x4{s[0], s[1], s[2], s[3]};
            q[1] = f32x4{s[4], s[5], s[6], s[7]};
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) best_of(best, bi, s[j], v0 + j);
    }
    wave_best(best, bi);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) {
        sv[w] = best;
        si[w] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int j = 1; j < 4; ++j) best_of(best, bi, sv[j], si[j]);
        bval[b * gridDim.x + blockIdx.x] = best;
        bidx[b * gridDim.x + blockIdx.x] = bi;
    }
}

// One wave per row: the best of the row's nblk block results.
__global__ void __launch_bounds__(64) argmax_kernel(const float* __restrict__ bval, const int* __restrict__ bidx,
                                                     int nblk, int* __restrict__ out_ids) {
    const int64_t b = blockIdx.x;
    float best = -INFINITY;
    int bi = INT_MAX;
    for (int j = threadIdx.x; j < nblk; j += 64) best_of(best, bi, bval[b * nblk + j], bidx[b * nblk + j]);
    wave_best(best, bi);
    if (threadIdx.x == 0) out_ids[b] = bi == INT_MAX ? 0 : bi;
}

hipError_t launch_embed(const int* ids, int64_t M, const uint16_t* E, int V, int H, uint16_t* x, hipStream_t st) {
    if (M < 1 || H % 8 != 0 || M > INT_MAX) return hipErrorInvalidValue;
    FP_LAUNCH(embed_kernel, dim3((unsigned)M), dim3(256), 0, st, ids, E, V, H, x);
    return hipGetLastError();
}

hipError_t launch_head_norm(const uint16_t* y, int B, int T, int H, const uint16_t* g, float eps, uint16_t* out,
                            hipStream_t st) {
    if (B < 1 || T < 1 || H % 8 != 0) return hipErrorInvalidValue;
    FP_LAUNCH(head_norm_kernel, dim3(B), dim3(256), 0, st, y, T, H, g, eps, out);
    return hipGetLastError();
}

int head_logit_blocks(int V) { return (V + LG_BLK - 1) / LG_BLK; }

hipError_t launch_logits_argmax(const float* part, int ks, int B, int V, float* logits, float* bval, int* bidx,
                                int* out_ids, hipStream_t st) {
    if (ks < 1 || B < 1 || V < 1 || V % 8 != 0) return hipErrorInvalidValue;
    const int nblk = head_logit_blocks(V);
    FP_LAUNCH(logits_kernel, dim3(nblk, B), dim3(256), 0, st, part, ks, B, V, logits, bval, bidx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    FP_LAUNCH(argmax_kernel, dim3(B), dim3(64), 0, st, bval, bidx, nblk, out_ids);
    return hipGetLastError();
}

}  // namespace fpk
