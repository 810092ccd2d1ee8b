// Row-wise kernels of the layer: RMSNorm, the residual / SwiGLU epilogues that
// reduce split-K partial sums, and the rotary-embedding + KV-append kernel.
//
// Layer reading (Llama-style decoder layer; the paper names the components --
// normalisation layer, attention, activation -- without their math, Sec. 5.1):
//   xn = bf16(x * rsqrt(mean(x^2) + eps) * g)
//   h  = bf16(x + o W_o^T),  y = bf16(h + a W_down^T)
//   a  = bf16(silu(g) * u),  silu(z) = z / (1 + e^-z)
//   rotary embedding: rotate-half pairs (i, i + d/2) with fp32 cos/sin tables
//   KV append: bf16, or int8 with s = fp16(absmax/127), code = rint(v/s) per
//   (sequence, position, kv head) -- the INT8 KV cache of Sec. 3.2.
#include <algorithm>

#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

// ---------------------------------------------------------------- RMSNorm
// One workgroup per row, 16-byte accesses (H is a multiple of 8).
// out = act(bf16(x * r * g)), r = 1 / sqrt(mean(x^2) + eps).  Rows of up to RMS_MAXV
// 16-byte pieces per thread stay in registers between the two passes; longer rows read
// their pieces again (from L2).
constexpr int RMS_MAXV = 8;
__global__ void __launch_bounds__(256) rmsnorm_kernel(const uint16_t* __restrict__ x, int H,
                                                       const uint16_t* __restrict__ g, float eps,
                                                       uint16_t* __restrict__ out, int out_fmt) {
    __shared__ float red[16];
    const int64_t row = blockIdx.x;
    const u32x4* xr = (const u32x4*)(x + row * (int64_t)H);
    const int nv = H / 8;
    u32x4 keep[RMS_MAXV];
#pragma unroll
    for (int i = 0; i < RMS_MAXV; ++i) {
        const int c = threadIdx.x + 256 * i;
        keep[i] = c < nv ? xr[c] : u32x4{0u, 0u, 0u, 0u};
    }
    float ss = 0.f;
    auto sq = [&](const u32x4& v) {
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float e0 = __uint_as_float(w4[j] << 16), e1 = __uint_as_float(w4[j] & 0xFFFF0000u);
            ss += e0 * e0 + e1 * e1;
        }
    };
#pragma unroll
    for (int i = 0; i < RMS_MAXV; ++i) sq(keep[i]);
    for (int c = threadIdx.x + 256 * RMS_MAXV; c < nv; c += 256) sq(xr[c]);
    ss = block_sum(ss, red);
    const float r = 1.0f / __fsqrt_rn(ss / (float)H + eps);
    u32x4* orow = (u32x4*)(out + row * (int64_t)H);
    const u32x4* gv = (const u32x4*)g;
    auto put = [&](int c, const u32x4& v) {
        const u32x4 gg = gv[c];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w}, g4[4] = {gg.x, gg.y, gg.z, gg.w};
        uint32_t o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float e0 = bfround(__uint_as_float(w4[j] << 16) * r * __uint_as_float(g4[j] << 16));
            const float e1 = bfround(__uint_as_float(w4[j] & 0xFFFF0000u) * r * __uint_as_float(g4[j] & 0xFFFF0000u));
            o[j] = (uint32_t)act_store(e0, out_fmt) | ((uint32_t)act_store(e1, out_fmt) << 16);
        }
        orow[c] = u32x4{o[0], o[1], o[2], o[3]};
    };
#pragma unroll
    for (int i = 0; i < RMS_MAXV; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c < nv) put(c, keep[i]);
    }
    for (int c = threadIdx.x + 256 * RMS_MAXV; c < nv; c += 256) put(c, xr[c]);
}

// ---------------------------------------------------------------- residual epilogue
// Decode rows are few (one per sequence), so the row-wise work is spread over column
// blocks of RB values: resid_ssq writes out = bf16(resid + sum_s part[s]) for its block
// and the block's sum of squares; norm_apply then forms r = 1/sqrt(mean + eps) from the
// row's block sums (fixed order) and writes act(bf16(out * r * g)).  With ks == 0 the
// first kernel only sums squares of resid (the RMSNorm of a layer input).
constexpr int RB = 256;

__global__ void __launch_bounds__(256) resid_ssq_kernel(const float* __restrict__ part, int ks, int M,
                                                         int N, const uint16_t* __restrict__ resid,
                                                         uint16_t* __restrict__ out,
                                                         float* __restrict__ ssq, int* __restrict__ d_pos) {
    __shared__ float red[16];
    const int64_t m = blockIdx.y;
    const int n0 = blockIdx.x * RB;
    float ss = 0.f;
    for (int n = n0 + threadIdx.x; n < min(N, n0 + RB); n += blockDim.x) {
        float v = bf2f(resid[m * (int64_t)N + n]);
        if (ks > 0) {
            v = bfround(v + sum_parts(part + m * (int64_t)N + n, ks, (int64_t)M * N));
            out[m * (int64_t)N + n] = f2bf(v);
        }
        ss += v * v;
    }
    ss = block_sum(ss, red);
    if (threadIdx.x == 0) ssq[m * gridDim.x + blockIdx.x] = ss;
    // the step's last kernel advances the decode position (every reader has run)
    if (d_pos && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *d_pos += 1;
}

__global__ void __launch_bounds__(256) norm_apply_kernel(const uint16_t* __restrict__ y, int N,
                                                          const float* __restrict__ ssq, int nblk,
                                                          const uint16_t* __restrict__ g, float eps,
                                                          uint16_t* __restrict__ nout, int nfmt) {
    const int64_t m = blockIdx.y;
    float ss = 0.f;
    for (int b = 0; b < nblk; ++b) ss += ssq[m * nblk + b];
    const float r = 1.0f / __fsqrt_rn(ss / (float)N + eps);
    const int n0 = blockIdx.x * RB;
    for (int n = n0 + threadIdx.x; n < min(N, n0 + RB); n += blockDim.x)
        nout[m * (int64_t)N + n] = act_store(bfround(bf2f(y[m * (int64_t)N + n]) * r * bf2f(g[n])), nfmt);
}

// Batches: one workgroup of 1024 threads per row does both steps, keeping the row in
// registers (8 consecutive values per thread and pass, N <= 16384): out = bf16(resid +
// sum_s part[s]) (skipped for ks == 0), the row's sum of squares by a block reduction,
// then nout = act(bf16(out * r * g)) (skipped for g == NULL).  One launch instead of two.
constexpr int RN_T = 1024;
__global__ void __launch_bounds__(RN_T) resid_norm_row_kernel(const float* __restrict__ part, int ks, int M, int N,
                                                               const uint16_t* __restrict__ resid,
                                                               uint16_t* __restrict__ out,
                                                               const uint16_t* __restrict__ g, float eps,
                                                               uint16_t* __restrict__ nout, int nfmt,
                                                               int* __restrict__ d_pos) {
    __shared__ float red[16];
    const int64_t m = blockIdx.x;
    const int64_t pstride = (int64_t)M * N;
    float v[2][8];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int n0 = (threadIdx.x + RN_T * j) * 8;
        if (n0 >= N) continue;
        // the residual piece goes out with the partials' loads below and is unpacked after them
        const u32x4 rv = *(const u32x4*)(resid + m * N + n0);
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.f;
        // eight splits' loads in flight together, added in split order
        for (int s0 = 0; s0 < ks; s0 += 8) {
            float4 a0[8], a1[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {                           // past the last split: + 0
                const float* p = part + (s0 + i) * pstride + m * N + n0;
                a0[i] = s0 + i < ks ? *(const float4*)p : float4{0.f, 0.f, 0.f, 0.f};
                a1[i] = s0 + i < ks ? *(const float4*)(p + 4) : float4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                acc[0] += a0[i].x; acc[1] += a0[i].y; acc[2] += a0[i].z; acc[3] += a0[i].w;
                acc[4] += a1[i].x; acc[5] += a1[i].y; acc[6] += a1[i].z; acc[7] += a1[i].w;
            }
        }
        {
            const uint32_t rw[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[j][2 * e] = __uint_as_float(rw[e] << 16);
                v[j][2 * e + 1] = __uint_as_float(rw[e] & 0xFFFF0000u);
            }
        }
        if (ks > 0) {
            uint32_t o[4];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[j][e] = bfround(v[j][e] + acc[e]);
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = (uint32_t)f2bf(v[j][2 * e]) | ((uint32_t)f2bf(v[j][2 * e + 1]) << 16);
            *(u32x4*)(out + m * N + n0) = u32x4{o[0], o[1], o[2], o[3]};
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[j][e] * v[j][e];
    }
    if (g != nullptr) {
        ss = block_sum(ss, red);
        const float r = 1.0f / __fsqrt_rn(ss / (float)N + eps);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n0 = (threadIdx.x + RN_T * j) * 8;
            if (n0 >= N) continue;
            const u32x4 gv = *(const u32x4*)(g + n0);
            const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
            uint32_t o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float e0 = bfround(v[j][2 * e] * r * __uint_as_float(gw[e] << 16));
                const float e1 = bfround(v[j][2 * e + 1] * r * __uint_as_float(gw[e] & 0xFFFF0000u));
                o[e] = (uint32_t)act_store(e0, nfmt) | ((uint32_t)act_store(e1, nfmt) << 16);
            }
            *(u32x4*)(nout + m * N + n0) = u32x4{o[0], o[1], o[2], o[3]};
        }
    }
    if (d_pos && blockIdx.x == 0 && threadIdx.x == 0) *d_pos += 1;
}

// ---------------------------------------------------------------- SwiGLU epilogue
// a[m, f] = act(bf16(silu(G) * U)), G = sum_s part[s, m, f], U = sum_s part[s, m, F + f].
__global__ void __launch_bounds__(256) swiglu_kernel(const float* __restrict__ part, int ks, int M,
                                                      int F, uint16_t* __restrict__ a, int afmt) {
    const int64_t m = blockIdx.y;
    const int f = blockIdx.x * blockDim.x + threadIdx.x;
    if (f >= F) return;
    const float* const cols[2] = {part + m * (2 * (int64_t)F) + f, part + m * (2 * (int64_t)F) + F + f};
    float sum[2];
    sum_parts_cols<2>(cols, ks, (int64_t)M * 2 * F, sum);
    a[m * (int64_t)F + f] = act_store(bfround(silu_f(sum[0]) * sum[1]), afmt);
}

// ---------------------------------------------------------------- rotary + KV append (prefill)
// qkv: the projection output [M, Nqkv] fp32 (columns: q heads, then k heads, then v
// heads); token m is sequence m / T at position m % T.
// Rotated queries head-major [M / T, nh, T, d] (each head's queries of a sequence
// contiguous) in the attention's operand format (fp16 with an int8 cache, else bf16;
// rounded to nearest even once here), one thread per two rotation pairs
// (j, j + d/2) and (j + 1, j + 1 + d/2), so that every store is a whole dword.
#pragma clang fp contract(off)
template <bool F16>
__global__ void __launch_bounds__(256) rope_q_kernel(const float* __restrict__ qkv, int M, int T, int nh,
                                                      int nkv, int d, const float* __restrict__ cos_t,
                                                      const float* __restrict__ sin_t, uint16_t* __restrict__ qout) {
    const int half = d / 2, hp = half / 2;
    const int Nqkv = (nh + 2 * nkv) * d;
    const int64_t n = (int64_t)M * nh * hp;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
        const int j = 2 * (int)(i % hp);
        const int64_t mh = i / hp;
        const int h = (int)(mh % nh);
        const int64_t m = mh / nh;
        const int pos = (int)(m % T);
        const float* p = qkv + m * Nqkv + (int64_t)h * d;
        const float2 u = *(const float2*)(p + j), v = *(const float2*)(p + j + half);
        const float2 c = *(const float2*)(cos_t + (int64_t)pos * half + j);
        const float2 s = *(const float2*)(sin_t + (int64_t)pos * half + j);
        const float lo0 = __fsub_rn(__fmul_rn(u.x, c.x), __fmul_rn(v.x, s.x));
        const float lo1 = __fsub_rn(__fmul_rn(u.y, c.y), __fmul_rn(v.y, s.y));
        const float hi0 = __fadd_rn(__fmul_rn(v.x, c.x), __fmul_rn(u.x, s.x));
        const float hi1 = __fadd_rn(__fmul_rn(v.y, c.y), __fmul_rn(u.y, s.y));
        uint16_t* q = qout + (((m / T) * nh + h) * T + pos) * d;
        *(uint32_t*)(q + j) = F16 ? pack_f16_hw(lo0, lo1) : pack_bf16_hw(lo0, lo1);
        *(uint32_t*)(q + j + half) = F16 ? pack_f16_hw(hi0, hi1) : pack_bf16_hw(hi0, hi1);
    }
}

// K / V of one block of VT_BLK prompt positions of one (sequence, kv head): rotated K
// rows go to the key cache; V is transposed in LDS into the value-block layout
// ([d][VT_BLK], slot vt_slot(kb)) and written out as one contiguous block.  int8:
// s = fp16(absmax/127), code = rint(v/s) per (position, kv head), separately for K
// and V.  Slots past the prompt are cleared.  Lane j handles dims j and j + d/2
// (d <= 128); wave w handles positions w, w + 4, ... of the block.
template <bool KV8>
__global__ void __launch_bounds__(256) kv_append_kernel(const float* __restrict__ qkv, int M, int T, int nh,
                                                         int nkv, int d, const float* __restrict__ cos_t,
                                                         const float* __restrict__ sin_t, int kv_stride, int nblk,
                                                         void* __restrict__ kc, void* __restrict__ vc,
                                                         uint16_t* __restrict__ ks_out,
                                                         uint16_t* __restrict__ vs_out, float* __restrict__ dump) {
    __shared__ __attribute__((aligned(16))) uint16_t vt[128 * VT_BLK];
    uint8_t* vt8 = (uint8_t*)vt;
    const int pb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int half = d / 2;
    const int Nqkv = (nh + 2 * nkv) * d;
    const int kcol = nh * d + kvh * d, vcol = nh * d + nkv * d + kvh * d;
    const int64_t crow0 = ((int64_t)b * nkv + kvh) * kv_stride;
    const int j = lane;
    for (int kb = w; kb < VT_BLK; kb += 4) {
        const int pos = pb * VT_BLK + kb;
        const int slot = vt_slot(kb);
        if (pos >= T) {
            if (j < half) {
                if constexpr (KV8) { vt8[j * VT_BLK + slot] = 0; vt8[(j + half) * VT_BLK + slot] = 0; }
                else { vt[j * VT_BLK + slot] = 0; vt[(j + half) * VT_BLK + slot] = 0; }
            }
            continue;
        }
        const int64_t m = (int64_t)b * T + pos;
        const float* p = qkv + m * Nqkv;
        float k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
        if (j < half) {
            const float u = p[kcol + j], x = p[kcol + j + half];
            const float c = cos_t[(int64_t)pos * half + j], s = sin_t[(int64_t)pos * half + j];
            k0 = __fsub_rn(__fmul_rn(u, c), __fmul_rn(x, s));
            k1 = __fadd_rn(__fmul_rn(x, c), __fmul_rn(u, s));
            v0 = p[vcol + j];
            v1 = p[vcol + j + half];
            if (dump) {   // [2, M, nkv, d]: dump[0] = K, dump[1] = V
                float* dk = dump + (m * nkv + kvh) * d;
                float* dv = dump + (int64_t)M * nkv * d + (m * nkv + kvh) * d;
                dk[j] = k0; dk[j + half] = k1;
                dv[j] = v0; dv[j + half] = v1;
            }
        }
        if constexpr (!KV8) {
            if (j < half) {
                uint16_t* kd = (uint16_t*)kc + (crow0 + pos) * d;
                kd[j] = f2bf(k0); kd[j + half] = f2bf(k1);
                vt[j * VT_BLK + slot] = f2bf(v0);
                vt[(j + half) * VT_BLK + slot] = f2bf(v1);
            }
        } else {
            const float ka = wave_max(fmaxf(fabsf(k0), fabsf(k1)));
            const float va = wave_max(fmaxf(fabsf(v0), fabsf(v1)));
            const uint16_t ksh = f2h(__fdiv_rn(ka, 127.0f)), vsh = f2h(__fdiv_rn(va, 127.0f));
            const float ksf = h2f(ksh), vsf = h2f(vsh);
            auto q8 = [](float v, float s) -> int8_t {
                if (s == 0.f) return 0;
                return (int8_t)(int)fminf(fmaxf(rintf(__fdiv_rn(v, s)), -127.f), 127.f);
            };
            if (j < half) {
                int8_t* kd = (int8_t*)kc + (crow0 + pos) * d;
                kd[j] = q8(k0, ksf); kd[j + half] = q8(k1, ksf);
                vt8[j * VT_BLK + slot] = (uint8_t)q8(v0, vsf);
                vt8[(j + half) * VT_BLK + slot] = (uint8_t)q8(v1, vsf);
            }
            if (j == 0) { ks_out[crow0 + pos] = ksh; vs_out[crow0 + pos] = vsh; }
        }
    }
    __syncthreads();
    const int esz = KV8 ? 1 : 2;
    const int nchunk = d * VT_BLK * esz / 16;
    u32x4* dst = (u32x4*)((char*)vc + (((int64_t)b * nkv + kvh) * nblk + pb) * d * VT_BLK * esz);
    for (int c = threadIdx.x; c < nchunk; c += 256) dst[c] = ((const u32x4*)vt)[c];
}
#pragma clang fp contract(on)

__global__ void set_pos_kernel(int* d_pos, int v) { *d_pos = v; }
__global__ void inc_pos_kernel(int* d_pos) { *d_pos += 1; }

// ---------------------------------------------------------------- launchers
hipError_t launch_rmsnorm(const uint16_t* x, int M, int H, const uint16_t* g, float eps, uint16_t* out,
                          int out_fmt, hipStream_t st) {
    FP_LAUNCH(rmsnorm_kernel, dim3(M), dim3(256), 0, st, x, H, g, eps, out, out_fmt);
    return hipGetLastError();
}

hipError_t launch_resid_norm(const float* part, int ks, int M, int N, const uint16_t* resid,
                             uint16_t* out, const uint16_t* g, float eps, uint16_t* nout, int nfmt,
                             float* ssq, int* inc_pos, hipStream_t st) {
    // the row kernel: with a norm, or a residual alone over enough rows to fill the GPU
    if ((g != nullptr || (ks > 0 && M >= 256)) && M > 1 && N % 8 == 0 && N <= 2 * RN_T * 8) {
        FP_LAUNCH(resid_norm_row_kernel, dim3(M), dim3(RN_T), 0, st, part, ks, M, N, resid, out, g, eps, nout, nfmt,
                  inc_pos);
        return hipGetLastError();
    }
    const int nblk = (N + RB - 1) / RB;
    FP_LAUNCH(resid_ssq_kernel, dim3(nblk, M), dim3(256), 0, st, part, ks, M, N, resid, out, ssq,
                       inc_pos);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || g == nullptr) return e;
    const uint16_t* y = ks > 0 ? out : resid;
    FP_LAUNCH(norm_apply_kernel, dim3(nblk, M), dim3(256), 0, st, y, N, ssq, nblk, g, eps, nout, nfmt);
    return hipGetLastError();
}

int resid_ssq_blocks(int N) { return (N + RB - 1) / RB; }

hipError_t launch_swiglu(const float* part, int ks, int M, int F, uint16_t* a, int afmt,
                         hipStream_t st) {
    FP_LAUNCH(swiglu_kernel, dim3((F + 255) / 256, M), dim3(256), 0, st, part, ks, M, F, a,
                       afmt);
    return hipGetLastError();
}

hipError_t launch_rope_kv(const RopeKvArgs& a, hipStream_t st) {
    if (a.ks != 1 || a.d_pos != nullptr || a.d > 128 || a.M % a.T != 0) return hipErrorInvalidValue;
    if (a.d % 4 != 0) return hipErrorInvalidValue;
    const int64_t pairs = (int64_t)a.M * a.nh * (a.d / 4);
    const int nb = (int)std::min<int64_t>((pairs + 255) / 256, 8192);
    if (a.kv_int8)
        FP_LAUNCH(rope_q_kernel<true>, dim3(nb), dim3(256), 0, st, a.part, a.M, a.T, a.nh, a.nkv, a.d, a.cos_t,
                  a.sin_t, a.qout);
    else
        FP_LAUNCH(rope_q_kernel<false>, dim3(nb), dim3(256), 0, st, a.part, a.M, a.T, a.nh, a.nkv, a.d, a.cos_t,
                  a.sin_t, a.qout);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid((a.T + VT_BLK - 1) / VT_BLK, a.nkv, a.M / a.T);
    if (a.kv_int8)
        FP_LAUNCH(kv_append_kernel<true>, grid, dim3(256), 0, st, a.part, a.M, a.T, a.nh, a.nkv, a.d, a.cos_t,
                  a.sin_t, a.kv_stride, a.nblk, a.kc, a.vc, a.ks_out, a.vs_out, a.dump);
    else
        FP_LAUNCH(kv_append_kernel<false>, grid, dim3(256), 0, st, a.part, a.M, a.T, a.nh, a.nkv, a.d, a.cos_t,
                  a.sin_t, a.kv_stride, a.nblk, a.kc, a.vc, a.ks_out, a.vs_out, a.dump);
    return hipGetLastError();
}

hipError_t launch_set_pos(int* d_pos, int v, hipStream_t st) {
    FP_LAUNCH(set_pos_kernel, dim3(1), dim3(1), 0, st, d_pos, v);
    return hipGetLastError();
}

hipError_t launch_inc_pos(int* d_pos, hipStream_t st) {
    FP_LAUNCH(inc_pos_kernel, dim3(1), dim3(1), 0, st, d_pos);
    return hipGetLastError();
}

}  // namespace fpk
