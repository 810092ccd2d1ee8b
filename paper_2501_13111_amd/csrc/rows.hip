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
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

// ---------------------------------------------------------------- RMSNorm
// One workgroup per row.  out = act(bf16(x * r * g)), r = 1 / sqrt(mean(x^2) + eps).
__global__ void __launch_bounds__(256) rmsnorm_kernel(const uint16_t* __restrict__ x, int H,
                                                       const uint16_t* __restrict__ g, float eps,
                                                       uint16_t* __restrict__ out, int out_fmt) {
    __shared__ float red[16];
    const int64_t row = blockIdx.x;
    const uint16_t* xr = x + row * (int64_t)H;
    float ss = 0.f;
    for (int k = threadIdx.x; k < H; k += blockDim.x) {
        const float v = bf2f(xr[k]);
        ss += v * v;
    }
    ss = block_sum(ss, red);
    const float r = 1.0f / __fsqrt_rn(ss / (float)H + eps);
    uint16_t* orow = out + row * (int64_t)H;
    for (int k = threadIdx.x; k < H; k += blockDim.x)
        orow[k] = act_store(bfround(bf2f(xr[k]) * r * bf2f(g[k])), out_fmt);
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

// ---------------------------------------------------------------- SwiGLU epilogue
// a[m, f] = act(bf16(silu(G) * U)), G = sum_s part[s, m, f], U = sum_s part[s, m, F + f].
__global__ void __launch_bounds__(256) swiglu_kernel(const float* __restrict__ part, int ks, int M,
                                                      int F, uint16_t* __restrict__ a, int afmt) {
    const int64_t m = blockIdx.y;
    const int f = blockIdx.x * blockDim.x + threadIdx.x;
    if (f >= F) return;
    const float gs = sum_parts(part + m * (2 * (int64_t)F) + f, ks, (int64_t)M * 2 * F);
    const float us = sum_parts(part + m * (2 * (int64_t)F) + F + f, ks, (int64_t)M * 2 * F);
    a[m * (int64_t)F + f] = act_store(bfround(silu_f(gs) * us), afmt);
}

// ---------------------------------------------------------------- rotary + KV append
// One 64-lane workgroup per (token row m, head slot).  Head slots 0..nh-1 are query
// heads, nh..nh+nkv-1 are kv heads (K and V).  qkv = sum of ks partials [ks, M, Nqkv]
// (columns: q heads, then k heads, then v heads).  Token m is sequence m / T at
// position pos0 + m % T, where pos0 = *d_pos (decode) or 0 (prefill).
// Writes rotated q (fp32, [M, nh*d]); stores K / V in the cache
// [B, nkv, max_seq, d] as bf16 or int8 + fp16 scale [B, nkv, max_seq].
#pragma clang fp contract(off)
__global__ void __launch_bounds__(64) rope_kv_kernel(const float* __restrict__ part, int ks, int M,
                                                      int T, int nh, int nkv, int d,
                                                      const int* __restrict__ d_pos,
                                                      const float* __restrict__ cos_t,
                                                      const float* __restrict__ sin_t, int max_seq,
                                                      float* __restrict__ qout, void* __restrict__ kc,
                                                      void* __restrict__ vc,
                                                      uint16_t* __restrict__ ks_out,
                                                      uint16_t* __restrict__ vs_out, int kv_int8,
                                                      float* __restrict__ dump) {
    const int m = blockIdx.x;
    const int slot = blockIdx.y;
    const int lane = threadIdx.x;
    const int half = d / 2;
    const int Nqkv = (nh + 2 * nkv) * d;
    const int b = m / T;
    const int pos = (d_pos ? *d_pos : 0) + (m % T);
    auto load = [&](int col) { return sum_parts(part + (int64_t)m * Nqkv + col, ks, (int64_t)M * Nqkv); };
    const float* cr = cos_t + (int64_t)pos * half;
    const float* sr = sin_t + (int64_t)pos * half;
    if (slot < nh) {
        const int base = slot * d;
        for (int i = lane; i < half; i += 64) {
            const float u = load(base + i), v = load(base + half + i);
            const float c = cr[i], s = sr[i];
            qout[(int64_t)m * nh * d + base + i] = __fsub_rn(__fmul_rn(u, c), __fmul_rn(v, s));
            qout[(int64_t)m * nh * d + base + half + i] = __fadd_rn(__fmul_rn(v, c), __fmul_rn(u, s));
        }
        return;
    }
    const int kvh = slot - nh;
    const int kbase = nh * d + kvh * d, vbase = nh * d + nkv * d + kvh * d;
    const int64_t cidx = (((int64_t)b * nkv + kvh) * max_seq + pos);   // (b, kvh, pos)
    // each lane holds up to 4 rotated k and 4 v values (d <= 256)
    float kr[4], vr[4];
    int cnt = 0;
    for (int i = lane; i < half; i += 64, ++cnt) {
        const float u = load(kbase + i), v = load(kbase + half + i);
        const float c = cr[i], s = sr[i];
        kr[2 * cnt] = __fsub_rn(__fmul_rn(u, c), __fmul_rn(v, s));
        kr[2 * cnt + 1] = __fadd_rn(__fmul_rn(v, c), __fmul_rn(u, s));
        vr[2 * cnt] = load(vbase + i);
        vr[2 * cnt + 1] = load(vbase + half + i);
    }
    if (dump) {
        // [2, M, nkv, d] slice of this step: dump[0] = K, dump[1] = V
        float* dk = dump + ((int64_t)m * nkv + kvh) * d;
        float* dv = dump + (int64_t)M * nkv * d + ((int64_t)m * nkv + kvh) * d;
        int c2 = 0;
        for (int i = lane; i < half; i += 64, ++c2) {
            dk[i] = kr[2 * c2]; dk[half + i] = kr[2 * c2 + 1];
            dv[i] = vr[2 * c2]; dv[half + i] = vr[2 * c2 + 1];
        }
    }
    if (!kv_int8) {
        uint16_t* kd = (uint16_t*)kc + cidx * d;
        uint16_t* vd = (uint16_t*)vc + cidx * d;
        int c2 = 0;
        for (int i = lane; i < half; i += 64, ++c2) {
            kd[i] = f2bf(kr[2 * c2]); kd[half + i] = f2bf(kr[2 * c2 + 1]);
            vd[i] = f2bf(vr[2 * c2]); vd[half + i] = f2bf(vr[2 * c2 + 1]);
        }
        return;
    }
    float ka = 0.f, va = 0.f;
    for (int j = 0; j < 2 * cnt; ++j) { ka = fmaxf(ka, fabsf(kr[j])); va = fmaxf(va, fabsf(vr[j])); }
    ka = wave_max(ka);
    va = wave_max(va);
    const uint16_t ksh = f2h(__fdiv_rn(ka, 127.0f)), vsh = f2h(__fdiv_rn(va, 127.0f));
    const float ksf = h2f(ksh), vsf = h2f(vsh);
    auto q8 = [](float v, float s) -> int8_t {
        if (s == 0.f) return 0;
        return (int8_t)(int)fminf(fmaxf(rintf(__fdiv_rn(v, s)), -127.f), 127.f);
    };
    int8_t* kd = (int8_t*)kc + cidx * d;
    int8_t* vd = (int8_t*)vc + cidx * d;
    int c2 = 0;
    for (int i = lane; i < half; i += 64, ++c2) {
        kd[i] = q8(kr[2 * c2], ksf); kd[half + i] = q8(kr[2 * c2 + 1], ksf);
        vd[i] = q8(vr[2 * c2], vsf); vd[half + i] = q8(vr[2 * c2 + 1], vsf);
    }
    if (lane == 0) { ks_out[cidx] = ksh; vs_out[cidx] = vsh; }
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
    FP_LAUNCH(rope_kv_kernel, dim3(a.M, a.nh + a.nkv), dim3(64), 0, st, a.part, a.ks, a.M,
                       a.T, a.nh, a.nkv, a.d, a.d_pos, a.cos_t, a.sin_t, a.max_seq, a.qout, a.kc,
                       a.vc, a.ks_out, a.vs_out, a.kv_int8, a.dump);
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
