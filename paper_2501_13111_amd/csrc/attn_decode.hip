// Decode attention: one new query per (sequence, head) against the whole cached
// prefix, which already holds the new token's K / V (appended just before).
//
// The KV cache is what keeps the per-token decode cost constant (paper Sec. 5.3);
// reading it is the second HBM stream of a decode step after the weights, and
// with an INT8 KV cache (Sec. 3.2) it is half as many bytes.
//
// Split-context scheme: workgroup (chunk c, kv head, sequence) covers 256 keys
// for the G = n_heads / n_kv_heads query heads that share the kv head (grouped-
// query attention), and writes an unnormalised partial (max m_c, sum l_c,
// sum_j e^{s_j - m_c} v_j).  The merge kernel combines the chunks with the exact
// log-sum-exp identity  m = max m_c,  l = sum l_c e^{m_c - m},
// o = sum o_c e^{m_c - m} / l.  The grid is sized for max_seq so that a captured
// graph can be replayed at every position; chunks past the current length exit.
//
// Scores: 8 consecutive dims per lane (16 B of bf16 or 8 B of int8 codes), head_dim/8
// lanes per key, butterfly sum across those lanes.  Values: each thread owns two
// dims of one key range, so a wave reads whole 256-byte value rows.
// int8 keys / values: s_k multiplies the dot product, s_v the probability.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

constexpr int DEC_CH = 256;   // keys per chunk

template <int D, int G>
__global__ void __launch_bounds__(256) attn_decode_kernel(AttnDecArgs a) {
    constexpr int NKG = 256 / (D / 2);       // key groups of the P.V phase
    __shared__ float q_s[G * D];
    __shared__ float sc[G * DEC_CH];
    __shared__ float red[NKG * G * D];
    __shared__ float stat_m[G], stat_l[G];

    const int c = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int len = *a.d_pos + 1;
    const int k_beg = c * DEC_CH;
    if (k_beg >= len) return;
    const int nk = min(DEC_CH, len - k_beg);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

    // queries of the G heads of this kv head
    for (int i = tid; i < G * D; i += 256) {
        const int h = kvh * G + i / D;
        q_s[i] = a.q[((int64_t)b * a.nh + h) * D + (i % D)];
    }
    __syncthreads();

    const int64_t cache_row0 = ((int64_t)b * a.nkv + kvh) * a.max_seq + k_beg;   // key index base
    // ---- scores
    constexpr int LPK = D / 8;               // lanes per key
    constexpr int KPS = 64 / LPK;            // keys per wave step
    const int kin = lane / LPK, part = lane % LPK;
    for (int kk = w * KPS; kk < nk; kk += 4 * KPS) {
        const int key = kk + kin;
        float kv[8];
        const bool valid = key < nk;
        if (a.kv_int8) {
            u32x2 raw = u32x2{0u, 0u};
            if (valid) raw = *(const u32x2*)((const int8_t*)a.kc + (cache_row0 + key) * D + 8 * part);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                kv[j] = (float)(int8_t)((raw.x >> (8 * j)) & 0xFF);
                kv[4 + j] = (float)(int8_t)((raw.y >> (8 * j)) & 0xFF);
            }
        } else {
            u32x4 raw = u32x4{0u, 0u, 0u, 0u};
            if (valid) raw = *(const u32x4*)((const uint16_t*)a.kc + (cache_row0 + key) * D + 8 * part);
            kv[0] = __uint_as_float(raw.x << 16); kv[1] = __uint_as_float(raw.x & 0xFFFF0000u);
            kv[2] = __uint_as_float(raw.y << 16); kv[3] = __uint_as_float(raw.y & 0xFFFF0000u);
            kv[4] = __uint_as_float(raw.z << 16); kv[5] = __uint_as_float(raw.z & 0xFFFF0000u);
            kv[6] = __uint_as_float(raw.w << 16); kv[7] = __uint_as_float(raw.w & 0xFFFF0000u);
        }
        const float ksc = (a.kv_int8 && valid) ? h2f(a.k_scales[cache_row0 + key]) : 1.0f;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float* qh = q_s + h * D + 8 * part;
            float dot = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) dot += qh[j] * kv[j];
#pragma unroll
            for (int o = LPK / 2; o >= 1; o >>= 1) dot += __shfl_xor(dot, o, 64);
            if (part == 0 && valid) sc[h * DEC_CH + key] = dot * ksc * a.scale;
        }
    }
    __syncthreads();

    // ---- softmax statistics per head over this chunk
    for (int h = w; h < G; h += 4) {
        float m = -INFINITY;
        for (int j = lane; j < nk; j += 64) m = fmaxf(m, sc[h * DEC_CH + j]);
        m = wave_max(m);
        float l = 0.f;
        for (int j = lane; j < nk; j += 64) {
            const float p = __expf(sc[h * DEC_CH + j] - m);
            sc[h * DEC_CH + j] = p;
            l += p;
        }
        l = wave_sum(l);
        if (lane == 0) { stat_m[h] = m; stat_l[h] = l; }
    }
    __syncthreads();

    // ---- P . V
    const int dp = tid % (D / 2), kg = tid / (D / 2);
    const int per = (nk + NKG - 1) / NKG;
    const int j0 = kg * per, j1 = min(nk, j0 + per);
    float o0[G], o1[G];
#pragma unroll
    for (int h = 0; h < G; ++h) { o0[h] = 0.f; o1[h] = 0.f; }
    for (int j = j0; j < j1; ++j) {
        float v0, v1;
        if (a.kv_int8) {
            const uint16_t raw = *(const uint16_t*)((const int8_t*)a.vc + (cache_row0 + j) * D + 2 * dp);
            const float vs = h2f(a.v_scales[cache_row0 + j]);
            v0 = (float)(int8_t)(raw & 0xFF) * vs;
            v1 = (float)(int8_t)(raw >> 8) * vs;
        } else {
            const uint32_t raw = *(const uint32_t*)((const uint16_t*)a.vc + (cache_row0 + j) * D + 2 * dp);
            v0 = __uint_as_float(raw << 16);
            v1 = __uint_as_float(raw & 0xFFFF0000u);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float p = sc[h * DEC_CH + j];
            o0[h] += p * v0;
            o1[h] += p * v1;
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
        red[(kg * G + h) * D + 2 * dp] = o0[h];
        red[(kg * G + h) * D + 2 * dp + 1] = o1[h];
    }
    __syncthreads();
    const int nch = gridDim.x;
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, dd = i % D;
        float s = 0.f;
        for (int k = 0; k < NKG; ++k) s += red[(k * G + h) * D + dd];
        const int hg = kvh * G + h;
        float* dst = a.ws + (((int64_t)b * a.nh + hg) * nch + c) * (D + 2);
        dst[dd] = s;
        if (dd == 0) { dst[D] = stat_m[h]; dst[D + 1] = stat_l[h]; }
    }
}

// One workgroup of D threads per (head, sequence): log-sum-exp merge of the chunks.
template <int D>
__global__ void __launch_bounds__(D) attn_merge_kernel(AttnDecArgs a, int nch) {
    const int h = blockIdx.x, b = blockIdx.y, i = threadIdx.x;
    const int len = *a.d_pos + 1;
    const int nv = (len + DEC_CH - 1) / DEC_CH;
    const float* src = a.ws + ((int64_t)b * a.nh + h) * nch * (D + 2);
    float m = -INFINITY;
    for (int c = 0; c < nv; ++c) m = fmaxf(m, src[c * (D + 2) + D]);
    float l = 0.f, o = 0.f;
    for (int c = 0; c < nv; ++c) {
        const float e = __expf(src[c * (D + 2) + D] - m);
        l += src[c * (D + 2) + D + 1] * e;
        o += src[c * (D + 2) + i] * e;
    }
    a.out[((int64_t)b * a.nh + h) * D + i] = act_store(bfround(o / l), a.out_fmt);
}

int attn_decode_chunks(int max_seq) { return (max_seq + DEC_CH - 1) / DEC_CH; }

template <int D, int G>
static hipError_t launch_dg(const AttnDecArgs& a, int B, int nch, hipStream_t st) {
    hipLaunchKernelGGL((attn_decode_kernel<D, G>), dim3(nch, a.nkv, B), dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_merge_kernel<D>, dim3(a.nh, B), dim3(D), 0, st, a, nch);
    return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const AttnDecArgs& a, int B, int nch, hipStream_t st) {
    switch (a.nh / a.nkv) {
        case 1: return launch_dg<D, 1>(a, B, nch, st);
        case 2: return launch_dg<D, 2>(a, B, nch, st);
        case 4: return launch_dg<D, 4>(a, B, nch, st);
        case 8: return launch_dg<D, 8>(a, B, nch, st);
        default: return hipErrorInvalidValue;
    }
}

bool attn_decode_supported(int d, int group) {
    return (d == 64 || d == 128) && (group == 1 || group == 2 || group == 4 || group == 8);
}

hipError_t launch_attn_decode(const AttnDecArgs& a, int B, hipStream_t st) {
    const int nch = attn_decode_chunks(a.max_seq);
    if (a.d == 128) return launch_d<128>(a, B, nch, st);
    if (a.d == 64) return launch_d<64>(a, B, nch, st);
    return hipErrorInvalidValue;
}

}  // namespace fpk
