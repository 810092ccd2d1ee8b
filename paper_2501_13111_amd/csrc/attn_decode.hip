// Decode attention: one new query per (sequence, head) against the whole cached
// prefix including the new token.  The kernel also applies the rotary embedding to
// the new q and k (from the qkv projection's split-K partial sums) and appends the
// new k, v to the cache -- as bf16, or as int8 with s = fp16(absmax/127),
// code = rint(v/s) per (sequence, position, kv head) -- in the workgroup whose chunk
// holds the new position.
//
// The KV cache is what keeps the per-token decode cost constant (paper Sec. 5.3);
// reading it is the second HBM stream of a decode step after the weights, and
// with an INT8 KV cache (Sec. 3.2) it is half as many bytes.
//
// Split-context scheme: workgroup (chunk c, kv head, sequence) covers 64 keys
// for the G = n_heads / n_kv_heads query heads that share the kv head (grouped-
// query attention), and writes an unnormalised partial (max m_c, sum l_c,
// sum_j e^{s_j - m_c} v_j).  The merge kernel combines the chunks with the exact
// log-sum-exp identity  m = max m_c,  l = sum l_c e^{m_c - m},
// o = sum o_c e^{m_c - m} / l.  The grid is sized for max_seq so that a captured
// graph can be replayed at every position; chunks past the current length exit.
//
// Scores: 8 consecutive dims per lane (16 B of bf16 or 8 B of int8 codes), head_dim/8
// lanes per key, butterfly sum across those lanes.  Values: each thread owns two
// dims of a group of keys, so a wave reads whole value rows.  All K and V loads of a
// thread are issued before any of them is used, so the chunk streams at full
// memory-level parallelism.
// int8 keys / values: s_k multiplies the dot product, s_v the probability.
#include "fp_device.h"
#include "fp_internal.h"



namespace fpk {

constexpr int DEC_CH = 64;    // keys per chunk (one workgroup)

template <int D, int G>
__global__ void __launch_bounds__(256) attn_decode_kernel(AttnDecArgs a) {
    constexpr int LPK = D / 8;                 // lanes per key in the score phase
    constexpr int KPI = 64 / LPK;              // keys per wave per load instruction
    constexpr int KPW = DEC_CH / 4;            // keys per wave
    constexpr int NLD = KPW / KPI;             // K loads per lane
    constexpr int NKG = 256 / (D / 2);         // key groups of the P.V phase
    constexpr int KPG = DEC_CH / NKG;          // keys per group
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
    const int64_t row0 = ((int64_t)b * a.nkv + kvh) * a.max_seq + k_beg;   // cache row of key 0

    // ---- rotary embedding of the G queries (sum of the qkv split-K partials first)
    const int pos = len - 1;
    const int Nqkv = (a.nh + 2 * a.nkv) * D;
    const int64_t pstride = (int64_t)gridDim.z * Nqkv;
    const float* prow = a.qkv_part + (int64_t)b * Nqkv;
    const float* cr = a.cos_t + (int64_t)pos * (D / 2);
    const float* sr = a.sin_t + (int64_t)pos * (D / 2);
    for (int i = tid; i < G * (D / 2); i += 256) {
        const int h = i / (D / 2), j = i % (D / 2);
        const int col = (kvh * G + h) * D + j;
        const float u = sum_parts(prow + col, a.ks, pstride), v = sum_parts(prow + col + D / 2, a.ks, pstride);
        q_s[h * D + j] = __fsub_rn(__fmul_rn(u, cr[j]), __fmul_rn(v, sr[j]));
        q_s[h * D + j + D / 2] = __fadd_rn(__fmul_rn(v, cr[j]), __fmul_rn(u, sr[j]));
    }
    // ---- the chunk holding the new token appends its K / V (rotated k; bf16 or int8)
    if (c == pos / DEC_CH && tid < 64) {
        const int kcol = a.nh * D + kvh * D, vcol = a.nh * D + a.nkv * D + kvh * D;
        const int64_t crow = ((int64_t)b * a.nkv + kvh) * a.max_seq + pos;
        float k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
        const int j = tid;
        if (j < D / 2) {
            const float u = sum_parts(prow + kcol + j, a.ks, pstride);
            const float w = sum_parts(prow + kcol + j + D / 2, a.ks, pstride);
            k0 = __fsub_rn(__fmul_rn(u, cr[j]), __fmul_rn(w, sr[j]));
            k1 = __fadd_rn(__fmul_rn(w, cr[j]), __fmul_rn(u, sr[j]));
            v0 = sum_parts(prow + vcol + j, a.ks, pstride);
            v1 = sum_parts(prow + vcol + j + D / 2, a.ks, pstride);
            if (a.dump) {
                float* dk = a.dump + ((int64_t)b * a.nkv + kvh) * D;
                float* dv = a.dump + ((int64_t)gridDim.z * a.nkv + (int64_t)b * a.nkv + kvh) * D;
                dk[j] = k0; dk[j + D / 2] = k1;
                dv[j] = v0; dv[j + D / 2] = v1;
            }
        }
        if (!a.kv_int8) {
            if (j < D / 2) {
                uint16_t* kd = (uint16_t*)a.kc + crow * D;
                uint16_t* vd = (uint16_t*)a.vc + crow * D;
                kd[j] = f2bf(k0); kd[j + D / 2] = f2bf(k1);
                vd[j] = f2bf(v0); vd[j + D / 2] = f2bf(v1);
            }
        } else {
            const float ka = wave_max(fmaxf(fabsf(k0), fabsf(k1)));
            const float va = wave_max(fmaxf(fabsf(v0), fabsf(v1)));
            const uint16_t ksh = f2h(__fdiv_rn(ka, 127.0f)), vsh = f2h(__fdiv_rn(va, 127.0f));
            const float ksf = h2f(ksh), vsf = h2f(vsh);
            auto q8 = [](float x, float sc) -> int8_t {
                if (sc == 0.f) return 0;
                return (int8_t)(int)fminf(fmaxf(rintf(__fdiv_rn(x, sc)), -127.f), 127.f);
            };
            if (j < D / 2) {
                int8_t* kd = (int8_t*)a.kc + crow * D;
                int8_t* vd = (int8_t*)a.vc + crow * D;
                kd[j] = q8(k0, ksf); kd[j + D / 2] = q8(k1, ksf);
                vd[j] = q8(v0, vsf); vd[j + D / 2] = q8(v1, vsf);
            }
            if (j == 0) { a.k_scales[crow] = ksh; a.v_scales[crow] = vsh; }
        }
        __threadfence();   // the appended row is read back below by this workgroup
    }
    __syncthreads();

    // ---- scores: issue every K load of the lane first
    const int kin = lane / LPK, part = lane % LPK;
    float kf[NLD][8];
    float ksc[NLD];
#pragma unroll
    for (int t = 0; t < NLD; ++t) {
        const int key = w * KPW + t * KPI + kin;
        const bool valid = key < nk;
        if (a.kv_int8) {
            u32x2 raw = u32x2{0u, 0u};
            if (valid) raw = *(const u32x2*)((const int8_t*)a.kc + (row0 + key) * D + 8 * part);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                kf[t][j] = (float)(int8_t)((raw.x >> (8 * j)) & 0xFF);
                kf[t][4 + j] = (float)(int8_t)((raw.y >> (8 * j)) & 0xFF);
            }
            ksc[t] = valid ? h2f(a.k_scales[row0 + key]) : 0.f;
        } else {
            u32x4 raw = u32x4{0u, 0u, 0u, 0u};
            if (valid) raw = *(const u32x4*)((const uint16_t*)a.kc + (row0 + key) * D + 8 * part);
            kf[t][0] = __uint_as_float(raw.x << 16); kf[t][1] = __uint_as_float(raw.x & 0xFFFF0000u);
            kf[t][2] = __uint_as_float(raw.y << 16); kf[t][3] = __uint_as_float(raw.y & 0xFFFF0000u);
            kf[t][4] = __uint_as_float(raw.z << 16); kf[t][5] = __uint_as_float(raw.z & 0xFFFF0000u);
            kf[t][6] = __uint_as_float(raw.w << 16); kf[t][7] = __uint_as_float(raw.w & 0xFFFF0000u);
            ksc[t] = 1.0f;
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
        float qv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) qv[j] = q_s[h * D + 8 * part + j];
#pragma unroll
        for (int t = 0; t < NLD; ++t) {
            float dot = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) dot += qv[j] * kf[t][j];
#pragma unroll
            for (int o = LPK / 2; o >= 1; o >>= 1) dot += __shfl_xor(dot, o, 64);
            const int key = w * KPW + t * KPI + kin;
            if (part == 0 && key < nk) sc[h * DEC_CH + key] = dot * ksc[t] * a.scale;
        }
    }

    // ---- value loads of this thread's keys (issued before the softmax)
    const int dp = tid % (D / 2), kg = tid / (D / 2);
    float v0[KPG], v1[KPG];
#pragma unroll
    for (int t = 0; t < KPG; ++t) {
        const int j = kg * KPG + t;
        v0[t] = 0.f;
        v1[t] = 0.f;
        if (j < nk) {
            if (a.kv_int8) {
                const uint16_t raw = *(const uint16_t*)((const int8_t*)a.vc + (row0 + j) * D + 2 * dp);
                const float vs = h2f(a.v_scales[row0 + j]);
                v0[t] = (float)(int8_t)(raw & 0xFF) * vs;
                v1[t] = (float)(int8_t)(raw >> 8) * vs;
            } else {
                const uint32_t raw = *(const uint32_t*)((const uint16_t*)a.vc + (row0 + j) * D + 2 * dp);
                v0[t] = __uint_as_float(raw << 16);
                v1[t] = __uint_as_float(raw & 0xFFFF0000u);
            }
        }
    }
    __syncthreads();

    // ---- softmax statistics per head over this chunk (one wave per head, one key per lane)
    for (int h = w; h < G; h += 4) {
        const float sv = lane < nk ? sc[h * DEC_CH + lane] : -INFINITY;
        const float m = wave_max(sv);
        const float p = lane < nk ? __expf(sv - m) : 0.f;
        sc[h * DEC_CH + lane] = p;
        const float l = wave_sum(p);
        if (lane == 0) { stat_m[h] = m; stat_l[h] = l; }
    }
    __syncthreads();

    // ---- P . V
    float o0[G], o1[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        o0[h] = 0.f;
        o1[h] = 0.f;
#pragma unroll
        for (int t = 0; t < KPG; ++t) {
            const float p = sc[h * DEC_CH + kg * KPG + t];
            o0[h] += p * v0[t];
            o1[h] += p * v1[t];
        }
        red[(kg * G + h) * D + 2 * dp] = o0[h];
        red[(kg * G + h) * D + 2 * dp + 1] = o1[h];
    }
    __syncthreads();
    const int nch = gridDim.x;
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, dd = i % D;
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NKG; ++k) s += red[(k * G + h) * D + dd];
        float* dst = a.ws + (((int64_t)b * a.nh + kvh * G + h) * nch + c) * (D + 2);
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
