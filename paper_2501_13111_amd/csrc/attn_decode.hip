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

constexpr int DEC_CH = 64;    // keys per chunk

template <int D, int G, bool KV8>
__global__ void __launch_bounds__(256) attn_decode_kernel(AttnDecArgs a) {
    constexpr int LPK = D / 8;                 // lanes per key in the score phase
    constexpr int KPI = 64 / LPK;              // keys per wave per load instruction
    constexpr int KPW = DEC_CH / 4;            // keys per wave per chunk
    constexpr int NLD = KPW / KPI;             // K loads per lane per chunk
    constexpr int TPR = D / 4;                 // P.V threads per value row (4 dims each)
    constexpr int NKG = 256 / TPR;             // P.V key groups
    constexpr int KPG = DEC_CH / NKG;          // keys per group per chunk
    __shared__ float q_s[G * D];
    __shared__ float sc[G * DEC_CH];
    __shared__ float red[NKG * G * D];
    __shared__ float m_run[G], l_run[G], alpha[G];
    __shared__ float newk[D], newv[D], newsc[2];   // stored value of the appended token

    const int sp = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int len = *a.d_pos + 1;
    const int pos = len - 1;
    const int k_beg = sp * a.keys_per_split;
    if (k_beg >= len) return;
    const int k_end = min(len, k_beg + a.keys_per_split);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.max_seq;   // cache row of position 0

    // ---- rotary embedding of the G queries (sum of the qkv split-K partials first)
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
    if (tid < G) { m_run[tid] = -INFINITY; l_run[tid] = 0.f; }

    // ---- the split holding the new token appends its K / V (rotated k; bf16 or int8).
    // It then takes that token's K / V from LDS rather than reading the row back, so
    // no memory fence is needed.
    const bool writer = (pos < k_end);
    if (writer && tid < 64) {
        const int kcol = a.nh * D + kvh * D, vcol = a.nh * D + a.nkv * D + kvh * D;
        const int64_t crow = crow0 + pos;
        float k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
        const int j = tid;
        if (j < D / 2) {
            const float u = sum_parts(prow + kcol + j, a.ks, pstride);
            const float x = sum_parts(prow + kcol + j + D / 2, a.ks, pstride);
            k0 = __fsub_rn(__fmul_rn(u, cr[j]), __fmul_rn(x, sr[j]));
            k1 = __fadd_rn(__fmul_rn(x, cr[j]), __fmul_rn(u, sr[j]));
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
                const uint16_t bk0 = f2bf(k0), bk1 = f2bf(k1), bv0 = f2bf(v0), bv1 = f2bf(v1);
                kd[j] = bk0; kd[j + D / 2] = bk1;
                vd[j] = bv0; vd[j + D / 2] = bv1;
                newk[j] = bf2f(bk0); newk[j + D / 2] = bf2f(bk1);
                newv[j] = bf2f(bv0); newv[j + D / 2] = bf2f(bv1);
            }
            if (j == 0) { newsc[0] = 1.f; newsc[1] = 1.f; }
        } else {
            const float ka = wave_max(fmaxf(fabsf(k0), fabsf(k1)));
            const float va = wave_max(fmaxf(fabsf(v0), fabsf(v1)));
            const uint16_t ksh = f2h(__fdiv_rn(ka, 127.0f)), vsh = f2h(__fdiv_rn(va, 127.0f));
            const float ksf = h2f(ksh), vsf = h2f(vsh);
            auto q8 = [](float x, float scl) -> int8_t {
                if (scl == 0.f) return 0;
                return (int8_t)(int)fminf(fmaxf(rintf(__fdiv_rn(x, scl)), -127.f), 127.f);
            };
            if (j < D / 2) {
                int8_t* kd = (int8_t*)a.kc + crow * D;
                int8_t* vd = (int8_t*)a.vc + crow * D;
                const int8_t ck0 = q8(k0, ksf), ck1 = q8(k1, ksf), cv0 = q8(v0, vsf), cv1 = q8(v1, vsf);
                kd[j] = ck0; kd[j + D / 2] = ck1;
                vd[j] = cv0; vd[j + D / 2] = cv1;
                newk[j] = (float)ck0; newk[j + D / 2] = (float)ck1;
                newv[j] = (float)cv0; newv[j + D / 2] = (float)cv1;
            }
            if (j == 0) {
                a.k_scales[crow] = ksh;
                a.v_scales[crow] = vsh;
                newsc[0] = ksf;
                newsc[1] = vsf;
            }
        }
    }
    __syncthreads();

    const int kin = lane / LPK, part = lane % LPK;   // score phase
    const int dq = tid % TPR, kg = tid / TPR;        // P.V phase: dims 4 dq .. 4 dq + 3
    float o[G][4];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e) o[h][e] = 0.f;

    for (int base = k_beg; base < k_end; base += DEC_CH) {
        const int nk = min(DEC_CH, k_end - base);
        const int newkey = pos - base;                   // chunk-local index of the new token
        // ---- K loads and scores
        float kf[NLD][8];
        float ksc[NLD];
#pragma unroll
        for (int t = 0; t < NLD; ++t) {
            const int key = w * KPW + t * KPI + kin;
            const bool valid = key < nk && key != newkey;
            const int64_t row = crow0 + base + key;
            if constexpr (KV8) {
                u32x2 raw = u32x2{0u, 0u};
                if (valid) raw = *(const u32x2*)((const int8_t*)a.kc + row * D + 8 * part);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    kf[t][j] = (float)(int8_t)((raw.x >> (8 * j)) & 0xFF);
                    kf[t][4 + j] = (float)(int8_t)((raw.y >> (8 * j)) & 0xFF);
                }
                ksc[t] = valid ? h2f(a.k_scales[row]) : 0.f;
            } else {
                u32x4 raw = u32x4{0u, 0u, 0u, 0u};
                if (valid) raw = *(const u32x4*)((const uint16_t*)a.kc + row * D + 8 * part);
                kf[t][0] = __uint_as_float(raw.x << 16); kf[t][1] = __uint_as_float(raw.x & 0xFFFF0000u);
                kf[t][2] = __uint_as_float(raw.y << 16); kf[t][3] = __uint_as_float(raw.y & 0xFFFF0000u);
                kf[t][4] = __uint_as_float(raw.z << 16); kf[t][5] = __uint_as_float(raw.z & 0xFFFF0000u);
                kf[t][6] = __uint_as_float(raw.w << 16); kf[t][7] = __uint_as_float(raw.w & 0xFFFF0000u);
                ksc[t] = 1.0f;
            }
            if (key == newkey) {
#pragma unroll
                for (int j = 0; j < 8; ++j) kf[t][j] = newk[8 * part + j];
                ksc[t] = newsc[0];
            }
        }
        // ---- V loads of this thread's keys (in flight during the scores and softmax)
        float vv[KPG][4];
#pragma unroll
        for (int t = 0; t < KPG; ++t) {
            const int j = kg * KPG + t;
            const int64_t row = crow0 + base + j;
#pragma unroll
            for (int e = 0; e < 4; ++e) vv[t][e] = 0.f;
            if (j == newkey) {
#pragma unroll
                for (int e = 0; e < 4; ++e) vv[t][e] = newv[4 * dq + e] * newsc[1];
            } else if (j < nk) {
                if constexpr (KV8) {
                    const uint32_t raw = *(const uint32_t*)((const int8_t*)a.vc + row * D + 4 * dq);
                    const float vs = h2f(a.v_scales[row]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) vv[t][e] = (float)(int8_t)((raw >> (8 * e)) & 0xFF) * vs;
                } else {
                    const u32x2 raw = *(const u32x2*)((const uint16_t*)a.vc + row * D + 4 * dq);
                    vv[t][0] = __uint_as_float(raw.x << 16); vv[t][1] = __uint_as_float(raw.x & 0xFFFF0000u);
                    vv[t][2] = __uint_as_float(raw.y << 16); vv[t][3] = __uint_as_float(raw.y & 0xFFFF0000u);
                }
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
                for (int sh = LPK / 2; sh >= 1; sh >>= 1) dot += __shfl_xor(dot, sh, 64);
                const int key = w * KPW + t * KPI + kin;
                if (part == 0) sc[h * DEC_CH + key] = key < nk ? dot * ksc[t] * a.scale : -INFINITY;
            }
        }
        __syncthreads();
        // ---- online softmax over the chunk (one wave per head, one key per lane)
        for (int h = w; h < G; h += 4) {
            const float sv = sc[h * DEC_CH + lane];
            const float mc = wave_max(sv);
            const float mo = m_run[h];
            const float mn = fmaxf(mo, mc);
            const float p = __expf(sv - mn);            // masked keys: exp(-inf) = 0
            sc[h * DEC_CH + lane] = p;
            const float ps = wave_sum(p);
            if (lane == 0) {
                const float al = __expf(mo - mn);       // 0 on the first chunk
                alpha[h] = al;
                l_run[h] = l_run[h] * al + ps;
                m_run[h] = mn;
            }
        }
        __syncthreads();
        // ---- P . V into the running accumulators
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float al = alpha[h];
#pragma unroll
            for (int e = 0; e < 4; ++e) o[h][e] *= al;
#pragma unroll
            for (int t = 0; t < KPG; ++t) {
                const float p = sc[h * DEC_CH + kg * KPG + t];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[h][e] += p * vv[t][e];
            }
        }
        __syncthreads();
    }

    // ---- sum the key groups, then normalise (one split) or write the split's partial
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[(kg * G + h) * D + 4 * dq + e] = o[h][e];
    __syncthreads();
    const int nsplit = gridDim.x;
    for (int i = tid; i < G * D; i += 256) {
        const int h = i / D, dd = i % D;
        float sum = 0.f;
#pragma unroll
        for (int k = 0; k < NKG; ++k) sum += red[(k * G + h) * D + dd];
        const int hg = kvh * G + h;
        if (nsplit == 1) {
            a.out[((int64_t)b * a.nh + hg) * D + dd] = act_store(bfround(sum / l_run[h]), a.out_fmt);
        } else {
            float* dst = a.ws + (((int64_t)b * a.nh + hg) * nsplit + sp) * (D + 4);
            dst[dd] = sum;
            if (dd == 0) { dst[D] = m_run[h]; dst[D + 1] = l_run[h]; }
        }
    }
}

// ---------------------------------------------------------------------------------
// Wave-per-item variant for small query groups (G <= 2, e.g. multi-head attention):
// each wave owns one (sequence, kv head, split) and walks its keys in 64-key chunks
// with no workgroup barrier.  A lane owns 8 dims of one key per load (head_dim/8
// lanes per key) for both K and V, and issues all K and V loads of a chunk before
// using any; scores are summed by a butterfly inside each key's lane group (every
// lane of the group ends with the score), the online softmax by shuffles across
// groups, and P.V accumulates the lane's 8 dims over its keys, summed across the
// key groups once at the end.  The four waves of a workgroup are independent items.
template <int D, int G, bool KV8>
__global__ void __launch_bounds__(256) attn_decode_wave_kernel(AttnDecArgs a, int nsplit) {
    constexpr int KC = 32;                     // keys per chunk
    constexpr int LPK = D / 8;                 // lanes per key (scores)
    constexpr int KPI = 64 / LPK;              // keys per load instruction
    constexpr int NT = KC / KPI;               // K loads per lane per chunk
    __shared__ float qsh[4][G * D];            // per-wave scratch (no cross-wave sharing)
    __shared__ float nks[4][2 * D + 2];        // appended token: k, v stored values, scales

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int item = blockIdx.x * 4 + w;
    const int B = a.batch;
    if (item >= B * a.nkv * nsplit) return;
    const int sp = item % nsplit;
    const int kvh = (item / nsplit) % a.nkv;
    const int b = item / (nsplit * a.nkv);
    const int len = *a.d_pos + 1;
    const int pos = len - 1;
    const int k_beg = sp * a.keys_per_split;
    if (k_beg >= len) return;
    const int k_end = min(len, k_beg + a.keys_per_split);
    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.max_seq;
    float* qs = qsh[w];
    float* nk = nks[w];

    // ---- rotary embedding of the queries, and the appended token (lane = pair index)
    const int Nqkv = (a.nh + 2 * a.nkv) * D;
    const int64_t pstride = (int64_t)B * Nqkv;
    const float* prow = a.qkv_part + (int64_t)b * Nqkv;
    const float* cr = a.cos_t + (int64_t)pos * (D / 2);
    const float* sr = a.sin_t + (int64_t)pos * (D / 2);
    for (int j = lane; j < D / 2; j += 64) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const int col = (kvh * G + h) * D + j;
            const float u = sum_parts(prow + col, a.ks, pstride), v = sum_parts(prow + col + D / 2, a.ks, pstride);
            qs[h * D + j] = __fsub_rn(__fmul_rn(u, cr[j]), __fmul_rn(v, sr[j]));
            qs[h * D + j + D / 2] = __fadd_rn(__fmul_rn(v, cr[j]), __fmul_rn(u, sr[j]));
        }
    }
    const bool writer = pos < k_end;
    if (writer) {
        const int kcol = a.nh * D + kvh * D, vcol = a.nh * D + a.nkv * D + kvh * D;
        const int64_t crow = crow0 + pos;
        const int j = lane;
        float k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
        if (j < D / 2) {
            const float u = sum_parts(prow + kcol + j, a.ks, pstride);
            const float x = sum_parts(prow + kcol + j + D / 2, a.ks, pstride);
            k0 = __fsub_rn(__fmul_rn(u, cr[j]), __fmul_rn(x, sr[j]));
            k1 = __fadd_rn(__fmul_rn(x, cr[j]), __fmul_rn(u, sr[j]));
            v0 = sum_parts(prow + vcol + j, a.ks, pstride);
            v1 = sum_parts(prow + vcol + j + D / 2, a.ks, pstride);
            if (a.dump) {
                float* dk = a.dump + ((int64_t)b * a.nkv + kvh) * D;
                float* dv = a.dump + ((int64_t)B * a.nkv + (int64_t)b * a.nkv + kvh) * D;
                dk[j] = k0; dk[j + D / 2] = k1;
                dv[j] = v0; dv[j + D / 2] = v1;
            }
        }
        if (!a.kv_int8) {
            if (j < D / 2) {
                uint16_t* kd = (uint16_t*)a.kc + crow * D;
                uint16_t* vd = (uint16_t*)a.vc + crow * D;
                const uint16_t bk0 = f2bf(k0), bk1 = f2bf(k1), bv0 = f2bf(v0), bv1 = f2bf(v1);
                kd[j] = bk0; kd[j + D / 2] = bk1;
                vd[j] = bv0; vd[j + D / 2] = bv1;
                nk[j] = bf2f(bk0); nk[j + D / 2] = bf2f(bk1);
                nk[D + j] = bf2f(bv0); nk[D + j + D / 2] = bf2f(bv1);
            }
            if (j == 0) { nk[2 * D] = 1.f; nk[2 * D + 1] = 1.f; }
        } else {
            const float ka = wave_max(fmaxf(fabsf(k0), fabsf(k1)));
            const float va = wave_max(fmaxf(fabsf(v0), fabsf(v1)));
            const uint16_t ksh = f2h(__fdiv_rn(ka, 127.0f)), vsh = f2h(__fdiv_rn(va, 127.0f));
            const float ksf = h2f(ksh), vsf = h2f(vsh);
            auto q8 = [](float x, float scl) -> int8_t {
                if (scl == 0.f) return 0;
                return (int8_t)(int)fminf(fmaxf(rintf(__fdiv_rn(x, scl)), -127.f), 127.f);
            };
            if (j < D / 2) {
                int8_t* kd = (int8_t*)a.kc + crow * D;
                int8_t* vd = (int8_t*)a.vc + crow * D;
                const int8_t ck0 = q8(k0, ksf), ck1 = q8(k1, ksf), cv0 = q8(v0, vsf), cv1 = q8(v1, vsf);
                kd[j] = ck0; kd[j + D / 2] = ck1;
                vd[j] = cv0; vd[j + D / 2] = cv1;
                nk[j] = (float)ck0; nk[j + D / 2] = (float)ck1;
                nk[D + j] = (float)cv0; nk[D + j + D / 2] = (float)cv1;
            }
            if (j == 0) {
                a.k_scales[crow] = ksh;
                a.v_scales[crow] = vsh;
                nk[2 * D] = ksf;
                nk[2 * D + 1] = vsf;
            }
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    const int kin = lane / LPK, part = lane % LPK;
    float qv[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int j = 0; j < 8; ++j) qv[h][j] = qs[h * D + 8 * part + j];

    float m_run[G], l_run[G], o[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m_run[h] = -INFINITY;
        l_run[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
    }

    for (int base = k_beg; base < k_end; base += KC) {
        const int nkeys = min(KC, k_end - base);
        const int newkey = pos - base;
        // ---- all K and V loads of the chunk
        u32x4 kraw[NT];
        float ksc[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int key = t * KPI + kin;
            const int64_t row = crow0 + base + key;
            kraw[t] = u32x4{0u, 0u, 0u, 0u};
            ksc[t] = 1.f;
            if (key < nkeys && key != newkey) {
                if constexpr (KV8) {
                    const u32x2 r2 = *(const u32x2*)((const int8_t*)a.kc + row * D + 8 * part);
                    kraw[t].x = r2.x;
                    kraw[t].y = r2.y;
                    ksc[t] = h2f(a.k_scales[row]);
                } else {
                    kraw[t] = *(const u32x4*)((const uint16_t*)a.kc + row * D + 8 * part);
                }
            }
        }
        u32x4 vraw[NT];
        float vsc[KV8 ? NT : 1];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int key = t * KPI + kin;
            const int64_t row = crow0 + base + key;
            vraw[t] = u32x4{0u, 0u, 0u, 0u};
            if constexpr (KV8) vsc[t] = 0.f;
            if (key < nkeys && key != newkey) {
                if constexpr (KV8) {
                    const u32x2 r2 = *(const u32x2*)((const int8_t*)a.vc + row * D + 8 * part);
                    vraw[t].x = r2.x;
                    vraw[t].y = r2.y;
                    vsc[t] = h2f(a.v_scales[row]);
                } else {
                    vraw[t] = *(const u32x4*)((const uint16_t*)a.vc + row * D + 8 * part);
                }
            }
        }
        // ---- scores (every lane of key group kin ends with the key's score)
        float sc[G][NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int key = t * KPI + kin;
            float kf[8];
            if (key == newkey) {
#pragma unroll
                for (int j = 0; j < 8; ++j) kf[j] = nk[8 * part + j];
                ksc[t] = nk[2 * D];
            } else if constexpr (KV8) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    kf[j] = (float)(int8_t)((kraw[t].x >> (8 * j)) & 0xFF);
                    kf[4 + j] = (float)(int8_t)((kraw[t].y >> (8 * j)) & 0xFF);
                }
            } else {
                kf[0] = __uint_as_float(kraw[t].x << 16); kf[1] = __uint_as_float(kraw[t].x & 0xFFFF0000u);
                kf[2] = __uint_as_float(kraw[t].y << 16); kf[3] = __uint_as_float(kraw[t].y & 0xFFFF0000u);
                kf[4] = __uint_as_float(kraw[t].z << 16); kf[5] = __uint_as_float(kraw[t].z & 0xFFFF0000u);
                kf[6] = __uint_as_float(kraw[t].w << 16); kf[7] = __uint_as_float(kraw[t].w & 0xFFFF0000u);
            }
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float dot = 0.f;
#pragma unroll
                for (int j = 0; j < 8; ++j) dot += qv[h][j] * kf[j];
#pragma unroll
                for (int sh = LPK / 2; sh >= 1; sh >>= 1) dot += __shfl_xor(dot, sh, 64);
                sc[h][t] = key < nkeys ? dot * ksc[t] * a.scale : -INFINITY;
            }
        }
        // ---- online softmax and P.V
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float mc = sc[h][0];
#pragma unroll
            for (int t = 1; t < NT; ++t) mc = fmaxf(mc, sc[h][t]);
#pragma unroll
            for (int sh = LPK; sh < 64; sh <<= 1) mc = fmaxf(mc, __shfl_xor(mc, sh, 64));
            const float mn = fmaxf(m_run[h], mc);
            const float al = __expf(m_run[h] - mn);
            float ps = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                sc[h][t] = __expf(sc[h][t] - mn);
                ps += sc[h][t];
            }
#pragma unroll
            for (int sh = LPK; sh < 64; sh <<= 1) ps += __shfl_xor(ps, sh, 64);
            l_run[h] = l_run[h] * al + ps;
            m_run[h] = mn;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[h][e] *= al;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int key = t * KPI + kin;
                float vf[8];
                if (key == newkey) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) vf[e] = nk[D + 8 * part + e] * nk[2 * D + 1];
                } else if constexpr (KV8) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        vf[e] = (float)(int8_t)((vraw[t].x >> (8 * e)) & 0xFF) * vsc[t];
                        vf[4 + e] = (float)(int8_t)((vraw[t].y >> (8 * e)) & 0xFF) * vsc[t];
                    }
                } else {
                    vf[0] = __uint_as_float(vraw[t].x << 16); vf[1] = __uint_as_float(vraw[t].x & 0xFFFF0000u);
                    vf[2] = __uint_as_float(vraw[t].y << 16); vf[3] = __uint_as_float(vraw[t].y & 0xFFFF0000u);
                    vf[4] = __uint_as_float(vraw[t].z << 16); vf[5] = __uint_as_float(vraw[t].z & 0xFFFF0000u);
                    vf[6] = __uint_as_float(vraw[t].w << 16); vf[7] = __uint_as_float(vraw[t].w & 0xFFFF0000u);
                }
                const float p = sc[h][t];
#pragma unroll
                for (int e = 0; e < 8; ++e) o[h][e] += p * vf[e];
            }
        }
    }

    // sum the key groups (lanes with equal part)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int sh = LPK; sh < 64; sh <<= 1) o[h][e] += __shfl_xor(o[h][e], sh, 64);

    // ---- one split: normalise and store; several: write the partial for the merge
    if (kin == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const int hg = kvh * G + h;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int dd = 8 * part + e;
                if (nsplit == 1) {
                    a.out[((int64_t)b * a.nh + hg) * D + dd] = act_store(bfround(o[h][e] / l_run[h]), a.out_fmt);
                } else {
                    float* dst = a.ws + (((int64_t)b * a.nh + hg) * nsplit + sp) * (D + 4);
                    dst[dd] = o[h][e];
                    if (dd == 0) { dst[D] = m_run[h]; dst[D + 1] = l_run[h]; }
                }
            }
        }
    }
}

// One workgroup of D threads per (head, sequence): log-sum-exp merge of the chunks.
template <int D>
__global__ void __launch_bounds__(D) attn_merge_kernel(AttnDecArgs a, int nch) {
    const int h = blockIdx.x, b = blockIdx.y, i = threadIdx.x;
    const int len = *a.d_pos + 1;
    const int nv = (len + a.keys_per_split - 1) / a.keys_per_split;
    const float* src = a.ws + ((int64_t)b * a.nh + h) * nch * (D + 4);
    float m = -INFINITY;
    for (int c = 0; c < nv; ++c) m = fmaxf(m, src[c * (D + 4) + D]);
    float l = 0.f, o = 0.f;
    for (int c = 0; c < nv; ++c) {
        const float e = __expf(src[c * (D + 4) + D] - m);
        l += src[c * (D + 4) + D + 1] * e;
        o += src[c * (D + 4) + i] * e;
    }
    a.out[((int64_t)b * a.nh + h) * D + i] = act_store(bfround(o / l), a.out_fmt);
}

// Splits of the context: enough workgroups to fill the GPU, at least one 64-key chunk
// each.  The grid depends only on the capacity, so a captured graph replays at every
// position (splits past the current length exit at once).
void attn_decode_split(int max_seq, int B, int nkv, int group, int* nsplit, int* keys_per_split) {
    // small groups run one wave per split (aim at ~4096 waves), larger groups one
    // workgroup per split (aim at ~1024 workgroups)
    const int target = group <= 2 ? 4096 : 1024;
    const int want = (target + B * nkv - 1) / (B * nkv);
    const int chunks = (max_seq + DEC_CH - 1) / DEC_CH;
    int ns = want < chunks ? want : chunks;
    if (ns < 1) ns = 1;
    const int cps = (chunks + ns - 1) / ns;
    *keys_per_split = cps * DEC_CH;
    *nsplit = (max_seq + *keys_per_split - 1) / *keys_per_split;
}

int attn_decode_chunks(int max_seq) { return (max_seq + DEC_CH - 1) / DEC_CH; }

template <int D, int G, bool KV8>
static hipError_t launch_dgk(const AttnDecArgs& a, int B, int nsplit, hipStream_t st) {
    if constexpr (G <= 2) {
        const int items = B * a.nkv * nsplit;
        FP_LAUNCH((attn_decode_wave_kernel<D, G, KV8>), dim3((items + 3) / 4), dim3(256), 0, st, a, nsplit);
    } else {
        FP_LAUNCH((attn_decode_kernel<D, G, KV8>), dim3(nsplit, a.nkv, B), dim3(256), 0, st, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || nsplit == 1 || a.skip_merge) return e;
    FP_LAUNCH(attn_merge_kernel<D>, dim3(a.nh, B), dim3(D), 0, st, a, nsplit);
    return hipGetLastError();
}

template <int D, int G>
static hipError_t launch_dg(const AttnDecArgs& a, int B, int nsplit, hipStream_t st) {
    return a.kv_int8 ? launch_dgk<D, G, true>(a, B, nsplit, st) : launch_dgk<D, G, false>(a, B, nsplit, st);
}

template <int D>
static hipError_t launch_d(const AttnDecArgs& a, int B, int nsplit, hipStream_t st) {
    switch (a.nh / a.nkv) {
        case 1: return launch_dg<D, 1>(a, B, nsplit, st);
        case 2: return launch_dg<D, 2>(a, B, nsplit, st);
        case 4: return launch_dg<D, 4>(a, B, nsplit, st);
        case 8: return launch_dg<D, 8>(a, B, nsplit, st);
        default: return hipErrorInvalidValue;
    }
}

bool attn_decode_supported(int d, int group) {
    return (d == 64 || d == 128) && (group == 1 || group == 2 || group == 4 || group == 8);
}

hipError_t launch_attn_decode(const AttnDecArgs& a, int B, hipStream_t st) {
    const int nsplit = (a.max_seq + a.keys_per_split - 1) / a.keys_per_split;
    if (a.d == 128) return launch_d<128>(a, B, nsplit, st);
    if (a.d == 64) return launch_d<64>(a, B, nsplit, st);
    return hipErrorInvalidValue;
}

}  // namespace fpk
