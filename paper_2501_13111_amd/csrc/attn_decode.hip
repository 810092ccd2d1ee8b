// Decode attention: one new query per (sequence, head) against the whole cached
// prefix including the new token, for grouped-query attention with G = n_heads /
// n_kv_heads query heads per kv head (G <= 16; G = 1 is multi-head attention).
//
// The KV cache is what keeps the per-token decode cost constant (paper Sec. 5.3);
// reading it is the second HBM stream of a decode step after the weights, and
// with an INT8 KV cache (Sec. 3.2) it is half as many bytes.
//
// One kernel, attn_decode_kernel.  Each workgroup reduces the qkv projection's split-K
// partial sums for the queries of its group and rotates them; the workgroup whose
// keys include the new position also rotates k and appends k and v to the cache --
// bf16, or int8 with s = fp16(absmax/127), code = rint(v/s) per (sequence, position,
// kv head) -- before its waves load that block.  Both contractions run on MFMA 16x16x32 (bf16 for a
//    bf16 cache, fp16 for int8 codes, which are exact in fp16), in the transposed form
//        S^T = K Q^T     A = 16 cached keys (rows), B = the G queries (columns)
//        O^T += V^T P^T  A = 16 dims of a value block, B = the probabilities
//    so each lane holds the scores of 4 keys for one query head, which are exactly
//    the values it supplies as B for the next product.  The value cache is stored
//    transposed in 32-position blocks, [head_dim][32] with the positions of a block
//    in the order the probability fragment takes them (vt_slot), so the A operand of
//    P.V is one contiguous 16-byte (bf16) or 8-byte (int8) load per lane.  int8
//    caches: s_k scales the score, s_v the probability.  Online softmax per query
//    column; max and sum across the four lane groups by shuffles.
//
// Context splits: each wave takes keys_per_split keys (a multiple of 32) of one
// (sequence, kv head) and walks them in 32-key chunks, the next chunk's loads in
// flight while the current one is multiplied.  The 4 waves of a workgroup take 4
// consecutive splits and merge them in LDS with the exact log-sum-exp identity
//     m = max m_w,  l = sum l_w e^{m_w - m},  o = sum o_w e^{m_w - m} / l;
// a workgroup that covers the whole context writes the output, otherwise its
// unnormalised partial (o, m, l) for a second merge by the consumer.  The grid is
// sized for max_seq so that a captured graph replays at every position; splits
// past the current length do nothing.
#include <type_traits>

#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

// ---------------------------------------------------------------------------------
// The new token's k and v for kv head kvh of sequence b, done by one wave (lane j
// handles the rotation pair (j, j + D/2)): reduce the qkv projection's split-K
// partial sums, rotate k, and append k and v to the cache (bf16, or int8 with
// s = fp16(absmax/127), code = rint(x/s)).
template <int D, bool KV8>
__device__ __forceinline__ void append_kv(const AttnDecArgs& a, int b, int kvh, int pos, int j) {
    const int Nqkv = (a.nh + 2 * a.nkv) * D;
    const int64_t pstride = (int64_t)a.batch * Nqkv;
    const float* prow = a.qkv_part + (int64_t)b * Nqkv;
    const int kcol = a.nh * D + kvh * D, vcol = a.nh * D + a.nkv * D + kvh * D;
    float k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
    if (j < D / 2) {
        const float c = a.cos_t[(int64_t)pos * (D / 2) + j], sn = a.sin_t[(int64_t)pos * (D / 2) + j];
        const float* const cols[4] = {prow + kcol + j, prow + kcol + j + D / 2, prow + vcol + j, prow + vcol + j + D / 2};
        float sum[4];
        sum_parts_cols<4>(cols, a.ks, pstride, sum);
        const float u = sum[0], x = sum[1];
        k0 = __fsub_rn(__fmul_rn(u, c), __fmul_rn(x, sn));
        k1 = __fadd_rn(__fmul_rn(x, c), __fmul_rn(u, sn));
        v0 = sum[2];
        v1 = sum[3];
        if (a.dump) {   // [2, B, nkv, D] pre-quantisation K, V
            float* dk = a.dump + ((int64_t)b * a.nkv + kvh) * D;
            float* dv = a.dump + ((int64_t)a.batch * a.nkv + (int64_t)b * a.nkv + kvh) * D;
            dk[j] = k0; dk[j + D / 2] = k1;
            dv[j] = v0; dv[j + D / 2] = v1;
        }
    }
    const int64_t crow = ((int64_t)b * a.nkv + kvh) * a.kv_stride + pos;
    const int64_t vrow = (((int64_t)b * a.nkv + kvh) * a.nblk + pos / VT_BLK) * D * VT_BLK + vt_slot(pos % VT_BLK);
    if constexpr (!KV8) {
        if (j < D / 2) {
            uint16_t* kd = (uint16_t*)a.kc + crow * D;
            uint16_t* vd = (uint16_t*)a.vc + vrow;
            kd[j] = f2bf(k0); kd[j + D / 2] = f2bf(k1);
            vd[(int64_t)j * VT_BLK] = f2bf(v0);
            vd[(int64_t)(j + D / 2) * VT_BLK] = f2bf(v1);
        }
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
            int8_t* vd = (int8_t*)a.vc + vrow;
            kd[j] = q8(k0, ksf); kd[j + D / 2] = q8(k1, ksf);
            vd[(int64_t)j * VT_BLK] = q8(v0, vsf);
            vd[(int64_t)(j + D / 2) * VT_BLK] = q8(v1, vsf);
        }
        if (j == 0) {
            a.k_scales[crow] = ksh;
            a.v_scales[crow] = vsh;
        }
    }
}

// ---------------------------------------------------------------------------------
// Lane (r, g) of a key tile holds key r, k-step j: bf16 dims 32 j + 8 g .. + 7 (each
// load instruction reads 64 contiguous bytes of 16 key rows); int8 dims
// 64 (j / 2) + 16 g + 8 (j % 2) .. + 7 (16 codes per load).  The query fragments
// use the same assignment.
template <int D, bool KV8>
__device__ __forceinline__ int qdim(int j, int g) {
    if constexpr (KV8) return 64 * (j >> 1) + 16 * g + 8 * (j & 1);
    else return 32 * j + 8 * g;
}

#ifndef ATTN_DEC_PD
#define ATTN_DEC_PD 2
#endif
template <int D, bool KV8>
struct DecChunk {
    static constexpr int NK = KV8 ? D / 64 : D / 32;   // 16-byte K loads per key tile
    // chunks in flight per wave (measured: three or four in flight are no faster than
    // two on the batched workloads, four slower)
    static constexpr int PD = ATTN_DEC_PD;
    u32x4 k[2][NK];
    typename std::conditional<KV8, u32x2, u32x4>::type v[D / 16];   // int8: 8 codes; bf16: 8 values
    u32x2 ks[2], vs[2];                                 // int8: fp16 scales of keys 16 t + 4 g + i
};

template <int D, bool KV8>
__global__ void __launch_bounds__(256, 2) attn_decode_kernel(AttnDecArgs a, int nsplit) {
    constexpr int AF = KV8 ? ACT_F16 : ACT_BF16;       // MFMA operand format
    constexpr int NJ = D / 32;                         // MFMA k-steps over head_dim
    constexpr int ND = D / 16;                         // 16-dim tiles of the output
    constexpr int NK = DecChunk<D, KV8>::NK;
    __shared__ float mw[4][16], lw[4][16];
    __shared__ __attribute__((aligned(16))) float ow[4][16 * D];
    __shared__ __attribute__((aligned(16))) uint16_t qs[16 * D];    // rotated queries of the group

    const int G = a.nh / a.nkv;
    const int kvh = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int len = *a.d_pos + 1;
    const int kps = a.keys_per_split;
    const int wg_beg = 4 * (int)blockIdx.x * kps;
    // The queries' split-K partial sums are read before anything waits for the position
    // (their addresses do not depend on it), so the two round trips overlap.  The thread's
    // rotation pairs are i = i0 + 256 n: up to NIQ for a group of several heads, one (both
    // halves together) when the group's pairs fit the 256 threads; wave 0 takes the last
    // ones, so a small group leaves it free to append.
    constexpr int NIQ = (16 * (D / 2) + 255) / 256;
    const int i0 = (tid + 192) & 255;
    const int npairs = G * (D / 2);
    float qsum[2 * NIQ];
    {
        const int Nqkv = (a.nh + 2 * a.nkv) * D;
        const int64_t pstride = (int64_t)a.batch * Nqkv;
        const float* prow = a.qkv_part + (int64_t)b * Nqkv + (int64_t)kvh * G * D;
        auto col = [&](int i, int half) { return prow + (i / (D / 2)) * D + i % (D / 2) + half * (D / 2); };
        if (npairs <= 256) {
            if (i0 < npairs) {
                const float* const cols[2] = {col(i0, 0), col(i0, 1)};
                sum_parts_cols<2>(cols, a.ks, pstride, *(float(*)[2])qsum);
            }
        } else {
            const float* cols[2 * NIQ];
#pragma unroll
            for (int n = 0; n < NIQ; ++n) {
                const int i = i0 + 256 * n;
                const bool live = i < npairs;
                cols[2 * n] = live ? col(i, 0) : nullptr;
                cols[2 * n + 1] = live ? col(i, 1) : nullptr;
            }
            sum_parts_cols<2 * NIQ>(cols, a.ks, pstride, qsum);
        }
    }
    if (wg_beg >= len) return;                         // the whole workgroup is past the context
    const int sp = 4 * blockIdx.x + w;
    const int k_beg = sp * kps;
    const int k_end = min(len, k_beg + kps);           // empty for a wave past the context
    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.kv_stride;
    const int64_t vblk0 = ((int64_t)b * a.nkv + kvh) * a.nblk;

    // All loads of a 32-key chunk, unconditional: key rows are padded to whole chunks
    // and rows past the context hold finite stale or zero values that are masked.
    auto load = [&](int base, DecChunk<D, KV8>& c) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const char* src = (const char*)a.kc + (crow0 + base + 16 * t + r) * D * (KV8 ? 1 : 2);
#pragma unroll
            for (int i = 0; i < NK; ++i) c.k[t][i] = *(const u32x4*)(src + 64 * i + 16 * g);
        }
        const int64_t vb = (vblk0 + base / VT_BLK) * D * VT_BLK;
#pragma unroll
        for (int dd = 0; dd < ND; ++dd) {
            const int64_t off = vb + (int64_t)(16 * dd + r) * VT_BLK + 8 * g;
            if constexpr (KV8) c.v[dd] = *(const u32x2*)((const int8_t*)a.vc + off);
            else c.v[dd] = *(const u32x4*)((const uint16_t*)a.vc + off);
        }
        if constexpr (KV8) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                c.ks[t] = *(const u32x2*)(a.k_scales + crow0 + base + 16 * t + 4 * g);
                c.vs[t] = *(const u32x2*)(a.v_scales + crow0 + base + 16 * t + 4 * g);
            }
        }
    };

    // The workgroup whose range holds the new position appends its k and v first (one
    // wave; the barrier below publishes the row to the other waves, and no other
    // workgroup reads that position).  Every workgroup rotates the queries of its group
    // into LDS, in the MFMA operand format.
    const int pos = len - 1;
    if (pos / (4 * kps) == (int)blockIdx.x && w == 0) append_kv<D, KV8>(a, b, kvh, pos, lane);
    {
        auto rotate = [&](int i, float u, float v) {
            const int c = i / (D / 2), j = i % (D / 2);
            const float cs = a.cos_t[(int64_t)pos * (D / 2) + j], sn = a.sin_t[(int64_t)pos * (D / 2) + j];
            qs[c * D + j] = act_store(__fsub_rn(__fmul_rn(u, cs), __fmul_rn(v, sn)), AF);
            qs[c * D + j + D / 2] = act_store(__fadd_rn(__fmul_rn(v, cs), __fmul_rn(u, sn)), AF);
        };
        if (npairs <= 256) {
            if (i0 < npairs) rotate(i0, qsum[0], qsum[1]);
        } else {
#pragma unroll
            for (int n = 0; n < NIQ; ++n)
                if (i0 + 256 * n < npairs) rotate(i0 + 256 * n, qsum[2 * n], qsum[2 * n + 1]);
        }
    }
    __syncthreads();

    // query fragments: column c = head c of the group
    u32x4 qf[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        qf[j] = u32x4{0u, 0u, 0u, 0u};
        if (r < G) qf[j] = *(const u32x4*)(qs + r * D + qdim<D, KV8>(j, g));
    }

    f32x4 oacc[ND];
#pragma unroll
    for (int dd = 0; dd < ND; ++dd) oacc[dd] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    auto compute = [&](int base, const DecChunk<D, KV8>& c) {
        const int nk = k_end - base;                   // valid keys of the chunk (may exceed 32)
        float s[2][4];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                u32x4 kf;
                if constexpr (KV8) {
                    const u32x4 c16 = c.k[t][j >> 1];
                    const uint32_t lo = (j & 1) ? c16.z : c16.x, hi = (j & 1) ? c16.w : c16.y;
                    const u32x2 c0 = i8x4_to_f16x4(lo), c1 = i8x4_to_f16x4(hi);
                    kf = u32x4{c0.x, c0.y, c1.x, c1.y};
                } else {
                    kf = c.k[t][j];
                }
                acc = mfma16<AF>(kf, qf[j], acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = 16 * t + 4 * g + i;
                float v = acc[i] * a.scale;
                if constexpr (KV8) v *= h2f((uint16_t)((i < 2 ? c.ks[t].x : c.ks[t].y) >> (16 * (i & 1))));
                s[t][i] = key < nk ? v : -INFINITY;
            }
        }
        // ---- online softmax for this lane's head column
        float mx = s[0][0];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[t][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx);
        const float al = __expf(m_run - m_new);       // 0 on the first chunk
        float ps = 0.f;
        uint32_t pw[4];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            float p[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p[i] = __expf(s[t][i] - m_new);     // masked keys: exp(-inf) = 0
                ps += p[i];
                if constexpr (KV8) p[i] *= h2f((uint16_t)((i < 2 ? c.vs[t].x : c.vs[t].y) >> (16 * (i & 1))));
            }
            // slots 8 g + 4 t + i of the value block hold key 16 t + 4 g + i
            pw[2 * t] = (uint32_t)act_store(p[0], AF) | ((uint32_t)act_store(p[1], AF) << 16);
            pw[2 * t + 1] = (uint32_t)act_store(p[2], AF) | ((uint32_t)act_store(p[3], AF) << 16);
        }
        ps += __shfl_xor(ps, 16, 64);
        ps += __shfl_xor(ps, 32, 64);
        l_run = l_run * al + ps;
        m_run = m_new;
        const u32x4 pf = u32x4{pw[0], pw[1], pw[2], pw[3]};
#pragma unroll
        for (int dd = 0; dd < ND; ++dd) {
            u32x4 vf;
            if constexpr (KV8) {
                const u32x2 c0 = i8x4_to_f16x4(c.v[dd].x), c1 = i8x4_to_f16x4(c.v[dd].y);
                vf = u32x4{c0.x, c0.y, c1.x, c1.y};
            } else {
                vf = c.v[dd];
            }
            oacc[dd] *= al;
            oacc[dd] = mfma16<AF>(vf, pf, oacc[dd]);
        }
    };

    // the wave's chunks through a ring of PD register sets: PD chunks of loads in flight
    // while one is multiplied.  Every trip of the main loop issues its loads unconditionally
    // (past the wave's range: its last chunk again, never used), so the compiler's wait
    // counts stay exact; the last nch % PD chunks follow without loads.
    constexpr int PD = DecChunk<D, KV8>::PD;
    const int nch = k_beg < k_end ? (k_end - k_beg + VT_BLK - 1) / VT_BLK : 0;
    if (nch > 0) {
        DecChunk<D, KV8> cr[PD];
#pragma unroll
        for (int p = 0; p < PD; ++p) load(k_beg + VT_BLK * min(p, nch - 1), cr[p]);
        int i = 0;
        for (; i + PD <= nch; i += PD) {
#pragma unroll
            for (int p = 0; p < PD; ++p) {
                compute(k_beg + VT_BLK * (i + p), cr[p]);
                load(k_beg + VT_BLK * min(i + p + PD, nch - 1), cr[p]);
            }
        }
#pragma unroll
        for (int p = 0; p < PD - 1; ++p)
            if (i + p < nch) compute(k_beg + VT_BLK * (i + p), cr[p]);
    }

    // ---- merge the 4 splits of the workgroup: lane (c, g) holds dims 16 dd + 4 g + i of head c
    if (g == 0) { mw[w][r] = m_run; lw[w][r] = l_run; }
#pragma unroll
    for (int dd = 0; dd < ND; ++dd) *(f32x4*)(&ow[w][r * D + 16 * dd + 4 * g]) = oacc[dd];
    __syncthreads();
    const int nsw = (nsplit + 3) / 4;                  // workgroup partials per head
    for (int i = tid; i < G * D; i += 256) {
        const int c = i / D, dd = i % D;
        float m = -INFINITY;
#pragma unroll
        for (int v = 0; v < 4; ++v) m = fmaxf(m, mw[v][c]);
        float l = 0.f, o = 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float e = mw[v][c] == -INFINITY ? 0.f : __expf(mw[v][c] - m);
            l += lw[v][c] * e;
            o += ow[v][c * D + dd] * e;
        }
        const int hg = kvh * G + c;
        if (nsw == 1) {
            a.out[((int64_t)b * a.nh + hg) * D + dd] = act_store(bfround(o / l), a.out_fmt);
        } else {
            float* dst = a.ws + (((int64_t)b * a.nh + hg) * nsw + blockIdx.x) * (D + 4);
            dst[dd] = o;
            if (dd == 0) { dst[D] = m; dst[D + 1] = l; }
        }
    }
}

// One workgroup of D threads per (head, sequence): log-sum-exp merge of the
// workgroup partials.  Up to eight partials: their m, l and o values load together (one
// memory round trip); more go eight at a time, maxima first.  Sums in partial order.
template <int D>
__global__ void __launch_bounds__(D) attn_merge_kernel(AttnDecArgs a, int nsw) {
    const int h = blockIdx.x, b = blockIdx.y, i = threadIdx.x;
    const int len = *a.d_pos + 1;
    const int kpw = 4 * a.keys_per_split;
    const int nv = (len + kpw - 1) / kpw;
    const float* src = a.ws + ((int64_t)b * a.nh + h) * nsw * (D + 4);
    float m = -INFINITY, l = 0.f, o = 0.f;
    if (nv <= 8) {
        float mc[8], lc[8], oc[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const float* q = src + c * (D + 4);
            mc[c] = c < nv ? q[D] : -INFINITY;
            lc[c] = c < nv ? q[D + 1] : 0.f;
            oc[c] = c < nv ? q[i] : 0.f;
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) m = fmaxf(m, mc[c]);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            if (c >= nv) break;
            const float e = __expf(mc[c] - m);
            l += lc[c] * e;
            o += oc[c] * e;
        }
    } else {
        for (int c0 = 0; c0 < nv; c0 += 8) {
            float mc[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) mc[c] = c0 + c < nv ? src[(c0 + c) * (D + 4) + D] : -INFINITY;
#pragma unroll
            for (int c = 0; c < 8; ++c) m = fmaxf(m, mc[c]);
        }
        for (int c0 = 0; c0 < nv; c0 += 8) {
            float mc[8], lc[8], oc[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const float* q = src + (c0 + c) * (D + 4);
                mc[c] = c0 + c < nv ? q[D] : 0.f;
                lc[c] = c0 + c < nv ? q[D + 1] : 0.f;
                oc[c] = c0 + c < nv ? q[i] : 0.f;
            }
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                if (c0 + c >= nv) break;
                const float e = __expf(mc[c] - m);
                l += lc[c] * e;
                o += oc[c] * e;
            }
        }
    }
    a.out[((int64_t)b * a.nh + h) * D + i] = act_store(bfround(o / l), a.out_fmt);
}

// Splits of the context: about 1024 waves over all (sequence, kv head) pairs for a
// batch (long waves keep their chunk loads pipelined), fewer for one sequence (fewer
// partials for the consumer to merge), at least one 32-key block each and four
// splits per pair when the context has four blocks.  The grid depends only on the
// capacity, so a captured graph replays at every position.
void attn_decode_split(int max_seq, int B, int nkv, int group, int* nsplit, int* keys_per_split) {
    (void)group;
#ifndef FP_ATTN_WAVES
#define FP_ATTN_WAVES 1024
#endif
    const int target = B == 1 ? 512 : FP_ATTN_WAVES;
    const int want = (target + B * nkv - 1) / (B * nkv);
    const int blocks = (max_seq + VT_BLK - 1) / VT_BLK;
    int ns = want < blocks ? want : blocks;
    // at least the four splits a workgroup holds (its waves would idle otherwise)
    if (ns < 4) ns = blocks < 4 ? blocks : 4;
    if (ns < 1) ns = 1;
    const int bps = (blocks + ns - 1) / ns;
    *keys_per_split = bps * VT_BLK;
    *nsplit = (max_seq + *keys_per_split - 1) / *keys_per_split;
}

// Workgroup partials per head the consumer merges (1: the kernel writes the output).
int attn_decode_partials(int nsplit) { return (nsplit + 3) / 4; }

int attn_decode_max_splits(int max_seq) { return (max_seq + VT_BLK - 1) / VT_BLK; }

bool attn_decode_supported(int d, int group) { return (d == 64 || d == 128) && group >= 1 && group <= 16; }

template <int D, bool KV8>
static hipError_t launch_dk(const AttnDecArgs& a, int B, int nsplit, hipStream_t st) {
    FP_LAUNCH((attn_decode_kernel<D, KV8>), dim3((nsplit + 3) / 4, a.nkv, B), dim3(256), 0, st, a, nsplit);
    hipError_t e = hipGetLastError();
    const int nsw = attn_decode_partials(nsplit);
    if (e != hipSuccess || nsw == 1 || a.skip_merge) return e;
    FP_LAUNCH(attn_merge_kernel<D>, dim3(a.nh, B), dim3(D), 0, st, a, nsw);
    return hipGetLastError();
}

hipError_t launch_attn_decode(const AttnDecArgs& a, int B, hipStream_t st) {
    const int G = a.nh / a.nkv;
    if (!attn_decode_supported(a.d, G) || a.nh % a.nkv != 0 || a.batch != B) return hipErrorInvalidValue;
    if (a.keys_per_split <= 0 || a.keys_per_split % VT_BLK != 0) return hipErrorInvalidValue;
    const int nsplit = (a.max_seq + a.keys_per_split - 1) / a.keys_per_split;
    if (a.d == 128) return a.kv_int8 ? launch_dk<128, true>(a, B, nsplit, st) : launch_dk<128, false>(a, B, nsplit, st);
    return a.kv_int8 ? launch_dk<64, true>(a, B, nsplit, st) : launch_dk<64, false>(a, B, nsplit, st);
}

}  // namespace fpk
