// Decode projections: weight-streaming skinny GEMM  part[s] = A[M, K] . W[N, K]^T
// over the split-K range s, M tokens (one per sequence): skinny_kernel for a single
// sequence (M <= 16), skinny_batch_kernel for batches (M <= 64).
//
// Decode is where the fingerprint's per-token time goes (TPOT, paper Sec. 5.3):
// every step streams all weights once, so the kernel is bound by HBM bandwidth.
// Weight-only quantisation (Sec. 3.2) shrinks those bytes; the cost the paper
// points at is converting the codes back to 16-bit values for the arithmetic.
// Here the codes go straight from a 128-bit load into MFMA operands with a few
// integer ops per dword:
//   bf16  W: 16 B per lane = 8 weights  -> 1 MFMA  (bf16 x bf16)
//   int8  W: 16 B per lane = 16 weights -> 2 MFMAs (fp16 x exact fp16 codes); the
//            row scale is applied once at the end
//   int4  W: 16 B per lane = 32 weights = a quarter of one 128-group of a row ->
//            4 MFMAs on fp16((q - z) * s)
// MFMA 16x16x32 layout: lane l supplies row (l % 16) of A and column (l % 16) of
// B, each with 8 consecutive k from the lane's k-slice (l / 16); the output lane
// holds C[4 (l/16) + i][l % 16].  A and B use the same k assignment, so the order
// of k inside a K-step is free; the int4 nibble order on the device makes nibble
// pairs come out as consecutive k.  Batches of 17 to 64 use 32x32x16 instead (see
// skinny_batch_kernel).  int4 scale / zero words are stored group-major, so the words
// of consecutive rows for one group are consecutive in memory.
//
// Weights are stored fragment-major: the 64 lanes' 16-byte operands of one 16-row
// subtile and one K-step form a contiguous 1 KiB block, and a row of blocks runs
// along K, so every wave-wide load reads 1 KiB of contiguous memory and each wave
// streams long contiguous runs.  The loads are non-temporal: each weight is read once
// per step.
//
// Workgroup = 4 waves; each wave owns NS subtiles of 16 weight rows and streams
// them over the workgroup's K-range with UNR K-steps of loads in flight (double
// buffered in registers).  The activation slice A[:, K-range] is staged once in
// LDS, transformed on the way in:
//   XF_COPY   A = X                                   (attention output)
//   XF_NORM   A = bf16(y * rsqrt(mean(y^2) + eps) * g) (RMSNorm of the layer input
//             or of h; the row's sum of squares comes as block sums)
//   XF_SWIGLU A = bf16(silu(gate) * up) from the gate|up partial sums
//   XF_MERGE  A = attention output, merged from its context splits by the exact
//             log-sum-exp identity
// so the normalisation, the activation and the merge never run as kernels of
// their own.
// In dual mode (the [gate; up] matrix) the first NS/2 subtiles of a wave read gate
// rows f and the others up rows F + f of the same f.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

template <int WF>
struct SkinnyTraits;
template <> struct SkinnyTraits<W_BF16> { static constexpr int KS = 32; static constexpr int NJ = 1; };
template <> struct SkinnyTraits<W_INT8> { static constexpr int KS = 64; static constexpr int NJ = 2; };
template <> struct SkinnyTraits<W_INT4> { static constexpr int KS = 128; static constexpr int NJ = 4; };

constexpr int SK_LDS_ELEMS = 31744;   // u16 elements of the staged activation slice (62 KiB)
constexpr int SK_PAD = 8;

template <int WF, int MT, int NS, int UNR, int XF>
__global__ void __launch_bounds__(256) skinny_kernel(SkinnyArgs a) {
    constexpr int KS = SkinnyTraits<WF>::KS;
    constexpr int NJ = SkinnyTraits<WF>::NJ;
    constexpr int KL = KS / 4;                       // k per lane group in one K-step
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    extern __shared__ __attribute__((aligned(16))) uint16_t As[];
    __shared__ float rrow[64];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int sp = blockIdx.y;
    const int kb = sp * a.krange;
    const int ke = min(a.K, kb + a.krange);
    const int klen = ke - kb;
    const int ld = a.krange + SK_PAD;               // LDS row stride (u16)

    // ---- rows of this wave's subtiles
    int row[NS];
    bool rv[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (a.dual_F > 0) {
            const int fw = blockIdx.x * (32 * NS) + w * (8 * NS);
            const int f = fw + 16 * (s % (NS / 2)) + r;
            rv[s] = f < a.dual_F;
            row[s] = (s < NS / 2 ? 0 : a.dual_F) + f;
        } else {
            row[s] = blockIdx.x * (64 * NS) + w * (16 * NS) + 16 * s + r;
            rv[s] = row[s] < a.N;
        }
    }

    // ---- weight loads of one K-step: one 1 KiB block per wave (16 rows x one K-step),
    // and for int4 the row's scale | zero << 16 word of the step's 128-input group.
    // Rows past the matrix and steps past the k-range read past the end of the buffer
    // resources (zeros, no memory access), so every load is issued unconditionally and
    // the compiler's wait counts stay exact.
    const int nrows = a.dual_F > 0 ? 2 * a.dual_F : a.N;
    const int ngr = a.K / 128;
    const __amdgpu_buffer_rsrc_t wres = buf_rsrc(a.W, (uint32_t)((nrows / 16) * a.kst * 1024));
    const __amdgpu_buffer_rsrc_t szres = buf_rsrc(a.sz, WF == W_INT4 ? (uint32_t)(ngr * nrows * 4) : 0u);
    auto load_w = [&](int kk, u32x4* dst, uint32_t* szd) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const uint32_t blk = (uint32_t)((row[s] >> 4) * a.kst + kk / KS);
            dst[s] = buf_load_nt(wres, off_or_oob(rv[s] && kk < ke, (blk * 64 + lane) * 16));
            if constexpr (WF == W_INT4)
                szd[s] = __builtin_amdgcn_raw_buffer_load_b32(
                    szres, off_or_oob(rv[s] && kk < ke, (uint32_t)((kk / 128) * nrows + row[s]) * 4u), 0, 0);
        }
    };

    // ---- activation-side loads go out before the weight loads: wait counts are in issue
    // order, so the staging below then does not wait for the weights.  Each thread takes
    // its first staged piece (and gain) and one of the rows' sum-of-squares partials.
    const int chunks = klen / 8;                     // 8-element chunks per row
    u32x4 xv0 = u32x4{0u, 0u, 0u, 0u}, gv0 = u32x4{0u, 0u, 0u, 0u};
    if constexpr (XF == XF_COPY || XF == XF_NORM) {
        if (tid < a.M * chunks) {
            const int k = kb + (tid % chunks) * 8;
            xv0 = *(const u32x4*)(a.X + (int64_t)(tid / chunks) * a.K + k);
            if constexpr (XF == XF_NORM) gv0 = *(const u32x4*)(a.gain + k);
        }
    }
    // XF_MERGE: the first piece's attention partials (the first NVP splits) likewise
    constexpr int NVP = XF == XF_MERGE ? 4 : 1;
    float pm[NVP], pl[NVP];
    float4 po0[NVP], po1[NVP];
    if constexpr (XF == XF_MERGE) {
        if (tid < a.M * chunks) {
            const int D = a.head_dim, nhd = a.K / D;
            const int k = kb + (tid % chunks) * 8, h = k / D, dd = k % D;
            const int nv = (*a.d_pos + a.att_kps) / a.att_kps;
            const float* src = a.att_ws + ((int64_t)(tid / chunks) * nhd + h) * a.att_nsplit * (D + 4);
#pragma unroll
            for (int i = 0; i < NVP; ++i)
                if (i < nv) {
                    const float* q = src + i * (D + 4);
                    pm[i] = q[D];
                    pl[i] = q[D + 1];
                    po0[i] = *(const float4*)(q + dd);
                    po1[i] = *(const float4*)(q + dd + 4);
                }
        }
    }
    // XF_SWIGLU: the first piece's gate / up partials of the first KSP splits likewise
    constexpr int KSP = XF == XF_SWIGLU ? 2 : 1;
    float4 sg0[KSP], sg1[KSP], su0[KSP], su1[KSP];
    if constexpr (XF == XF_SWIGLU) {
        if (tid < a.M * chunks) {
            const int F = a.K, k = kb + (tid % chunks) * 8;
#pragma unroll
            for (int i = 0; i < KSP; ++i)
                if (i < a.src_ks) {
                    const float* p = a.src_part + ((int64_t)i * a.M + tid / chunks) * (2 * (int64_t)F);
                    sg0[i] = *(const float4*)(p + k);
                    sg1[i] = *(const float4*)(p + k + 4);
                    su0[i] = *(const float4*)(p + F + k);
                    su1[i] = *(const float4*)(p + F + k + 4);
                }
        }
    }
    const bool ssq_lds = XF == XF_NORM && a.ssq != nullptr && a.M * a.ssq_blocks <= 256;
    float ssp = 0.f;
    if (ssq_lds && tid < a.M * a.ssq_blocks) ssp = a.ssq[tid];

    u32x4 wa[UNR][NS], wb[UNR][NS];
    uint32_t sza[UNR][NS], szb[UNR][NS];
#pragma unroll
    for (int u = 0; u < UNR; ++u) load_w(kb + u * KS, wa[u], sza[u]);

    // ---- stage the activation slice (with its transform) into LDS
    if constexpr (XF == XF_NORM) {
        if (ssq_lds) {
            __shared__ float ssl[256];
            ssl[tid] = ssp;
            __syncthreads();
            if (tid < a.M) {
                float ss = 0.f;
                for (int b = 0; b < a.ssq_blocks; ++b) ss += ssl[tid * a.ssq_blocks + b];
                rrow[tid] = 1.0f / __fsqrt_rn(ss / (float)a.K + a.eps);
            }
        } else if (a.ssq != nullptr) {
            if (tid < a.M) {
                float ss = 0.f;
                for (int b = 0; b < a.ssq_blocks; ++b) ss += a.ssq[tid * a.ssq_blocks + b];
                rrow[tid] = 1.0f / __fsqrt_rn(ss / (float)a.K + a.eps);
            }
        } else {   // small batches: sum the squares of the whole rows here
            __shared__ float red[16];
            for (int m = 0; m < a.M; ++m) {
                float ss = 0.f;
                for (int k = tid * 8; k < a.K; k += 256 * 8) {
                    const u32x4 v = *(const u32x4*)(a.X + (int64_t)m * a.K + k);
                    const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float e0 = __uint_as_float(vv[j] << 16), e1 = __uint_as_float(vv[j] & 0xFFFF0000u);
                        ss += e0 * e0 + e1 * e1;
                    }
                }
                ss = block_sum(ss, red);
                if (tid == 0) rrow[m] = 1.0f / __fsqrt_rn(ss / (float)a.K + a.eps);
            }
        }
        __syncthreads();
    }
    {
        // the thread's first piece uses the values loaded before the weights; the loop
        // takes the rest (several per thread only for long slices)
        auto stage = [&](int c, bool pre) {
            const int m = c / chunks, kc = (c % chunks) * 8;
            const int k = kb + kc;
            uint32_t o[4];
            if constexpr (XF == XF_COPY) {
                const u32x4 v = pre ? xv0 : *(const u32x4*)(a.X + (int64_t)m * a.K + k);
                o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
            } else if constexpr (XF == XF_NORM) {
                const u32x4 v = pre ? xv0 : *(const u32x4*)(a.X + (int64_t)m * a.K + k);
                const u32x4 gg = pre ? gv0 : *(const u32x4*)(a.gain + k);
                const uint32_t vv[4] = {v.x, v.y, v.z, v.w}, gv[4] = {gg.x, gg.y, gg.z, gg.w};
                const float rm = rrow[m];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float e0 = bfround(__uint_as_float(vv[j] << 16) * rm * __uint_as_float(gv[j] << 16));
                    const float e1 = bfround(__uint_as_float(vv[j] & 0xFFFF0000u) * rm * __uint_as_float(gv[j] & 0xFFFF0000u));
                    o[j] = (uint32_t)act_store(e0, AF) | ((uint32_t)act_store(e1, AF) << 16);
                }
            } else if constexpr (XF == XF_MERGE) {
                // log-sum-exp merge of the context splits of head k / head_dim
                const int D = a.head_dim, nhd = a.K / D;
                const int h = k / D, dd = k % D;
                const int nv = (*a.d_pos + a.att_kps) / a.att_kps;     // splits holding keys
                const float* src = a.att_ws + ((int64_t)m * nhd + h) * a.att_nsplit * (D + 4);
                float mx = -INFINITY;
#pragma unroll
                for (int i = 0; i < NVP; ++i)
                    if (i < nv) mx = fmaxf(mx, pre ? pm[i] : src[i * (D + 4) + D]);
                for (int sp2 = NVP; sp2 < nv; ++sp2) mx = fmaxf(mx, src[sp2 * (D + 4) + D]);
                float L = 0.f, ov[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) ov[j] = 0.f;
                auto add = [&](float mv, float lv, float4 o0, float4 o1) {
                    const float e = __expf(mv - mx);
                    L += lv * e;
                    ov[0] += o0.x * e; ov[1] += o0.y * e; ov[2] += o0.z * e; ov[3] += o0.w * e;
                    ov[4] += o1.x * e; ov[5] += o1.y * e; ov[6] += o1.z * e; ov[7] += o1.w * e;
                };
#pragma unroll
                for (int i = 0; i < NVP; ++i)
                    if (i < nv) {
                        if (pre) {
                            add(pm[i], pl[i], po0[i], po1[i]);
                        } else {
                            const float* q = src + i * (D + 4);
                            add(q[D], q[D + 1], *(const float4*)(q + dd), *(const float4*)(q + dd + 4));
                        }
                    }
                for (int sp2 = NVP; sp2 < nv; ++sp2) {
                    const float* q = src + sp2 * (D + 4);
                    add(q[D], q[D + 1], *(const float4*)(q + dd), *(const float4*)(q + dd + 4));
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    o[j] = (uint32_t)act_store(bfround(ov[2 * j] / L), AF) |
                           ((uint32_t)act_store(bfround(ov[2 * j + 1] / L), AF) << 16);
            } else {   // XF_SWIGLU: k indexes f; partials [src_ks, M, 2F]
                const int F = a.K;
                float gs[8], us[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) { gs[j] = 0.f; us[j] = 0.f; }
                auto add = [&](float4 g0, float4 g1, float4 u0, float4 u1) {
                    gs[0] += g0.x; gs[1] += g0.y; gs[2] += g0.z; gs[3] += g0.w;
                    gs[4] += g1.x; gs[5] += g1.y; gs[6] += g1.z; gs[7] += g1.w;
                    us[0] += u0.x; us[1] += u0.y; us[2] += u0.z; us[3] += u0.w;
                    us[4] += u1.x; us[5] += u1.y; us[6] += u1.z; us[7] += u1.w;
                };
                auto part = [&](int s2) { return a.src_part + ((int64_t)s2 * a.M + m) * (2 * (int64_t)F); };
#pragma unroll
                for (int i = 0; i < KSP; ++i)
                    if (i < a.src_ks) {
                        if (pre) {
                            add(sg0[i], sg1[i], su0[i], su1[i]);
                        } else {
                            const float* p = part(i);
                            add(*(const float4*)(p + k), *(const float4*)(p + k + 4), *(const float4*)(p + F + k),
                                *(const float4*)(p + F + k + 4));
                        }
                    }
                // the rest two splits at a time (one memory round trip per pair), added in order
                int s2 = KSP;
                for (; s2 + 1 < a.src_ks; s2 += 2) {
                    const float* p = part(s2);
                    const float* p1 = part(s2 + 1);
                    const float4 g0 = *(const float4*)(p + k), g1 = *(const float4*)(p + k + 4);
                    const float4 u0 = *(const float4*)(p + F + k), u1 = *(const float4*)(p + F + k + 4);
                    const float4 h0 = *(const float4*)(p1 + k), h1 = *(const float4*)(p1 + k + 4);
                    const float4 v0 = *(const float4*)(p1 + F + k), v1 = *(const float4*)(p1 + F + k + 4);
                    add(g0, g1, u0, u1);
                    add(h0, h1, v0, v1);
                }
                if (s2 < a.src_ks) {
                    const float* p = part(s2);
                    add(*(const float4*)(p + k), *(const float4*)(p + k + 4), *(const float4*)(p + F + k),
                        *(const float4*)(p + F + k + 4));
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    o[j] = (uint32_t)act_store(bfround(silu_f(gs[2 * j]) * us[2 * j]), AF) |
                           ((uint32_t)act_store(bfround(silu_f(gs[2 * j + 1]) * us[2 * j + 1]), AF) << 16);
            }
            *(u32x4*)(As + m * ld + kc) = u32x4{o[0], o[1], o[2], o[3]};
        };
        if (tid < a.M * chunks) stage(tid, true);
        for (int c = tid + 256; c < a.M * chunks; c += 256) stage(c, false);
    }
    __syncthreads();

    // ---- stream the weights
    f32x4 acc[MT][NS];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};
    bool mv[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) mv[t] = (16 * t + r) < a.M;

    auto compute = [&](int kk, const u32x4* wv, const uint32_t* sz) {
        if (kk >= ke) return;
        const bool kin = kk + KL * g < ke;
        u32x4 bop[NJ][NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if constexpr (WF == W_BF16) {
                bop[0][s] = wv[s];
            } else if constexpr (WF == W_INT8) {
                const u32x2 c0 = i8x4_to_f16x4(wv[s].x), c1 = i8x4_to_f16x4(wv[s].y);
                const u32x2 c2 = i8x4_to_f16x4(wv[s].z), c3 = i8x4_to_f16x4(wv[s].w);
                bop[0][s] = u32x4{c0.x, c0.y, c1.x, c1.y};
                bop[1][s] = u32x4{c2.x, c2.y, c3.x, c3.y};
            } else {
                const float sc = h2f((uint16_t)(sz[s] & 0xFFFFu)), zz = h2f((uint16_t)(sz[s] >> 16));
                const _Float16 bz = (_Float16)(1024.0f + zz);
                const f16x2 bias = {bz, bz};
                const _Float16 sh = (_Float16)sc;
                const f16x2 s2 = {sh, sh};
                const uint32_t wd[4] = {wv[s].x, wv[s].y, wv[s].z, wv[s].w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const u32x4 q = i4x8_to_f16x8(wd[j], bias);
                    bop[j][s] = u32x4{mul_h2(q.x, s2), mul_h2(q.y, s2), mul_h2(q.z, s2), mul_h2(q.w, s2)};
                }
            }
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            int koff;
            if constexpr (WF == W_BF16) koff = kk + 8 * g;
            else if constexpr (WF == W_INT8) koff = kk + 16 * g + 8 * j;
            else koff = kk + 32 * g + 8 * j;
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                u32x4 av = u32x4{0u, 0u, 0u, 0u};
                if (mv[t] && kin) av = *(const u32x4*)(As + (16 * t + r) * ld + (koff - kb));
#pragma unroll
                for (int s = 0; s < NS; ++s) acc[t][s] = mfma16<AF>(av, bop[j][s], acc[t][s]);
            }
        }
    };

    for (int base = kb; base < ke; base += 2 * UNR * KS) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) load_w(base + (UNR + u) * KS, wb[u], szb[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) compute(base + u * KS, wa[u], sza[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) load_w(base + (2 * UNR + u) * KS, wa[u], sza[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) compute(base + (UNR + u) * KS, wb[u], szb[u]);
    }

    // ---- partial sums of this split
    const int ncols = a.dual_F > 0 ? 2 * a.dual_F : a.N;
    float* out = a.part + (int64_t)sp * a.M * ncols;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (!rv[s]) continue;
        float rs = 1.f;
        if constexpr (WF == W_INT8) rs = h2f(a.scales[row[s]]);
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = 16 * t + 4 * g + i;
                if (m < a.M) out[(int64_t)m * ncols + row[s]] = acc[t][s][i] * rs;
            }
    }
}

// ---------------------------------------------------------------------------
// Batches (M > 1 tokens, one per sequence): the activation is a real M x K operand,
// so it is not staged whole -- that would cap the k-range per workgroup at the LDS
// size and force a split-K factor (and partial-sum traffic) that grows with M.
// Instead the workgroup walks its k-range in chunks of 128 (one int4 group, two
// int8 or four bf16 K-steps).  Activation chunks are loaded into registers PD
// chunks ahead and written to one of two LDS buffers one chunk ahead (rows of 256 B,
// 16-byte pieces XOR-swizzled by the row so MFMA fragment reads are free of bank
// conflicts); weight fragments (and int4 scale / zero words) run PD chunks ahead in
// registers.  The workgroup synchronises with a bare s_barrier after the LDS
// writes, so the global loads in flight are not drained at every chunk.  The
// split-K factor only has to fill the GPU.
constexpr int SB_KC = 128;              // k per activation chunk (one int4 group)
#ifndef SKINNY_I4_POST
#define SKINNY_I4_POST 1                // int4: scale the group sums instead of the weights
#endif
#ifndef SKINNY_BATCH_PD
#define SKINNY_BATCH_PD 4
#endif
constexpr int SB_PD = SKINNY_BATCH_PD;  // chunks of loads in flight (even: the LDS buffer is the chunk's parity)
static_assert(SB_PD >= 2 && SB_PD % 2 == 0, "load depth");

// M32: 32x32x16 MFMA (batches of 17 to 64: MT = 2 or 4 sixteen-row tiles of the
// activation chunk).  Each wave's two 16-row weight blocks form one 32-column tile; lane
// l takes the weight row (l % 32) and, of its block's fragment pieces, the two whose
// k-groups are (l / 32) and (l / 32) + 2.  The k order inside an MFMA only has to agree
// between the two operands, so the activation fragments follow the pieces' k.
template <int WF, int MT, int NS, int NWV, bool M32>
__global__ void __launch_bounds__(64 * NWV, 1) skinny_batch_kernel(SkinnyArgs a) {
    static_assert(!M32 || (NS == 2 && MT % 2 == 0), "32-row tiles: two blocks per wave, whole 32-row activation tiles");
    constexpr int NT = 64 * NWV;                     // threads
    constexpr int NPA = (256 * MT + NT - 1) / NT;    // activation pieces per thread
    constexpr int KS = SkinnyTraits<WF>::KS;
    constexpr int NJ = SkinnyTraits<WF>::NJ;
    constexpr int SPC = SB_KC / KS;                  // K-steps per chunk
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    constexpr int ABUF = 16 * MT * 256;              // bytes of one activation chunk
    // chunks of loads in flight: four for int8; two for int4 (measured faster: its chunks
    // are half the bytes and its unpacking keeps the waves busy) and bf16 (four K-steps
    // of weights per chunk)
    constexpr int PD = WF == W_INT8 ? SB_PD : 2;
    __shared__ __attribute__((aligned(1024))) char As[2 * ABUF];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int kb = blockIdx.y * a.krange;
    const int ke = min(a.K, kb + a.krange);
    const int nch = (ke - kb + SB_KC - 1) / SB_KC;

    // weight rows of this wave's subtiles (rows past the matrix are clamped for the
    // loads and never stored)
    int row[NS];
    bool rv[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (a.dual_F > 0) {
            const int fw = blockIdx.x * (NWV * 8 * NS) + w * (8 * NS);
            constexpr int HS = NS / 2 > 0 ? NS / 2 : 1;   // dual tiling needs NS even (the launcher ensures it)
            const int f = fw + 16 * (s % HS) + r;
            rv[s] = f < a.dual_F;
            row[s] = (s < HS ? 0 : a.dual_F) + min(f, a.dual_F - 1);
        } else {
            const int n = blockIdx.x * (NWV * 16 * NS) + w * (16 * NS) + 16 * s + r;
            rv[s] = n < a.N;
            row[s] = min(n, a.N - 1);
        }
    }

    const int h32 = lane >> 5, bsel = (lane & 31) >> 4;   // M32: k half, block of the lane's row
    const int myrow = row[bsel & (NS - 1)];
    const bool myrv = rv[bsel & (NS - 1)];
    // activation chunk ci: thread piece c = tid + NT i is row c / 16, LDS slot c % 16,
    // which holds the row's 16-byte piece slot ^ (row % 16)
    // Loads are unconditional (clamped addresses): rows past M only feed output rows
    // that are never stored.  Pieces past the k-range (only in a ragged last chunk; the
    // weights there are padding or clamped copies) are zeroed when the chunk is written
    // to LDS, after its loads have landed, so no load has to be waited for early.
    auto load_a = [&](int ci, u32x4* ra) {
        const int kbase = kb + min(ci, nch - 1) * SB_KC;
#pragma unroll
        for (int i = 0; i < NPA; ++i) {
            const int c = tid + NT * i;
            const int rr = min(c >> 4, 16 * MT - 1), slot = c & 15;
            const int k = kbase + ((slot ^ (rr & 15)) * 8);
            ra[i] = *(const u32x4*)(a.X + (int64_t)min(rr, a.M - 1) * a.K + min(k, a.K - 8));
        }
    };
    auto store_a = [&](char* buf, const u32x4* ra, int ci) {
        const int kbase = kb + min(ci, nch - 1) * SB_KC;
        const bool ragged = kbase + SB_KC > ke;
#pragma unroll
        for (int i = 0; i < NPA; ++i) {
            const int c = tid + NT * i;
            u32x4 v = ra[i];
            if (ragged) {
                const int rr = min(c >> 4, 16 * MT - 1), slot = c & 15;
                if (kbase + ((slot ^ (rr & 15)) * 8) >= ke) v = u32x4{0u, 0u, 0u, 0u};
            }
            if ((256 * MT) % NT == 0 || c < 256 * MT) *(u32x4*)(buf + c * 16) = v;
        }
    };
    // weight fragments of chunk ci; chunks past the range read past the end of the
    // buffer resource (zeros, no memory traffic)
    const int nrows = a.dual_F > 0 ? 2 * a.dual_F : a.N;
    const __amdgpu_buffer_rsrc_t wres = buf_rsrc(a.W, (uint32_t)((nrows / 16) * a.kst * 1024));
    auto load_w = [&](int ci, u32x4 (*wv)[NS], uint32_t* sz) {
        const int cc = min(ci, nch - 1);
        const int st0 = (kb + cc * SB_KC) / KS;
#pragma unroll
        for (int u = 0; u < SPC; ++u)
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                if constexpr (M32) {
                    // piece (r, group h32 + 2 s) of the block holding the lane's row
                    const uint32_t blk = (uint32_t)((myrow >> 4) * a.kst + min(st0 + u, a.kst - 1));
                    wv[u][s] = buf_load_nt(wres, off_or_oob_uniform(ci < nch, (blk * 64 + r + 16 * (h32 + 2 * s)) * 16));
                } else {
                    const uint32_t blk = (uint32_t)((row[s] >> 4) * a.kst + min(st0 + u, a.kst - 1));
                    wv[u][s] = buf_load_nt(wres, off_or_oob_uniform(ci < nch, (blk * 64 + lane) * 16));
                }
            }
        if constexpr (WF == W_INT4) {
            if constexpr (M32) {
                sz[0] = a.sz[(int64_t)st0 * nrows + myrow];
            } else {
#pragma unroll
                for (int s = 0; s < NS; ++s) sz[s] = a.sz[(int64_t)st0 * nrows + row[s]];
            }
        }
    };

    f32x4 acc[MT][NS];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    // A chunk is four 32-k MFMA sub-steps.  Sub-step m's B operands (dequantised
    // weights) and A fragments (LDS) are formed while sub-step m - 1's MFMAs run: the
    // scheduler is asked for one MFMA, a share of the next sub-step's unpacking and
    // (for the first MT MFMAs) one LDS read, in turn, so the matrix pipe, the vector
    // ALU and LDS overlap within a wave.
    constexpr int NSUB = SB_KC / 32;
    constexpr bool I4_POST = WF == W_INT4 && SKINNY_I4_POST;
    auto a_frag = [&](const char* Ab, int m, int t) {
        int koff;
        if constexpr (WF == W_BF16) koff = 32 * m + 8 * g;
        else if constexpr (WF == W_INT8) koff = 64 * (m >> 1) + 16 * g + 8 * (m & 1);
        else koff = 32 * g + 8 * m;
        const int piece = koff >> 3;
        const int rr = 16 * t + r;
        return *(const u32x4*)(Ab + rr * 256 + ((piece ^ (rr & 15)) << 4));
    };
    auto b_op = [&](const u32x4 (*wv)[NS], const uint32_t* sz, int m, int s) {
        if constexpr (WF == W_BF16) {
            return wv[m][s];
        } else if constexpr (WF == W_INT8) {
            const u32x4 w = wv[m >> 1][s];
            const uint32_t d0 = (m & 1) ? w.z : w.x, d1 = (m & 1) ? w.w : w.y;
            const u32x2 c0 = i8x4_to_f16x4(d0), c1 = i8x4_to_f16x4(d1);
            return u32x4{c0.x, c0.y, c1.x, c1.y};
        } else {
            const _Float16 bz = (_Float16)(1024.0f + h2f((uint16_t)(sz[s] >> 16)));
            const f16x2 bias = {bz, bz};
            const _Float16 sh = __builtin_bit_cast(_Float16, (uint16_t)(sz[s] & 0xFFFFu));
            const f16x2 s2 = {sh, sh};
            const u32x4 w = wv[0][s];
            const uint32_t d = m == 0 ? w.x : m == 1 ? w.y : m == 2 ? w.z : w.w;
            const u32x4 q = i4x8_to_f16x8(d, bias);
            if constexpr (I4_POST) return q;             // exact q - z; the group scale is applied to the sums
            return u32x4{mul_h2(q.x, s2), mul_h2(q.y, s2), mul_h2(q.z, s2), mul_h2(q.w, s2)};
        }
    };
    constexpr int VALU_PER_B = WF == W_BF16 ? 0 : (WF == W_INT8 ? 10 : (I4_POST ? 12 : 16));   // per B operand
    constexpr int NMF = MT * NS;                                              // MFMAs per sub-step
    constexpr int VPS = (VALU_PER_B * NS + NMF - 1) / NMF;                     // VALU per MFMA slot
    auto compute = [&](const char* Ab, const u32x4 (*wv)[NS], const uint32_t* sz) {
        u32x4 av[2][MT], bq[2][NS];
        // int4 with I4_POST: a chunk is one 128-input group, summed over exact q - z into
        // fresh accumulators and scaled once per group in fp32
        f32x4 grp[I4_POST ? MT : 1][I4_POST ? NS : 1];
#pragma unroll
        for (int t = 0; t < MT; ++t) av[0][t] = a_frag(Ab, 0, t);
#pragma unroll
        for (int s = 0; s < NS; ++s) bq[0][s] = b_op(wv, sz, 0, s);
#pragma unroll
        for (int m = 0; m < NSUB; ++m) {
            const int c = m & 1, n = c ^ 1;
            __builtin_amdgcn_sched_barrier(0);
            if (m + 1 < NSUB) {
#pragma unroll
                for (int t = 0; t < MT; ++t) av[n][t] = a_frag(Ab, m + 1, t);
#pragma unroll
                for (int s = 0; s < NS; ++s) bq[n][s] = b_op(wv, sz, m + 1, s);
            }
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int s = 0; s < NS; ++s) {
                    if constexpr (I4_POST)
                        grp[t][s] = mfma16<AF>(av[c][t], bq[c][s], m == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : grp[t][s]);
                    else
                        acc[t][s] = mfma16<AF>(av[c][t], bq[c][s], acc[t][s]);
                }
            if (m + 1 < NSUB) {
#pragma unroll
                for (int i = 0; i < NMF; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);          // one MFMA
                    if (i < MT) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
                    if (VPS > 0) __builtin_amdgcn_sched_group_barrier(0x002, VPS, 0); // unpacking
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (I4_POST) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const float sc = h2f((uint16_t)(sz[s] & 0xFFFFu));
#pragma unroll
                for (int t = 0; t < MT; ++t) acc[t][s] += grp[t][s] * sc;
            }
        }
    };
    // M32: eight 16-k MFMA steps per chunk.  Step j of the lane's data (h = l / 32):
    // bf16 K-step j / 2, piece j % 2, k 16 j + 8 h; int8 K-step j / 4, piece (j / 2) % 2,
    // half j % 2, k 64 (j / 4) + 32 ((j / 2) % 2) + 16 h + 8 (j % 2); int4 piece j / 4,
    // dword j % 4, k 64 (j / 4) + 32 h + 8 (j % 4).
    constexpr int MT32 = MT / 2;
    f32x16 acc32[M32 ? MT32 : 1];
#pragma unroll
    for (int t = 0; t < (M32 ? MT32 : 1); ++t) acc32[t] = f32x16{};
    auto a_frag32 = [&](const char* Ab, int j, int t) {
        int koff;
        if constexpr (WF == W_BF16) koff = 16 * j + 8 * h32;
        else if constexpr (WF == W_INT8) koff = 64 * (j >> 2) + 32 * ((j >> 1) & 1) + 16 * h32 + 8 * (j & 1);
        else koff = 64 * (j >> 2) + 32 * h32 + 8 * (j & 3);
        const int piece = koff >> 3;
        const int rr = 32 * t + (lane & 31);
        return *(const u32x4*)(Ab + rr * 256 + ((piece ^ (rr & 15)) << 4));
    };
    auto b_op32 = [&](const u32x4 (*wv)[NS], const uint32_t* sz, int j) {
        if constexpr (WF == W_BF16) {
            return wv[j >> 1][(j & 1) & (NS - 1)];
        } else if constexpr (WF == W_INT8) {
            const u32x4 w = wv[j >> 2][((j >> 1) & 1) & (NS - 1)];
            const uint32_t d0 = (j & 1) ? w.z : w.x, d1 = (j & 1) ? w.w : w.y;
            const u32x2 c0 = i8x4_to_f16x4(d0), c1 = i8x4_to_f16x4(d1);
            return u32x4{c0.x, c0.y, c1.x, c1.y};
        } else {
            const _Float16 bz = (_Float16)(1024.0f + h2f((uint16_t)(sz[0] >> 16)));
            const f16x2 bias = {bz, bz};
            const _Float16 sh = __builtin_bit_cast(_Float16, (uint16_t)(sz[0] & 0xFFFFu));
            const f16x2 s2 = {sh, sh};
            const u32x4 w = wv[0][(j >> 2) & (NS - 1)];
            const int dd = j & 3;
            const uint32_t d = dd == 0 ? w.x : dd == 1 ? w.y : dd == 2 ? w.z : w.w;
            const u32x4 q = i4x8_to_f16x8(d, bias);
            if constexpr (I4_POST) return q;
            return u32x4{mul_h2(q.x, s2), mul_h2(q.y, s2), mul_h2(q.z, s2), mul_h2(q.w, s2)};
        }
    };
    constexpr int VPS32 = M32 ? (VALU_PER_B + MT32 - 1) / (MT32 > 0 ? MT32 : 1) : 0;   // VALU per MFMA slot
    auto compute32 = [&](const char* Ab, const u32x4 (*wv)[NS], const uint32_t* sz) {
        u32x4 av[2][MT32 > 0 ? MT32 : 1], bq[2];
        f32x16 grp[I4_POST && MT32 > 0 ? MT32 : 1];
#pragma unroll
        for (int t = 0; t < MT32; ++t) av[0][t] = a_frag32(Ab, 0, t);
        bq[0] = b_op32(wv, sz, 0);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int c = j & 1, n = c ^ 1;
            __builtin_amdgcn_sched_barrier(0);
            if (j + 1 < 8) {
#pragma unroll
                for (int t = 0; t < MT32; ++t) av[n][t] = a_frag32(Ab, j + 1, t);
                bq[n] = b_op32(wv, sz, j + 1);
            }
#pragma unroll
            for (int t = 0; t < MT32; ++t) {
                if constexpr (I4_POST) grp[t] = mfma32<AF>(av[c][t], bq[c], j == 0 ? f32x16{} : grp[t]);
                else acc32[t] = mfma32<AF>(av[c][t], bq[c], acc32[t]);
            }
            if (j + 1 < 8) {
#pragma unroll
                for (int i = 0; i < MT32; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);            // one LDS read
                    if (VPS32 > 0) __builtin_amdgcn_sched_group_barrier(0x002, VPS32, 0);   // unpacking
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (I4_POST) {
            const float sc = h2f((uint16_t)(sz[0] & 0xFFFFu));
#pragma unroll
            for (int t = 0; t < MT32; ++t) acc32[t] += grp[t] * sc;
        }
    };
    // LDS writes done, then a bare barrier (no drain of the global loads in flight)
    auto barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

    // register rings: slot i % PD holds chunk i's weights and activation pieces
    u32x4 wr[PD][SPC][NS];
    uint32_t szr[PD][NS];
    u32x4 ra[PD][NPA];
#pragma unroll
    for (int i = 0; i < PD; ++i) load_a(i, ra[i]);
#pragma unroll
    for (int i = 0; i < PD; ++i) load_w(i, wr[i], szr[i]);
    store_a(As, ra[0], 0);
    load_a(PD, ra[0]);
    barrier();
    // one chunk: multiply it out of LDS buffer p & 1, refill ring slot p with chunk
    // ci + PD, move chunk ci + 1 into the other LDS buffer (whose last reader was
    // chunk ci - 1: every wave has passed the barrier since) and refill its ring slot
    auto step = [&](int ci, int p) {
        if constexpr (M32) compute32(As + (p & 1) * ABUF, wr[p], szr[p]);
        else compute(As + (p & 1) * ABUF, wr[p], szr[p]);
        load_w(ci + PD, wr[p], szr[p]);
        const int q = (p + 1) % PD;
        store_a(As + ((p + 1) & 1) * ABUF, ra[q], ci + 1);
        load_a(ci + 1 + PD, ra[q]);
        barrier();
    };
    // whole groups of PD chunks run without a branch, so the compiler's wait counts
    // stay exact around the loop; the last nch % PD chunks follow
    int ci0 = 0;
    for (; ci0 + PD <= nch; ci0 += PD) {
#pragma unroll
        for (int p = 0; p < PD; ++p) step(ci0 + p, p);
    }
#pragma unroll
    for (int p = 0; p < PD - 1; ++p)
        if (ci0 + p < nch) step(ci0 + p, p);

    const int ncols = a.dual_F > 0 ? 2 * a.dual_F : a.N;
    float* out = a.part + (int64_t)blockIdx.y * a.M * ncols;
    if constexpr (M32) {
        // accumulator element e of lane l: activation row 8 (e / 4) + 4 (l / 32) + e % 4,
        // weight row of column l % 32
        if (myrv) {
            float rs = 1.f;
            if constexpr (WF == W_INT8) rs = h2f(a.scales[myrow]);
#pragma unroll
            for (int t = 0; t < MT32; ++t)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int m = 32 * t + 8 * (e >> 2) + 4 * h32 + (e & 3);
                    if (m < a.M) out[(int64_t)m * ncols + myrow] = acc32[t][e] * rs;
                }
        }
    } else {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if (!rv[s]) continue;
            float rs = 1.f;
            if constexpr (WF == W_INT8) rs = h2f(a.scales[row[s]]);
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int m = 16 * t + 4 * g + i;
                    if (m < a.M) out[(int64_t)m * ncols + row[s]] = acc[t][s][i] * rs;
                }
        }
    }
}

// Tiling: 16-row subtiles per wave (NS) and waves per workgroup (NWV).  bf16 weights
// run four waves of two subtiles; quantised weights run eight (more waves per SIMD to
// overlap the unpacking with the MFMAs and the loads).
struct BatchTiling {
    int nwv, ns;
};
// Narrow matrices (fewer than SB_NARROW_TILES workgroups of the regular tiling; not
// the [gate; up] matrix) take one subtile per wave: twice the workgroups, half the
// split-K factor, half the partial sums for the consumer to read.
#ifndef SB_NARROW_TILES
#define SB_NARROW_TILES 40
#endif
constexpr BatchTiling batch_tiling(int wf, bool narrow) {
    return wf == W_BF16 ? BatchTiling{4, 2} : (narrow ? BatchTiling{8, 1} : BatchTiling{8, 2});
}
static bool batch_narrow(int N, int dual_F, int wf) {
    const BatchTiling T = batch_tiling(wf, false);
    return wf != W_BF16 && dual_F == 0 && (N + T.nwv * 16 * T.ns - 1) / (T.nwv * 16 * T.ns) < SB_NARROW_TILES;
}

#ifndef SB_M32
#define SB_M32 1
#endif
template <int WF, int MT, bool NARROW>
static hipError_t launch_batch(const SkinnyArgs& a, int ks, hipStream_t st) {
    constexpr BatchTiling T = batch_tiling(WF, NARROW);
    static_assert((NARROW || T.ns % 2 == 0) && T.nwv * 64 <= 1024, "tiling");
    // batches above 16 on two-block waves: 32x32x16 MFMA over whole 32-row activation tiles
    constexpr bool M32 = SB_M32 && !NARROW && MT >= 2;
    constexpr int MTL = M32 ? (MT + 1) / 2 * 2 : MT;
    dim3 grid(skinny_batch_tiles(a.N, a.dual_F, WF), ks);
    FP_LAUNCH((skinny_batch_kernel<WF, MTL, T.ns, T.nwv, M32>), grid, dim3(64 * T.nwv), 0, st, a);
    return hipGetLastError();
}

template <int WF, int MT>
static hipError_t launch_batch_n(const SkinnyArgs& a, int ks, hipStream_t st) {
    if constexpr (WF != W_BF16) {
        if (batch_narrow(a.N, a.dual_F, WF)) return launch_batch<WF, MT, true>(a, ks, st);
    }
    return launch_batch<WF, MT, false>(a, ks, st);
}

template <int WF>
static hipError_t launch_batch_w(const SkinnyArgs& a, int ks, hipStream_t st) {
    switch ((a.M + 15) / 16) {
        case 1: return launch_batch_n<WF, 1>(a, ks, st);
        case 2: return launch_batch_n<WF, 2>(a, ks, st);
        case 3: return launch_batch_n<WF, 3>(a, ks, st);
        case 4: return launch_batch_n<WF, 4>(a, ks, st);
        default: return hipErrorInvalidValue;
    }
}

int skinny_batch_rows(int N, int dual_F, int wf) {
    const BatchTiling T = batch_tiling(wf, batch_narrow(N, dual_F, wf));
    return T.nwv * 16 * T.ns;
}

int skinny_batch_tiles(int N, int dual_F, int wf) {
    const int rows = skinny_batch_rows(N, dual_F, wf);
    return dual_F > 0 ? (dual_F + rows / 2 - 1) / (rows / 2) : (N + rows - 1) / rows;
}

int skinny_batch_chunk() { return SB_KC; }

hipError_t launch_skinny_batch(const SkinnyArgs& a, int wf, int ks, hipStream_t st) {
    if (a.M < 1 || a.M > 64 || a.xf != XF_COPY || a.krange <= 0 || a.krange % SB_KC != 0) return hipErrorInvalidValue;
    if ((int64_t)ks * a.krange < a.K || (int64_t)(ks - 1) * a.krange >= a.K) return hipErrorInvalidValue;
    if (wf == W_INT4 && a.sz == nullptr) return hipErrorInvalidValue;
    const int64_t nrows = a.dual_F > 0 ? 2 * (int64_t)a.dual_F : a.N;
    if (nrows % 16 != 0 || (nrows / 16) * a.kst * 1024 >= ((int64_t)1 << 32) - 16) return hipErrorInvalidValue;   // buffer offsets are 32-bit
    switch (wf) {
        case W_BF16: return launch_batch_w<W_BF16>(a, ks, st);
        case W_INT8: return launch_batch_w<W_INT8>(a, ks, st);
        case W_INT4: return launch_batch_w<W_INT4>(a, ks, st);
        default: return hipErrorInvalidValue;
    }
}

template <int WF, int MT, int NS, int XF>
static hipError_t launch4(const SkinnyArgs& a, dim3 grid, hipStream_t st) {
#ifdef SKINNY_UNR
    constexpr int UNR = SKINNY_UNR;
#else
    constexpr int UNR = (WF == W_INT4) ? 2 : 4;
#endif
    const size_t lds = (size_t)a.M * (a.krange + SK_PAD) * 2;
    FP_LAUNCH((skinny_kernel<WF, MT, NS, UNR, XF>), grid, dim3(256), lds, st, a);
    return hipGetLastError();
}

template <int WF, int MT, int NS>
static hipError_t launch3(const SkinnyArgs& a, dim3 grid, hipStream_t st) {
    switch (a.xf) {
        case XF_COPY: return launch4<WF, MT, NS, XF_COPY>(a, grid, st);
        case XF_NORM: return launch4<WF, MT, NS, XF_NORM>(a, grid, st);
        case XF_SWIGLU: return launch4<WF, MT, NS, XF_SWIGLU>(a, grid, st);
        case XF_MERGE: return launch4<WF, MT, NS, XF_MERGE>(a, grid, st);
        default: return hipErrorInvalidValue;
    }
}

// subtiles per wave: batches stream more rows per workgroup so the staged activation
// slice is shared by more weights
// One 16-token tile: the schedule runs this kernel for a single sequence only (batches
// use skinny_batch_kernel).
static int skinny_ns(int M) { return (void)M, SKINNY_NS; }

template <int WF>
static hipError_t launch2(const SkinnyArgs& a, dim3 grid, hipStream_t st) {
    if (a.M < 1 || a.M > 16) return hipErrorInvalidValue;
    return launch3<WF, 1, SKINNY_NS>(a, grid, st);
}

int skinny_kstep(int wf) { return weight_kstep(wf); }

int skinny_max_krange(int M) {
    int kr = SK_LDS_ELEMS / (M > 0 ? M : 1) - SK_PAD;
    return kr - kr % 128;
}

int skinny_tiles(int N, int dual_F, int M) {
    const int ns = skinny_ns(M);
    return dual_F > 0 ? (dual_F + 32 * ns - 1) / (32 * ns) : (N + 64 * ns - 1) / (64 * ns);
}

hipError_t launch_skinny(const SkinnyArgs& a, int wf, int ks, hipStream_t st) {
    if (a.krange > skinny_max_krange(a.M) || a.krange % skinny_kstep(wf) != 0) return hipErrorInvalidValue;
    const int64_t nrows = a.dual_F > 0 ? 2 * (int64_t)a.dual_F : a.N;
    if (nrows % 16 != 0 || (nrows / 16) * a.kst * 1024 >= ((int64_t)1 << 32) - 16) return hipErrorInvalidValue;   // buffer offsets are 32-bit
    dim3 grid(skinny_tiles(a.N, a.dual_F, a.M), ks);
    switch (wf) {
        case W_BF16: return launch2<W_BF16>(a, grid, st);
        case W_INT8: return launch2<W_INT8>(a, grid, st);
        case W_INT4: return launch2<W_INT4>(a, grid, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace fpk
