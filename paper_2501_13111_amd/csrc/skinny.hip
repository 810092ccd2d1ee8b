// Decode projections: weight-streaming skinny GEMM  part[s] = X[M, K] . W[N, K]^T
// over the split-K range s, for M <= 64 tokens (one per sequence in the batch).
//
// Decode is where the fingerprint's per-token time goes (TPOT, paper Sec. 5.3):
// every step streams all weights once, so the kernel is bound by HBM bandwidth.
// Weight-only quantisation (Sec. 3.2) shrinks those bytes; the cost the paper
// points at is converting the codes back to 16-bit values for the arithmetic.
// Here the codes go straight from a 128-bit load into fp16 MFMA operands with a
// few integer ops per dword:
//   bf16   W: 16 B per lane = 8 weights  -> 1 MFMA  (bf16 x bf16)
//   int8   W: 16 B per lane = 16 weights -> 2 MFMAs (fp16 x exact fp16 codes),
//             per-row scale applied once at the end
//   int4   W: 16 B per lane = 32 weights = one 128-group of a row (4 lanes) ->
//             4 MFMAs on exact (q - z), then acc += s * group sum
// MFMA 16x16x32 layout: lane l supplies row (l % 16) of A and column (l % 16) of
// B, each with 8 consecutive k from the lane's k-slice (l / 16); the output lane
// holds C[4 (l/16) + i][l % 16].  A and B use the same k assignment, so any
// permutation of k inside a K-step is allowed; the int4 nibble order on the
// device is chosen so that pairs of nibbles come out as consecutive k.
//
// Workgroup = 4 waves over one 32-row tile (two 16-row subtiles) and one split-K
// range; the waves interleave K-steps and are summed through LDS.  In "dual"
// mode (SwiGLU) subtile 0 reads gate rows f and subtile 1 up rows F + f of the
// concatenated [gate; up] matrix, so one tile covers 16 values of f.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

template <int WF>
struct SkinnyTraits;
template <> struct SkinnyTraits<W_BF16> { static constexpr int KS = 32; static constexpr int NJ = 1; };
template <> struct SkinnyTraits<W_INT8> { static constexpr int KS = 64; static constexpr int NJ = 2; };
template <> struct SkinnyTraits<W_INT4> { static constexpr int KS = 128; static constexpr int NJ = 4; };

template <int WF, int MT, int UNR>
__global__ void __launch_bounds__(256) skinny_kernel(SkinnyArgs a) {
    constexpr int KS = SkinnyTraits<WF>::KS;
    constexpr int NJ = SkinnyTraits<WF>::NJ;
    constexpr int KL = KS / 4;   // k per lane group in one K-step
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    __shared__ f32x4 red[3][MT][2][64];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int tb = blockIdx.x, sp = blockIdx.y;
    const int kb = sp * a.krange;
    const int ke = min(a.K, kb + a.krange);

    int row[2];
    bool rv[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        if (a.dual_F > 0) {
            const int f = tb * 16 + r;
            rv[s] = f < a.dual_F;
            row[s] = s * a.dual_F + f;
        } else {
            row[s] = tb * 32 + 16 * s + r;
            rv[s] = row[s] < a.N;
        }
    }

    f32x4 acc[MT][2];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int s = 0; s < 2; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};

    bool mv[MT];
    const uint16_t* xrow[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        mv[t] = (16 * t + r) < a.M;
        xrow[t] = a.X + (int64_t)(mv[t] ? 16 * t + r : 0) * a.K;
    }

    for (int k0 = kb + w * KS; k0 < ke; k0 += 4 * KS * UNR) {
        u32x4 wv[UNR][2];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int kk = k0 + u * 4 * KS;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                wv[u][s] = u32x4{0u, 0u, 0u, 0u};
                if (rv[s] && kk + KL * g < ke) {
                    if constexpr (WF == W_BF16) {
                        wv[u][s] = *(const u32x4*)((const uint16_t*)a.W + (int64_t)row[s] * a.K + kk + 8 * g);
                    } else if constexpr (WF == W_INT8) {
                        wv[u][s] = *(const u32x4*)((const int8_t*)a.W + (int64_t)row[s] * a.K + kk + 16 * g);
                    } else {
                        wv[u][s] = *(const u32x4*)((const uint32_t*)a.W + (int64_t)row[s] * (a.K / 8) + (kk + 32 * g) / 8);
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int kk = k0 + u * 4 * KS;
            if (kk >= ke) break;
            // B operands (dequantised weights) for the NJ MFMAs of this K-step
            u32x4 bop[NJ][2];
            float gscale[2];
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                if constexpr (WF == W_BF16) {
                    bop[0][s] = wv[u][s];
                } else if constexpr (WF == W_INT8) {
                    const u32x2 c0 = i8x4_to_f16x4(wv[u][s].x), c1 = i8x4_to_f16x4(wv[u][s].y);
                    const u32x2 c2 = i8x4_to_f16x4(wv[u][s].z), c3 = i8x4_to_f16x4(wv[u][s].w);
                    bop[0][s] = u32x4{c0.x, c0.y, c1.x, c1.y};
                    bop[1][s] = u32x4{c2.x, c2.y, c3.x, c3.y};
                } else {
                    const int grp = kk / 128;
                    float sc = 0.f, zz = 0.f;
                    if (rv[s]) {
                        sc = h2f(a.scales[(int64_t)row[s] * (a.K / 128) + grp]);
                        zz = h2f(a.zeros[(int64_t)row[s] * (a.K / 128) + grp]);
                    }
                    gscale[s] = sc;
                    const _Float16 bz = (_Float16)(1024.0f + zz);
                    const f16x2 bias = {bz, bz};
                    bop[0][s] = i4x8_to_f16x8(wv[u][s].x, bias);
                    bop[1][s] = i4x8_to_f16x8(wv[u][s].y, bias);
                    bop[2][s] = i4x8_to_f16x8(wv[u][s].z, bias);
                    bop[3][s] = i4x8_to_f16x8(wv[u][s].w, bias);
                }
            }
            f32x4 tmp[MT][2];
            if constexpr (WF == W_INT4) {
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int s = 0; s < 2; ++s) tmp[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                // k-offset of this MFMA's 8 values for lane group g
                int koff;
                if constexpr (WF == W_BF16) koff = kk + 8 * g;
                else if constexpr (WF == W_INT8) koff = kk + 16 * g + 8 * j;
                else koff = kk + 32 * g + 8 * j;
                const bool kin = kk + KL * g < ke;
#pragma unroll
                for (int t = 0; t < MT; ++t) {
                    u32x4 av = u32x4{0u, 0u, 0u, 0u};
                    if (mv[t] && kin) av = *(const u32x4*)(xrow[t] + koff);
#pragma unroll
                    for (int s = 0; s < 2; ++s) {
                        if constexpr (WF == W_INT4) tmp[t][s] = mfma16<AF>(av, bop[j][s], tmp[t][s]);
                        else acc[t][s] = mfma16<AF>(av, bop[j][s], acc[t][s]);
                    }
                }
            }
            if constexpr (WF == W_INT4) {
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int s = 0; s < 2; ++s) acc[t][s] += gscale[s] * tmp[t][s];
            }
        }
    }

    // sum the four waves' partial sums through LDS
    if (w > 0) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int s = 0; s < 2; ++s) red[w - 1][t][s][lane] = acc[t][s];
    }
    __syncthreads();
    if (w != 0) return;
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int s = 0; s < 2; ++s)
            acc[t][s] += red[0][t][s][lane] + red[1][t][s][lane] + red[2][t][s][lane];

    const int ncols = a.dual_F > 0 ? 2 * a.dual_F : a.N;
    float* out = a.part + (int64_t)sp * a.M * ncols;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        if (!rv[s]) continue;
        float rs = 1.f;
        if constexpr (WF == W_INT8) rs = h2f(a.scales[row[s]]);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = 16 * t + 4 * g + i;
                if (m < a.M) out[(int64_t)m * ncols + row[s]] = acc[t][s][i] * rs;
            }
        }
    }
}

template <int WF, int MT>
static hipError_t launch_mt(const SkinnyArgs& a, dim3 grid, hipStream_t st) {
    constexpr int UNR = (WF == W_INT4) ? 2 : 4;
    hipLaunchKernelGGL((skinny_kernel<WF, MT, UNR>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int WF>
static hipError_t launch_wf(const SkinnyArgs& a, dim3 grid, hipStream_t st) {
    const int mt = (a.M + 15) / 16;
    switch (mt) {
        case 1: return launch_mt<WF, 1>(a, grid, st);
        case 2: return launch_mt<WF, 2>(a, grid, st);
        case 3: return launch_mt<WF, 3>(a, grid, st);
        case 4: return launch_mt<WF, 4>(a, grid, st);
        default: return hipErrorInvalidValue;
    }
}

int skinny_kstep(int wf) { return wf == W_BF16 ? 32 : (wf == W_INT8 ? 64 : 128); }

hipError_t launch_skinny(const SkinnyArgs& a, int wf, int ks, hipStream_t st) {
    const int tiles = a.dual_F > 0 ? (a.dual_F + 15) / 16 : (a.N + 31) / 32;
    dim3 grid(tiles, ks);
    switch (wf) {
        case W_BF16: return launch_wf<W_BF16>(a, grid, st);
        case W_INT8: return launch_wf<W_INT8>(a, grid, st);
        case W_INT4: return launch_wf<W_INT4>(a, grid, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace fpk
